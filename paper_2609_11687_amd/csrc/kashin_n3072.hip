// Launch configuration for vectors of length 3072.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(3072, 256, 3, 16, 12, 16)
}  // namespace kashin
