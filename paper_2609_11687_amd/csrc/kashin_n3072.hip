// Launch configuration for vectors of length 3072.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(3072, 192, 3, 16, 16, 4, 3)
}  // namespace kashin
