// Launch configuration for vectors of length 1024.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(1024, 64, 2, 16, 4, 16)
}  // namespace kashin
