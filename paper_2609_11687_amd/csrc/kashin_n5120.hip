// Launch configuration for vectors of length 5120.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(5120, 320, 3, 16, 16, 4, 5)
}  // namespace kashin
