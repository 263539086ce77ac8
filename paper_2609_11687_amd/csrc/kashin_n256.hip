// Launch configuration for vectors of length 256.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(256, 64, 2, 16, 16)
}  // namespace kashin
