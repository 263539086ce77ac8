// Launch configuration for vectors of length 512.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(512, 64, 4, 8, 8, 8)
}  // namespace kashin
