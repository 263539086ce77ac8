// Launch configuration for vectors of length 64.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(64, 64, 2, 8, 8)
}  // namespace kashin
