// Launch configuration for vectors of length 96.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(96, 64, 2, 16, 3, 2)
}  // namespace kashin
