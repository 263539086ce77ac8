// Launch configuration for vectors of length 6144.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(6144, 384, 3, 16, 16, 8, 3)
}  // namespace kashin
