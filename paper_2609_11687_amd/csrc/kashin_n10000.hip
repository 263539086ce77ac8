// Launch configuration for vectors of length 10000.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(10000, 640, 3, 16, 5, 5, 5, 5)
}  // namespace kashin
