// Launch configuration for vectors of length 16384.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(16384, 1024, 4, 16, 8, 8, 16)
}  // namespace kashin
