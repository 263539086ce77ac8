// Launch configuration for vectors of length 4096.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(4096, 256, 3, 16, 16, 16)
}  // namespace kashin
