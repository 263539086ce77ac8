// Launch configuration for vectors of length 8192.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(8192, 512, 2, 16, 16, 16, 2)
}  // namespace kashin
