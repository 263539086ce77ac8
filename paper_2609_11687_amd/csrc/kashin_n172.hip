// Launch configuration for vectors of length 172.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(172, 64, 2, 4, 43)
}  // namespace kashin
