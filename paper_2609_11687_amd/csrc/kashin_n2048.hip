// Launch configuration for vectors of length 2048.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(2048, 128, 2, 16, 8, 16)
}  // namespace kashin
