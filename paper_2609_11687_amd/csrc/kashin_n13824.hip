// Launch configuration for vectors of length 13824.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(13824, 448, 2, 16, 16, 2, 3, 9)
}  // namespace kashin
