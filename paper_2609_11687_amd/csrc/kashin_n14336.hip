// Launch configuration for vectors of length 14336.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(14336, 448, 2, 16, 16, 8, 7)
}  // namespace kashin
