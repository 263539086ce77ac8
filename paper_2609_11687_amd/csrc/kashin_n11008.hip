// Launch configuration for vectors of length 11008.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(11008, 768, 3, 16, 43, 16)
}  // namespace kashin
