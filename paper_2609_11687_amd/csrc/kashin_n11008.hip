// Launch configuration for vectors of length 11008.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(11008, 704, 3, 16, 16, 43)
}  // namespace kashin
