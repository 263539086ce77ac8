// Launch configuration for vectors of length 768.
#include "kashin_pair_impl.h"

namespace kashin {
KASHIN_DEFINE_SIZE(768, 64, 3, 16, 3, 16)
}  // namespace kashin
