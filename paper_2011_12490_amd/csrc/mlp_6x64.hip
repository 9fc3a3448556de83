// Grouped per-head MLP variants: 6 layers of 64, no skip, colour hidden layer of 32.
#include "mlp_kernel.h"

namespace derf {

const MlpVariant *mlp_variant_6x64(bool bf16)
{
    return bf16 ? variant<Cfg<true, 64, 6, -1, 32, 10>>() : variant<Cfg<false, 64, 6, -1, 32, 10>>();
}

}  // namespace derf
