// Grouped per-head MLP variants: 8 layers of 128, skip at layer 5, colour hidden layer of 64.
#include "mlp_kernel.h"

namespace derf {

const MlpVariant *mlp_variant_8x128(bool bf16)
{
    return bf16 ? variant<Cfg<true, 128, 8, 5, 64, 10>>() : variant<Cfg<false, 128, 8, 5, 64, 10>>();
}

}  // namespace derf
