// Grouped per-head MLP variants: 8 layers of 256, skip at layer 5, colour hidden layer of 128 (the NeRF head; bf16 only).
#include "mlp_kernel.h"

namespace derf {

const MlpVariant *mlp_variant_8x256(bool bf16)
{
    return bf16 ? variant<Cfg<true, 256, 8, 5, 128, 10>>() : nullptr;
}

}  // namespace derf
