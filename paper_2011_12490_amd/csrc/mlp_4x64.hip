// Grouped per-head MLP variants: 4 layers of 64, no skip, colour straight from [h; gamma(d)] (pos_freqs 6).
#include "mlp_kernel.h"

namespace derf {

const MlpVariant *mlp_variant_4x64(bool bf16)
{
    return bf16 ? variant<Cfg<true, 64, 4, -1, 0, 6>>() : variant<Cfg<false, 64, 4, -1, 0, 6>>();
}

}  // namespace derf
