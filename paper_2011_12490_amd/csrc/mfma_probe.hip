// Matrix-core throughput probe for gfx950: how fast the 32x32x16 bf16 MFMA
// runs back to back on every SIMD of the chip, with operands of a chosen bit
// pattern and an optional share of ordinary vector instructions beside each
// MFMA.  The grouped head MLP issues this MFMA; its rate under the same
// operand statistics and instruction mix is the ceiling that the MLP's
// fraction of the nominal 2.5 PFLOP/s is to be read against (the chip lowers
// its clock under matrix load, more so when the operands toggle more bits).
//
// Not part of the renderer: a separate library (libderf_probe.so) that the
// benchmark loads for its --mfma-ceiling report.
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kChains = 4;  // independent accumulators per wave

__device__ __forceinline__ uint32_t mix(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

// One operand register set (8 bf16 values) for pattern `mode`:
// 0 random values in [-1, 1) (every bit toggles between operands),
// 1 one constant value, 2 zeros.  (Mode 3 of the kernel, random A and a B
// whose 32 columns are equal, draws both with mode 0.)
__device__ bf16x8 operand(uint32_t seed, int mode)
{
    bf16x8 v;
    for (int j = 0; j < 8; ++j) {
        float f = 0.0f;
        if (mode == 0)
            f = (float)(int)(mix(seed * 8u + (uint32_t)j) >> 8) * 0x1.0p-23f - 1.0f;
        else if (mode == 1)
            f = 0.375f;
        v[j] = (__bf16)f;
    }
    return v;
}

// valu: vector instructions issued per MFMA beside it (0, 2 or 4), the
// conversion and ReLU pattern of the MLP's epilogue (a bf16 pack and a packed
// int16 max per pair of accumulator values) on an independent register set.
template <int VALU>
__global__ __launch_bounds__(256, 2) void mfma_probe_kernel(int iters, uint32_t seed, int mode,
                                                            float *out)
{
    const uint32_t lane_seed = seed ^ (blockIdx.x * 256u + threadIdx.x);
    // mode 3: B lane n + 32 g holds column n's k-entries of group g; one seed
    // per half-wave makes the 32 columns (the samples) equal, A stays random
    const uint32_t col_seed = seed ^ (blockIdx.x * 256u + (threadIdx.x & ~31u));
    const int draw = mode == 3 ? 0 : mode;
    bf16x8 a[kChains], b[kChains];
    f32x16 acc[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k) {
        a[k] = operand(lane_seed * 131u + (uint32_t)k, draw);
        b[k] = operand((mode == 3 ? col_seed : lane_seed) * 137u + (uint32_t)k + 7u, draw);
        for (int i = 0; i < 16; ++i)
            acc[k][i] = 0.0f;
    }
    // two chains of (bf16 pack, packed max), each feeding the next pack, so
    // that neither instruction can leave the loop
    float side[4] = {1.0f, -2.0f, 3.0f, -4.0f};
    i16x2 packed[2] = {i16x2{0, 0}, i16x2{0, 0}};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int k = 0; k < kChains; ++k) {
            acc[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[k], b[(k + 1) % kChains], acc[k],
                                                             0, 0, 0);
            if constexpr (VALU >= 2) {
                const bf16x2 p = __builtin_convertvector(f32x2{side[0], side[1]}, bf16x2);
                packed[0] = __builtin_elementwise_max(__builtin_bit_cast(i16x2, p), packed[0]);
                side[0] = __builtin_bit_cast(float, packed[0]);
            }
            if constexpr (VALU >= 4) {
                const bf16x2 p = __builtin_convertvector(f32x2{side[2], side[3]}, bf16x2);
                packed[1] = __builtin_elementwise_max(__builtin_bit_cast(i16x2, p), packed[1]);
                side[2] = __builtin_bit_cast(float, packed[1]);
            }
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int k = 0; k < kChains; ++k)
        for (int i = 0; i < 16; ++i)
            s += acc[k][i];
    s += (float)packed[0][0] + (float)packed[1][1];
    // one word per lane keeps every chain live; the values are not used
    out[blockIdx.x * 256u + threadIdx.x] = s;
}

}  // namespace

extern "C" {

// Launch the probe: grid workgroups of 256 threads (two per CU fill the
// chip's SIMDs with two waves each), `iters` rounds of kChains MFMAs per
// wave.  mode: 0 random, 1 constant, 2 zero operands, 3 random A with the
// 32 columns of B equal.  out: device float [grid * 256].  valu: 0, 2 or 4.  Returns the HIP
// status of the launch; MFMAs per launch = grid * 4 * iters * kChains.
int derf_probe_mfma(int grid, int iters, unsigned seed, int mode, int valu, float *out,
                    void *stream)
{
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (grid < 1 || iters < 1 || mode < 0 || mode > 3 || !out)
        return (int)hipErrorInvalidValue;
    switch (valu) {
    case 0:
        mfma_probe_kernel<0><<<grid, 256, 0, s>>>(iters, seed, mode, out);
        break;
    case 2:
        mfma_probe_kernel<2><<<grid, 256, 0, s>>>(iters, seed, mode, out);
        break;
    case 4:
        mfma_probe_kernel<4><<<grid, 256, 0, s>>>(iters, seed, mode, out);
        break;
    default:
        return (int)hipErrorInvalidValue;
    }
    return (int)hipGetLastError();
}

int derf_probe_chains(void) { return kChains; }

}  // extern "C"
