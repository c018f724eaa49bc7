// kernels_quant.hip -- drafter refresh: RTN int4 quantization of a weight
// matrix into the packed tile layout read by the int4 GEMMs (Sec. 4.1: the
// FFN and QKVO projections are re-quantized at every training step).
//
// Symmetric groups of 128 consecutive weights along K within an output row:
//   s = fp16(max|w| / 7),  q = clamp(rint(w / s), -8, 7)  (q = 0 when s = 0).
// fp32 division is correctly rounded and rint rounds half to even, so codes
// and scales are a deterministic function of the weights.
#include "common.h"
#include "kernels.h"

namespace {

// One wave per (32-column block nb, group g).  Lane l takes column
// 32 nb + (l & 31) and k-half h = l >> 5: for k-step st = 0..7 the 8 weights
// k = 128 g + 16 st + 8 h + e, which become its packed word st (the layout
// the int4 GEMM reads, kernels_q4.hip).
template <typename T>
__global__ void __launch_bounds__(64) k_quant_rtn4(const T* __restrict__ W, int N, int K, uint32_t* __restrict__ Wq,
                                                   uint16_t* __restrict__ Sc)
{
    const int lane = threadIdx.x;
    const int nb = blockIdx.x, g = blockIdx.y;
    const int G = K / 128;
    const int n = nb * 32 + (lane & 31), h = lane >> 5;
    const T* wr = W + (size_t)n * K + (size_t)g * 128 + 8 * h;
    float v[8][8];
    float amax = 0.f;
#pragma unroll
    for (int st = 0; st < 8; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            v[st][e] = elem<T>::load(wr, (size_t)st * 16 + e);
            amax = fmaxf(amax, fabsf(v[st][e]));
        }
    amax = fmaxf(amax, __shfl_xor(amax, 32, WAVE));
    const _Float16 sh = (_Float16)(amax / 7.0f);
    const float s = (float)sh;
    u32x4 out[2];
#pragma unroll
    for (int st = 0; st < 8; ++st) {
        uint32_t word = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            int q = 0;
            if (s != 0.f) {
                const float r = rintf(v[st][e] / s);
                q = r < -8.f ? -8 : (r > 7.f ? 7 : (int)r);
            }
            word |= (uint32_t)(q + 8) << (4 * (e >> 1) + 16 * (e & 1));
        }
        out[st >> 2][st & 3] = word;
    }
    u32x4* dst = (u32x4*)Wq + ((size_t)nb * G + g) * 128;
    dst[lane] = out[0];
    dst[64 + lane] = out[1];
    if (lane < 32) Sc[((size_t)nb * G + g) * 32 + lane] = __builtin_bit_cast(uint16_t, sh);
}

}  // namespace

void launch_quant_rtn4(const void* W, int w_f32, int N, int K, uint32_t* Wq, uint16_t* Sc, hipStream_t s)
{
    dim3 grid(N / 32, K / 128);
    if (w_f32) k_quant_rtn4<float><<<grid, 64, 0, s>>>((const float*)W, N, K, Wq, Sc);
    else k_quant_rtn4<uint16_t><<<grid, 64, 0, s>>>((const uint16_t*)W, N, K, Wq, Sc);
}
