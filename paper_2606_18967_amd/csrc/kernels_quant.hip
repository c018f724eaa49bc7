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

template <typename T>
__global__ void __launch_bounds__(64) k_quant_rtn4(const T* __restrict__ W, int N, int K, uint32_t* __restrict__ Wq,
                                                   uint16_t* __restrict__ Sc)
{
    int lane = threadIdx.x;
    int nb = blockIdx.x, g = blockIdx.y;
    int G = K / 128;
    int n = nb * 16 + (lane & 15), c = lane >> 4;
    const T* wr = W + (size_t)n * K + (size_t)g * 128 + c * 8;
    float v[4][8];
    float amax = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            v[j][e] = elem<T>::load(wr, (size_t)j * 32 + e);
            amax = fmaxf(amax, fabsf(v[j][e]));
        }
    amax = fmaxf(amax, __shfl_xor(amax, 16, WAVE));
    amax = fmaxf(amax, __shfl_xor(amax, 32, WAVE));
    _Float16 sh = (_Float16)(amax / 7.0f);
    float s = (float)sh;
    u32x4 out;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        uint32_t word = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            int q = 0;
            if (s != 0.f) {
                float r = rintf(v[j][e] / s);
                q = r < -8.f ? -8 : (r > 7.f ? 7 : (int)r);
            }
            word |= (uint32_t)(q + 8) << (4 * (e >> 1) + 16 * (e & 1));
        }
        out[j] = word;
    }
    ((u32x4*)Wq)[((size_t)nb * G + g) * 64 + lane] = out;
    if (lane < 16) Sc[((size_t)nb * G + g) * 16 + lane] = __builtin_bit_cast(uint16_t, sh);
}

}  // namespace

void launch_quant_rtn4(const void* W, int w_f32, int N, int K, uint32_t* Wq, uint16_t* Sc, hipStream_t s)
{
    dim3 grid(N / 16, K / 128);
    if (w_f32) k_quant_rtn4<float><<<grid, 64, 0, s>>>((const float*)W, N, K, Wq, Sc);
    else k_quant_rtn4<uint16_t><<<grid, 64, 0, s>>>((const uint16_t*)W, N, K, Wq, Sc);
}
