// kernels_quant.hip -- drafter refresh: RTN quantization of a weight matrix
// into the packed tile layout read by the drafter GEMMs (Sec. 4.1: the FFN
// and QKVO projections are re-quantized at every training step).
//
// Groups of 128 consecutive weights along K within an output row, one fp16
// scale each:
//   int4 symmetric:   s = fp16(max|w| / 7),   q = clamp(rint(w / s), -8, 7)
//   int4 asymmetric:  s = fp16((max - min) / 15), z = clamp(rint(-min / s), 0, 15),
//                     q = clamp(rint(w / s) + z, 0, 15)   (App. B.2)
//   int8 symmetric:   s = fp16(max|w| / 127), q = clamp(rint(w / s), -128, 127)
// (q = 0, z = 0 when s = 0).  fp32 division is correctly rounded and rint
// rounds half to even, so codes, scales and zero points are a deterministic
// function of the weights.
#include "common.h"
#include "kernels.h"

namespace {

// One wave per (32-column block nb, group g).  Lane l takes column
// 32 nb + (l & 31) and k-half h = l >> 5: for k-step st = 0..7 the 8 weights
// k = 128 g + 16 st + 8 h + e.  In the int4 formats they become its packed
// word st (code e in the nibble at bit 4 (e / 2) + 16 (e % 2)); in the int8
// format its words 2 st and 2 st + 1 (code e in byte e % 4 of word
// 2 st + e / 4) -- the B operand layout of the GEMM's MFMA k-step st
// (kernels_q4.hip).
template <typename T, int FMT>
__global__ void __launch_bounds__(64) k_quant_rtn(const T* __restrict__ W, int N, int K, uint32_t* __restrict__ Wq,
                                                  uint16_t* __restrict__ Sc, uint8_t* __restrict__ Z)
{
    const int lane = threadIdx.x;
    const int nb = blockIdx.x, g = blockIdx.y;
    const int G = K / 128;
    const int n = nb * 32 + (lane & 31), h = lane >> 5;
    const T* wr = W + (size_t)n * K + (size_t)g * 128 + 8 * h;
    float v[8][8];
    float amax = 0.f, lo = INFINITY, hi = -INFINITY;
#pragma unroll
    for (int st = 0; st < 8; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            v[st][e] = elem<T>::load(wr, (size_t)st * 16 + e);
            amax = fmaxf(amax, fabsf(v[st][e]));
            lo = fminf(lo, v[st][e]);
            hi = fmaxf(hi, v[st][e]);
        }
    amax = fmaxf(amax, __shfl_xor(amax, 32, WAVE));
    lo = fminf(lo, __shfl_xor(lo, 32, WAVE));
    hi = fmaxf(hi, __shfl_xor(hi, 32, WAVE));
    const _Float16 sh = (_Float16)(FMT == QF_W4 ? amax / 7.0f : (FMT == QF_W8 ? amax / 127.0f : (hi - lo) / 15.0f));
    const float s = (float)sh;
    int z = 0;
    if (FMT == QF_W4A && s != 0.f) {
        const float zr = rintf(-lo / s);
        z = zr < 0.f ? 0 : (zr > 15.f ? 15 : (int)zr);
    }
    auto code = [&](float w) {   // the stored (unsigned) code
        if (s == 0.f) return FMT == QF_W4 ? 8 : (FMT == QF_W8 ? 128 : 0);
        const float r = rintf(w / s);
        if (FMT == QF_W4) return (r < -8.f ? -8 : (r > 7.f ? 7 : (int)r)) + 8;
        if (FMT == QF_W8) return (r < -128.f ? -128 : (r > 127.f ? 127 : (int)r)) + 128;
        const float rz = r + (float)z;
        return rz < 0.f ? 0 : (rz > 15.f ? 15 : (int)rz);
    };
    if (FMT == QF_W8) {
        u32x4 out[4];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            uint32_t word = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b) word |= (uint32_t)code(v[j >> 1][4 * (j & 1) + b]) << (8 * b);
            out[j >> 2][j & 3] = word;
        }
        u32x4* dst = (u32x4*)Wq + ((size_t)nb * G + g) * 256;
#pragma unroll
        for (int i = 0; i < 4; ++i) dst[64 * i + lane] = out[i];
    } else {
        u32x4 out[2];
#pragma unroll
        for (int st = 0; st < 8; ++st) {
            uint32_t word = 0;
#pragma unroll
            for (int e = 0; e < 8; ++e) word |= (uint32_t)code(v[st][e]) << (4 * (e >> 1) + 16 * (e & 1));
            out[st >> 2][st & 3] = word;
        }
        u32x4* dst = (u32x4*)Wq + ((size_t)nb * G + g) * 128;
        dst[lane] = out[0];
        dst[64 + lane] = out[1];
    }
    if (lane < 32) {
        Sc[((size_t)nb * G + g) * 32 + lane] = __builtin_bit_cast(uint16_t, sh);
        if (FMT == QF_W4A) Z[((size_t)nb * G + g) * 32 + lane] = (uint8_t)z;
    }
}

template <typename T>
void quant_t(int fmt, const T* W, int N, int K, uint32_t* Wq, uint16_t* Sc, uint8_t* Z, hipStream_t s)
{
    dim3 grid(N / 32, K / 128);
    if (fmt == QF_W4A) k_quant_rtn<T, QF_W4A><<<grid, 64, 0, s>>>(W, N, K, Wq, Sc, Z);
    else if (fmt == QF_W8) k_quant_rtn<T, QF_W8><<<grid, 64, 0, s>>>(W, N, K, Wq, Sc, Z);
    else k_quant_rtn<T, QF_W4><<<grid, 64, 0, s>>>(W, N, K, Wq, Sc, Z);
}

}  // namespace

void launch_quant(int fmt, const void* W, int w_f32, int N, int K, uint32_t* Wq, uint16_t* Sc, uint8_t* Z,
                  hipStream_t s)
{
    if (w_f32) quant_t<float>(fmt, (const float*)W, N, K, Wq, Sc, Z, s);
    else quant_t<uint16_t>(fmt, (const uint16_t*)W, N, K, Wq, Sc, Z, s);
}
