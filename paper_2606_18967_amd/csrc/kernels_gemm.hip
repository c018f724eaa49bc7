// kernels_gemm.hip -- the projections: C[M][N] (fp32) = or += A[M][K] W^T.
//
// Weights are row-major [N][K] (K contiguous), activations [M][K].
//   - gemm_bf16:  bf16 x bf16 on MFMA (v_mfma_f32_16x16x32_bf16), LDS-tiled.
//   - gemm_q4_f16: int4 group-128 weights in the packed tile layout written by
//     the RTN quantizer, dequantized in registers to exact fp16 integers and
//     fed to v_mfma_f32_16x16x32_f16; the per-group fp16 scale is applied to
//     the fp32 partial sum of each group.
//   - gemm_f32 / gemm_q4_f32: plain VALU versions for fp32 models.
//
// Packed int4 layout (per weight matrix, N % 16 == 0, K % 128 == 0): for
// n-block nb = n/16 and group g = k/128 there are 64 lanes x 4 words; lane
// l = (n % 16) + 16*c holds, in word j, the 8 weights k = 128g + 32j + 8c + e
// (e = 0..7) of row n, element e in the nibble at bit 4*(e/2) + 16*(e%2),
// stored as code + 8.  Word address: ((nb*G + g)*64 + l)*4 + j.  Scales are
// fp16 at ((nb*G + g)*16 + n%16).
#include "common.h"
#include "kernels.h"

namespace {

// ------------------------------------------------------------------ bf16 MFMA
constexpr int BM = 64, BN = 64, BK = 64, LDT = BK + 8;   // padded LDS row (bf16 elements)

__global__ void __launch_bounds__(256) k_gemm_bf16(const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
                                                   float* __restrict__ C, int M, int N, int K, int ldc, int mode)
{
    __shared__ __attribute__((aligned(16))) uint16_t As[BM * LDT];
    __shared__ __attribute__((aligned(16))) uint16_t Ws[BN * LDT];
    int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    int wm = w >> 1, wn = w & 1;
    int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    floatx4 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = (floatx4){0.f, 0.f, 0.f, 0.f};

    for (int k0 = 0; k0 < K; k0 += BK) {
        // 64 rows x 64 k = 512 chunks of 8 bf16 for each operand, 2 per thread
        u32x4 ra[2], rw[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            int ch = tid + t * 256;
            int row = ch >> 3, kc = (ch & 7) * 8;
            int gm = m0 + row;
            ra[t] = gm < M ? *(const u32x4*)(A + (size_t)gm * K + k0 + kc) : (u32x4){0u, 0u, 0u, 0u};
            rw[t] = *(const u32x4*)(W + (size_t)(n0 + row) * K + k0 + kc);
        }
        __syncthreads();
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            int ch = tid + t * 256;
            int row = ch >> 3, kc = (ch & 7) * 8;
            *(u32x4*)(As + row * LDT + kc) = ra[t];
            *(u32x4*)(Ws + row * LDT + kc) = rw[t];
        }
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            int kk = ks * 32 + (lane >> 4) * 8;
            bf16x8 af[2], bfr[2];
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                int row = wm * 32 + a * 16 + (lane & 15);
                af[a] = *(const bf16x8*)(As + row * LDT + kk);
            }
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                int row = wn * 32 + b * 16 + (lane & 15);
                bfr[b] = *(const bf16x8*)(Ws + row * LDT + kk);
            }
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
        }
    }
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            int col = n0 + wn * 32 + b * 16 + (lane & 15);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                int row = m0 + wm * 32 + a * 16 + (lane >> 4) * 4 + i;
                if (row < M) {
                    float* cp = C + (size_t)row * ldc + col;
                    *cp = mode == GEMM_ADD ? *cp + acc[a][b][i] : acc[a][b][i];
                }
            }
        }
}

// ------------------------------------------------------------------ fp32 VALU
constexpr int FT = 64, FK = 16;

__global__ void __launch_bounds__(256) k_gemm_f32(const float* __restrict__ A, const float* __restrict__ W,
                                                  float* __restrict__ C, int M, int N, int K, int ldc, int mode)
{
    __shared__ float As[FK][FT + 1];
    __shared__ float Ws[FK][FT + 1];
    int tid = threadIdx.x;
    int tm = tid >> 4, tn = tid & 15;   // 16 x 16 threads, 4 x 4 outputs each
    int m0 = blockIdx.y * FT, n0 = blockIdx.x * FT;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += FK) {
        for (int t = tid; t < FT * FK; t += 256) {
            int row = t / FK, kk = t % FK;
            int gm = m0 + row;
            As[kk][row] = gm < M ? A[(size_t)gm * K + k0 + kk] : 0.f;
            Ws[kk][row] = W[(size_t)(n0 + row) * K + k0 + kk];
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < FK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) { a[i] = As[kk][tm * 4 + i]; b[i] = Ws[kk][tn * 4 + i]; }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        int row = m0 + tm * 4 + i;
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float* cp = C + (size_t)row * ldc + n0 + tn * 4 + j;
            *cp = mode == GEMM_ADD ? *cp + acc[i][j] : acc[i][j];
        }
    }
}

// ------------------------------------------------------------------ int4 dequant helpers
// One packed word -> 8 fp16 values equal to the signed codes (exact).
__device__ __forceinline__ half8 dequant8(uint32_t x)
{
    const uint32_t MAGIC = 0x64006400u;       // fp16 1024.0 in both halves
    uint32_t r0 = (x & 0x000F000Fu) | MAGIC;
    uint32_t r1 = ((x >> 4) & 0x000F000Fu) | MAGIC;
    uint32_t r2 = ((x >> 8) & 0x000F000Fu) | MAGIC;
    uint32_t r3 = ((x >> 12) & 0x000F000Fu) | MAGIC;
    const half2v bias = {(_Float16)1032.0f, (_Float16)1032.0f};   // 1024 + 8
    half2v h0 = __builtin_bit_cast(half2v, r0) - bias;
    half2v h1 = __builtin_bit_cast(half2v, r1) - bias;
    half2v h2 = __builtin_bit_cast(half2v, r2) - bias;
    half2v h3 = __builtin_bit_cast(half2v, r3) - bias;
    half8 out = {h0[0], h0[1], h1[0], h1[1], h2[0], h2[1], h3[0], h3[1]};
    return out;
}

__device__ __forceinline__ float f16_bits_to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }

// ------------------------------------------------------------------ int4 x fp16 MFMA
// One wave per (16-column n-block, 64-row m-tile); A fragments straight from
// global memory.
__global__ void __launch_bounds__(64) k_gemm_q4_f16(const _Float16* __restrict__ A, const uint32_t* __restrict__ Wq,
                                                    const uint16_t* __restrict__ Sc, float* __restrict__ C, int M,
                                                    int N, int K, int ldc, int mode)
{
    int lane = threadIdx.x;
    int nb = blockIdx.x;
    int m0 = blockIdx.y * 64;
    int G = K / 128;
    int mtiles = min(4, (M - m0 + 15) / 16);
    floatx4 acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = (floatx4){0.f, 0.f, 0.f, 0.f};
    const u32x4* wp = (const u32x4*)Wq + (size_t)nb * G * 64 + lane;
    const uint16_t* sp = Sc + (size_t)nb * G * 16 + (lane & 15);
    int arow = lane & 15, akc = (lane >> 4) * 8;
    for (int g = 0; g < G; ++g) {
        u32x4 wv = wp[(size_t)g * 64];
        float s = f16_bits_to_f32(sp[(size_t)g * 16]);
        floatx4 tmp[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) tmp[t] = (floatx4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            half8 bq = dequant8(wv[j]);
            int k = g * 128 + j * 32 + akc;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                if (t < mtiles) {
                    int row = m0 + t * 16 + arow;
                    half8 af = row < M ? *(const half8*)(A + (size_t)row * K + k) : (half8){};
                    tmp[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, bq, tmp[t], 0, 0, 0);
                }
            }
        }
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[t][i] += s * tmp[t][i];
    }
    int col = nb * 16 + (lane & 15);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        if (t >= mtiles) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            int row = m0 + t * 16 + (lane >> 4) * 4 + i;
            if (row < M) {
                float* cp = C + (size_t)row * ldc + col;
                *cp = mode == GEMM_ADD ? *cp + acc[t][i] : acc[t][i];
            }
        }
    }
}

// ------------------------------------------------------------------ int4 x fp32 VALU
__device__ __forceinline__ int q4_code(const uint32_t* Wq, int G, int n, int k)
{
    int nb = n >> 4, g = k >> 7;
    int l = (n & 15) + 16 * ((k & 31) >> 3);
    int j = (k & 127) >> 5, e = k & 7;
    uint32_t word = Wq[(((size_t)nb * G + g) * 64 + l) * 4 + j];
    return (int)((word >> (4 * (e >> 1) + 16 * (e & 1))) & 15u) - 8;
}

__global__ void __launch_bounds__(256) k_gemm_q4_f32(const float* __restrict__ A, const uint32_t* __restrict__ Wq,
                                                     const uint16_t* __restrict__ Sc, float* __restrict__ C, int M,
                                                     int N, int K, int ldc, int mode)
{
    int n = blockIdx.x * 64 + (threadIdx.x & 63);
    int m = blockIdx.y * 4 + (threadIdx.x >> 6);
    if (m >= M || n >= N) return;
    int G = K / 128;
    const float* ar = A + (size_t)m * K;
    float acc = 0.f;
    for (int g = 0; g < G; ++g) {
        float part = 0.f;
        for (int k = g * 128; k < g * 128 + 128; ++k) part += ar[k] * (float)q4_code(Wq, G, n, k);
        acc += f16_bits_to_f32(Sc[((size_t)(n >> 4) * G + g) * 16 + (n & 15)]) * part;
    }
    float* cp = C + (size_t)m * ldc + n;
    *cp = mode == GEMM_ADD ? *cp + acc : acc;
}

}  // namespace

void launch_gemm_bf16(const uint16_t* A, const uint16_t* W, float* C, int M, int N, int K, int ldc, gemm_mode mode,
                      hipStream_t s)
{
    dim3 grid(N / BN, (M + BM - 1) / BM);
    k_gemm_bf16<<<grid, 256, 0, s>>>(A, W, C, M, N, K, ldc, mode);
}

void launch_gemm_f32(const float* A, const float* W, float* C, int M, int N, int K, int ldc, gemm_mode mode,
                     hipStream_t s)
{
    dim3 grid(N / FT, (M + FT - 1) / FT);
    k_gemm_f32<<<grid, 256, 0, s>>>(A, W, C, M, N, K, ldc, mode);
}

void launch_gemm_q4_f16(const _Float16* A, const uint32_t* Wq, const uint16_t* Sc, float* C, int M, int N, int K,
                        int ldc, gemm_mode mode, hipStream_t s)
{
    dim3 grid(N / 16, (M + 63) / 64);
    k_gemm_q4_f16<<<grid, 64, 0, s>>>(A, Wq, Sc, C, M, N, K, ldc, mode);
}

void launch_gemm_q4_f32(const float* A, const uint32_t* Wq, const uint16_t* Sc, float* C, int M, int N, int K,
                        int ldc, gemm_mode mode, hipStream_t s)
{
    dim3 grid((N + 63) / 64, (M + 3) / 4);
    k_gemm_q4_f32<<<grid, 256, 0, s>>>(A, Wq, Sc, C, M, N, K, ldc, mode);
}
