// mfma_valu.hip -- register-only microbenchmark of the matrix cores on gfx950:
//   1. the sustained rate of the MFMA shapes the kernels use (32x32x16 and
//      16x16x32, f16 and bf16), four independent accumulators per wave, one
//      or two waves per SIMD;
//   2. how much independent VALU work issued between MFMAs slows them: two
//      MFMAs plus NV VALU ops (fp32 FMA, packed fp16 FMA or v_and_or_b32,
//      the ops of the drafter GEMM's int4 dequantization) per iteration.
// It touches no memory besides one store per thread at the end, so the
// figures are the core's own: the drafter GEMM (k_gemm_q4) needs about two
// MFMAs and 13 VALU ops per 512 weights per wave, and part 2 gives the time
// of exactly that mix.
//
// Build and run (not part of the library):
//   hipcc -O3 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//         paper_2606_18967_amd/probes/mfma_valu.hip -o /tmp/mfma_valu && /tmp/mfma_valu
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

#define CK(x)                                                                                    \
    do {                                                                                         \
        hipError_t e_ = (x);                                                                     \
        if (e_ != hipSuccess) {                                                                  \
            printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);                \
            exit(1);                                                                             \
        }                                                                                        \
    } while (0)

constexpr int CUS = 256;    // one work-group per CU, 4 * waves-per-SIMD waves each

// ---------------------------------------------------------------- 1. shape rates
// KIND 0: 32x32x16 f16, 1: 32x32x16 bf16, 2: 16x16x32 f16, 3: 16x16x32 bf16;
// each iteration does 4 x 32768 FLOP (four 32x32x16 or eight 16x16x32)
template <int KIND>
__global__ void k_rate(float* out, int iters)
{
    const int lane = threadIdx.x & 63;
    half8 a, b;
    bf16x8 c, d;
    for (int i = 0; i < 8; ++i) {
        a[i] = (_Float16)(0.001f * (lane + i));
        b[i] = (_Float16)(0.002f * (lane - i));
        c[i] = (__bf16)(0.001f * (lane + i));
        d[i] = (__bf16)(0.002f * (lane - i));
    }
    floatx16 x0 = {}, x1 = {}, x2 = {}, x3 = {};
    floatx4 y0 = {}, y1 = {}, y2 = {}, y3 = {};
    for (int it = 0; it < iters; ++it) {
        if constexpr (KIND == 0) {
            x0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, x0, 0, 0, 0);
            x1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, x1, 0, 0, 0);
            x2 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, x2, 0, 0, 0);
            x3 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, x3, 0, 0, 0);
        } else if constexpr (KIND == 1) {
            x0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c, d, x0, 0, 0, 0);
            x1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c, d, x1, 0, 0, 0);
            x2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c, d, x2, 0, 0, 0);
            x3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c, d, x3, 0, 0, 0);
        } else {
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                if constexpr (KIND == 2) {
                    y0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, y0, 0, 0, 0);
                    y1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, y1, 0, 0, 0);
                    y2 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, y2, 0, 0, 0);
                    y3 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, y3, 0, 0, 0);
                } else {
                    y0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(c, d, y0, 0, 0, 0);
                    y1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(c, d, y1, 0, 0, 0);
                    y2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(c, d, y2, 0, 0, 0);
                    y3 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(c, d, y3, 0, 0, 0);
                }
            }
        }
    }
    float s = 0.f;
    for (int i = 0; i < 16; ++i) s += x0[i] + x1[i] + x2[i] + x3[i];
    for (int i = 0; i < 4; ++i) s += y0[i] + y1[i] + y2[i] + y3[i];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// ---------------------------------------------------------------- 2. MFMA + VALU
// per iteration: NM 32x32x16 f16 MFMAs on two accumulators and NV VALU ops on
// eight independent registers; VK 0 fp32 FMA, 1 packed fp16 FMA, 2 v_and_or_b32
template <int NM, int NV, int VK>
__global__ void k_mix(float* out, int iters)
{
    const int lane = threadIdx.x & 63;
    half8 a, b;
    for (int i = 0; i < 8; ++i) {
        a[i] = (_Float16)(0.001f * (lane + i));
        b[i] = (_Float16)(0.002f * (lane - i));
    }
    floatx16 acc0 = {}, acc1 = {};
    float x[8];
    half2v h[8];
    uint32_t u[8];
    for (int i = 0; i < 8; ++i) {
        x[i] = lane * 0.1f + i;
        h[i] = (half2v){(_Float16)(0.01f * i), (_Float16)0.5f};
        u[i] = lane * 77u + i;
    }
    const half2v hm = {(_Float16)0.999f, (_Float16)0.999f}, ha = {(_Float16)0.001f, (_Float16)0.001f};
    uint32_t m1 = 0x000F000Fu, m2 = 0x64006400u;
    asm volatile("" : "+v"(m1), "+v"(m2));
    auto valu = [&](int v) {
        if constexpr (VK == 0) x[v & 7] = __builtin_fmaf(x[v & 7], 1.0001f, 0.5f);
        else if constexpr (VK == 1) h[v & 7] = __builtin_elementwise_fma(h[v & 7], hm, ha);
        else {
            uint32_t r;
            asm volatile("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(u[v & 7]), "v"(m1), "v"(m2));
            u[v & 7] = r;
        }
    };
    constexpr int PER = NM ? NV / NM : 0;           // VALU ops after each MFMA
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            if (m & 1) acc1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc1, 0, 0, 0);
            else acc0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc0, 0, 0, 0);
#pragma unroll
            for (int v = 0; v < PER; ++v) valu(m * PER + v);
        }
        if constexpr (NM == 0) {
#pragma unroll
            for (int v = 0; v < NV; ++v) valu(v);
        }
    }
    float s = 0.f;
    for (int i = 0; i < 16; ++i) s += acc0[i] + acc1[i];
    for (int i = 0; i < 8; ++i) s += x[i] + (float)h[i][0] + (float)(u[i] & 1u);
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

static float time_ms(void (*launch)(float*, int, int, hipStream_t), float* out, int iters, int wps, hipStream_t st)
{
    hipEvent_t e0, e1;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));
    launch(out, 16, wps, st);                      // warm-up
    CK(hipEventRecord(e0, st));
    launch(out, iters, wps, st);
    CK(hipEventRecord(e1, st));
    CK(hipEventSynchronize(e1));
    float ms = 0.f;
    CK(hipEventElapsedTime(&ms, e0, e1));
    CK(hipEventDestroy(e0));
    CK(hipEventDestroy(e1));
    return ms;
}

template <int KIND>
static void launch_rate(float* out, int iters, int wps, hipStream_t st)
{
    k_rate<KIND><<<CUS, 256 * wps, 0, st>>>(out, iters);
}

template <int NM, int NV, int VK>
static void launch_mix(float* out, int iters, int wps, hipStream_t st)
{
    k_mix<NM, NV, VK><<<CUS, 256 * wps, 0, st>>>(out, iters);
}

int main()
{
    float* out;
    CK(hipMalloc(&out, (size_t)CUS * 512 * sizeof(float)));
    hipStream_t st;
    CK(hipStreamCreate(&st));
    const char* names[] = {"32x32x16 f16", "32x32x16 bf16", "16x16x32 f16", "16x16x32 bf16"};
    void (*rates[])(float*, int, int, hipStream_t) = {launch_rate<0>, launch_rate<1>, launch_rate<2>, launch_rate<3>};
    printf("1. sustained MFMA rate, 4 independent accumulators per wave\n");
    for (int wps = 1; wps <= 2; ++wps)
        for (int k = 0; k < 4; ++k) {
            const int iters = 8192;
            const float ms = time_ms(rates[k], out, iters, wps, st);
            const double flop = 4.0 * 32768 * iters * (double)CUS * 4 * wps;
            printf("  %-14s %d wave(s)/SIMD: %6.0f TFLOP/s\n", names[k], wps, flop / (ms * 1e-3) * 1e-12);
        }
    struct Mix { const char* what; int nm, nv; void (*f)(float*, int, int, hipStream_t); };
    Mix mixes[] = {
        {"2 MFMA", 2, 0, launch_mix<2, 0, 0>},
        {"16 fp32 FMA", 0, 16, launch_mix<0, 16, 0>},
        {"16 packed fp16 FMA", 0, 16, launch_mix<0, 16, 1>},
        {"16 v_and_or_b32", 0, 16, launch_mix<0, 16, 2>},
        {"2 MFMA + 8 fp32 FMA", 2, 8, launch_mix<2, 8, 0>},
        {"2 MFMA + 16 fp32 FMA", 2, 16, launch_mix<2, 16, 0>},
        {"2 MFMA + 16 packed fp16 FMA", 2, 16, launch_mix<2, 16, 1>},
        {"2 MFMA + 16 v_and_or_b32", 2, 16, launch_mix<2, 16, 2>},
        {"2 MFMA + 32 packed fp16 FMA", 2, 32, launch_mix<2, 32, 1>},
    };
    printf("2. cycles per iteration per wave at the nominal 2.4 GHz (all waves of a SIMD share it)\n");
    for (int wps = 1; wps <= 2; ++wps)
        for (const Mix& m : mixes) {
            const int iters = 4096;
            const float ms = time_ms(m.f, out, iters, wps, st);
            printf("  %-30s %d wave(s)/SIMD: %6.1f\n", m.what, wps, ms * 1e-3 * 2.4e9 / iters / wps);
        }
    CK(hipFree(out));
    return 0;
}
