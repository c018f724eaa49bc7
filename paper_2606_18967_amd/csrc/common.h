// common.h -- shared device helpers for the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define WAVE 64

// ------------------------------------------------------------ bf16 storage
// bf16 values are stored as raw uint16_t bit patterns.
struct bf16_t { uint16_t x; };

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
typedef float float2v __attribute__((ext_vector_type(2)));

// round to nearest even (v_cvt_pk_bf16_f32); NaN stays NaN
__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// one activation element in the GEMM input type (fp32, bf16 round-to-nearest-even, fp16)
template <typename T>
__device__ __forceinline__ void store_act(void* out, size_t idx, float v);
template <> __device__ __forceinline__ void store_act<float>(void* out, size_t idx, float v) { ((float*)out)[idx] = v; }
template <> __device__ __forceinline__ void store_act<uint16_t>(void* out, size_t idx, float v) { ((uint16_t*)out)[idx] = f32_to_bf16(v); }
template <> __device__ __forceinline__ void store_act<_Float16>(void* out, size_t idx, float v) { ((_Float16*)out)[idx] = (_Float16)v; }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((float2v){lo, hi}, bf16x2v));
}

// Element access for the two model dtypes.
template <typename T> struct elem;
template <> struct elem<float> {
    static __device__ __forceinline__ float load(const float* p, size_t i) { return p[i]; }
    static __device__ __forceinline__ void store(float* p, size_t i, float v) { p[i] = v; }
};
template <> struct elem<uint16_t> {
    static __device__ __forceinline__ float load(const uint16_t* p, size_t i) { return bf16_to_f32(p[i]); }
    static __device__ __forceinline__ void store(uint16_t* p, size_t i, float v) { p[i] = f32_to_bf16(v); }
};

// ------------------------------------------------------------ barriers
// Work-group barrier that orders LDS only.  __syncthreads() also fences
// global memory, which on this target waits for every outstanding global
// load (vmcnt counts loads and stores) and so drains a kernel's prefetch.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// ------------------------------------------------------------ reductions
__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}
__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, WAVE));
    return v;
}

// block-wide sum for blockDim.x a multiple of 64 (<= 1024); red has >= 16 floats
__device__ __forceinline__ float block_sum(float v, float* red)
{
    int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    v = wave_sum(v);
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    float t = 0.f;
    for (int i = 0; i < nw; ++i) t += red[i];
    return t;
}

// ------------------------------------------------------------ error flags
// Device-side error words: a kernel that meets an out-of-range index sets its
// word to 1 (plain vector store) and skips the work that would have gone out
// of bounds.  The host reads the words back in sd_sync.
enum : int {
    ERR_SLOT = 0,       // slot index outside [0, max_slots)
    ERR_TOKEN = 1,      // token id outside [0, vocab)
    ERR_CTX = 2,        // a position at or beyond max_ctx
    ERR_PAGE = 3,       // a block-table entry outside [0, n_pages) (paged KV)
    ERR_LEN = 4,        // a prefill length outside [0, row width]
    ERR_COUNT = 5
};
// v + P[0][idx] + P[1][idx] + ... + P[S - 1][idx] (split stride st floats),
// added in split order.  The loads of eight splits go out before their adds,
// so their memory round trips overlap; past the last split the loads repeat
// split S - 1 (in bounds, never added).
__device__ __forceinline__ float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
__device__ __forceinline__ float add_splits(float v, const float* P, int S, size_t st, size_t idx)
{
    for (int s0 = 0; s0 < S; s0 += 8) {
        float p[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) p[u] = P[(size_t)min(s0 + u, S - 1) * st + idx];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (s0 + u < S) v += p[u];
    }
    return v;
}
__device__ __forceinline__ float4 add_splits(float4 v, const float* P, int S, size_t st, size_t idx)
{
    for (int s0 = 0; s0 < S; s0 += 8) {
        float4 p[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) p[u] = *(const float4*)(P + (size_t)min(s0 + u, S - 1) * st + idx);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (s0 + u < S) v = add4(v, p[u]);
    }
    return v;
}

// two float4 columns (idx_a, idx_b) summed over S splits, the loads of both in the same batch
__device__ __forceinline__ void add_splits2(float4& va, float4& vb, const float* P, int S, size_t st, size_t idx_a,
                                            size_t idx_b)
{
    for (int s0 = 0; s0 < S; s0 += 8) {
        float4 pa[8], pb[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const size_t o = (size_t)min(s0 + u, S - 1) * st;
            pa[u] = *(const float4*)(P + o + idx_a);
            pb[u] = *(const float4*)(P + o + idx_b);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (s0 + u < S) {
                va = add4(va, pa[u]);
                vb = add4(vb, pb[u]);
            }
    }
}

__device__ __forceinline__ void flag_error(uint32_t* err, int kind) { ((volatile uint32_t*)err)[kind] = 1u; }
