// kernels_q4.hip -- the drafter's weight-only quantized projections:
// C[M][N] (+)= A[M][K] Wq^T with A in fp16, RTN weights in groups of 128
// along K with one fp16 scale per (column, group) (Sec. 4.1), fp32
// accumulation.  Formats: int4 symmetric (the default), int4 asymmetric with
// a zero point per (column, group) (App. B.2) and int8 symmetric (the W8
// drafter of App. B.3).  Drafting runs one token per sequence, so M is the
// live batch (64 in the 8B-shaped workload) and the weights are streamed
// from HBM exactly once per m-tile of 64 rows.
//
// Packed int4 layout (written by the drafter refresh): for column block
// nb = n / 32 and group g = k / 128 of a [N][K] matrix, G = K / 128, lane
// l in 0..63 stands for column 32 nb + (l & 31) and k-half h = l >> 5.  For
// k-step s in 0..7 (16 k each) lane l owns the uint32 word with the 8 codes
// k = 128 g + 16 s + 8 h + e, e = 0..7; code e sits in the nibble at bit
// 4 (e / 2) + 16 (e % 2), stored as q + 8 (symmetric) or q (asymmetric).
// The word of (nb, g, l, s) is at index (((nb G + g) 2 + s / 4) 64 + l) 4 +
// s % 4, so each wave reads one group of its block with two fully contiguous
// 1 KB loads.  The int8 layout has two words per k-step: code e of k-step s
// is byte e % 4 of word j = 2 s + e / 4, stored as q + 128, at index
// (((nb G + g) 4 + j / 4) 64 + l) 4 + j % 4 (four 1 KB loads per group).
// Scale and zero point of column n, group g are at (nb G + g) 32 + n % 32.
//
// Those words are exactly lane l's B operand of v_mfma_f32_32x32x16_f16
// for k-step s (column l & 31, k 8 h .. 8 h + 7 of the step).
// Dequantization uses the fp16 pattern 0x6400 = 1024: OR-ing a nibble into
// mantissa bits 0..3 gives 1024 + c and into bits 4..7 gives 1024 + 16 c
// for the stored code c, so a subtract of 1024 + z (z = 8 symmetric, the
// group's zero point asymmetric), or a fused multiply by 1/16 and add of
// -(64 + z), leaves q - z exactly; an int8 code is placed in the low byte
// of an fp16 1024 by a byte permute and 1152 subtracted.  The group's
// partial product is scaled in fp32.
//
// Work-group: 8 waves = 4 column blocks (128 columns) x 2 k-halves.  Waves
// of k-half hh take the groups g0 + hh, g0 + hh + 2, ... of the split, so
// each iteration covers two groups; the halves are summed through LDS at the
// end.  Two waves per SIMD let one wave's dequantization overlap the other's
// MFMAs.  A (both groups of an iteration) is staged through LDS; the weights
// go from HBM straight into registers.  Loads of iteration i + D - 1 are
// issued while iteration i computes, through a ring of D register sets; the
// iteration count is padded to a multiple of D (padding iterations read a
// clamped group and scale its product by 0) so the unrolled loop body has no
// branches and the compiler's wait counts stay exact.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int QK = 128;             // k per group
constexpr int QLD = QK + 8;         // LDS row stride (fp16 elements)
constexpr int QSMAX = 32;           // most groups one split may cover (scales staged in LDS)
constexpr int QCOLS = 128;          // columns per work-group

__device__ __forceinline__ float h2f(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }

// (w & mask) | or_bits in one VALU op (the compiler splits it in two when
// both constants are literals)
__device__ __forceinline__ uint32_t and_or(uint32_t w, uint32_t mask, uint32_t or_bits)
{
    uint32_t r;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(w), "v"(mask), "v"(or_bits));
    return r;
}

// lane's B operand for one k-step from its packed int4 word; lo / hi are the
// nibble masks 0x000F000F / 0x00F000F0 and magic the fp16 pair 1024, 1024,
// passed in registers; sub = 1024 + z and mhi = -(64 + z) as fp16 pairs
__device__ __forceinline__ half8 dq_word(uint32_t w, uint32_t lo, uint32_t hi, uint32_t magic, half2v sub, half2v mhi)
{
    const half2v sixteenth = {(_Float16)0.0625f, (_Float16)0.0625f};
    const uint32_t w2 = w >> 8;
    const half2v p0 = __builtin_bit_cast(half2v, and_or(w, lo, magic)) - sub;
    const half2v p1 = __builtin_elementwise_fma(__builtin_bit_cast(half2v, and_or(w, hi, magic)), sixteenth, mhi);
    const half2v p2 = __builtin_bit_cast(half2v, and_or(w2, lo, magic)) - sub;
    const half2v p3 = __builtin_elementwise_fma(__builtin_bit_cast(half2v, and_or(w2, hi, magic)), sixteenth, mhi);
    return (half8){p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

// the same for the int8 format: codes 0..3 of w0, then of w1; magic holds
// 0x64 in every byte, so each permute builds the fp16 pair 1024 + c0, 1024 + c1
__device__ __forceinline__ half8 dq_bytes(uint32_t w0, uint32_t w1, uint32_t magic)
{
    const half2v sub = {(_Float16)1152.0f, (_Float16)1152.0f};
    const half2v p0 = __builtin_bit_cast(half2v, __builtin_amdgcn_perm(magic, w0, 0x04010400u)) - sub;
    const half2v p1 = __builtin_bit_cast(half2v, __builtin_amdgcn_perm(magic, w0, 0x04030402u)) - sub;
    const half2v p2 = __builtin_bit_cast(half2v, __builtin_amdgcn_perm(magic, w1, 0x04010400u)) - sub;
    const half2v p3 = __builtin_bit_cast(half2v, __builtin_amdgcn_perm(magic, w1, 0x04030402u)) - sub;
    return (half8){p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

// SW: the SwiGLU epilogue.  The weights are [2F][K], gate rows then up rows;
// tile t takes the gate column blocks 2t, 2t + 1 (waves cb = 0, 1) and the up
// blocks F/32 + 2t, F/32 + 2t + 1 of the same 64 features (cb = 2, 3), runs
// without split-K, and writes out[m][f] = SiLU(g) u (type out_t) instead of C.
template <int MT, int D, int FMT, bool SW>
__global__ void __launch_bounds__(512) k_gemm_q4(const uint16_t* __restrict__ A, const uint32_t* __restrict__ Wq,
                                                 const uint16_t* __restrict__ Sc, const uint8_t* __restrict__ Zp,
                                                 float* __restrict__ C,
                                                 float* __restrict__ P, int M, int N, int K, int ldc, int mode,
                                                 int S, int msup, int total, void* __restrict__ out, int out_t)
{
    constexpr int ROWS = 32 * MT;                      // rows of one m-tile
    constexpr int AP = ROWS * 2 * (QK / 8) / 512;      // 16-byte A pieces per thread per iteration
    constexpr int WPL = FMT == QF_W8 ? 4 : 2;          // 16-byte weight pieces per lane per group
    __shared__ __attribute__((aligned(16))) uint16_t As[2][2][ROWS * QLD];
    __shared__ __attribute__((aligned(16))) uint16_t Ss[4 * QSMAX * 32];
    __shared__ __attribute__((aligned(16))) uint8_t Zs[FMT == QF_W4A ? 4 * QSMAX * 32 : 16];

    const int per_xcd = gridDim.x >> 3;                // gridDim.x is a multiple of 8
    const int w = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (w >= total) return;
    const int ms = w % msup, rest = w / msup;
    const int s = rest % S, tile = rest / S;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: keeps per-wave math scalar
    const int cb = wv & 3, hh = wv >> 2;
    const int m0 = ms * ROWS;
    const int G = K / QK, Gs = G / S, g0 = s * Gs, g1 = g0 + Gs;
    const int rows = min(M - m0, ROWS);
    const int nblk = N / 32;
    // column block of wave slot c of this tile
    auto blk_of = [&](int c) { return SW ? (c < 2 ? tile * 2 + c : nblk / 2 + tile * 2 + c - 2) : tile * 4 + c; };
    const int nb = blk_of(cb);                         // this wave's column block (stores only if < nblk)
    const int nbl = min(nb, nblk - 1);                 // block it loads
    const int nit = (Gs + 1) >> 1;                     // iterations (groups per k-half)
    const int nend = (nit + D - 1) / D * D;

    // scales of the work-group's 4 blocks over the split: 4 runs of Gs*32
    // contiguous fp16, at most 512 16-byte pieces, one per thread; loaded
    // before the ring so that waiting for them does not wait for the ring
    const int sidx = min(tid, 16 * Gs - 1);
    const int sb = sidx / (Gs * 4), sr = sidx - sb * (Gs * 4);
    const u32x4 sv = *(const u32x4*)(Sc + ((size_t)min(blk_of(sb), nblk - 1) * G + g0) * 32 + sr * 8);
    // zero points (asymmetric format): 4 runs of Gs*32 bytes, one 16-byte piece per thread
    const int zidx = min(tid, 8 * Gs - 1);
    const int zb = zidx / (Gs * 2), zr = zidx - zb * (Gs * 2);
    u32x4 zv = {0u, 0u, 0u, 0u};
    if (FMT == QF_W4A) zv = *(const u32x4*)(Zp + ((size_t)min(blk_of(zb), nblk - 1) * G + g0) * 32 + zr * 16);

    // A pieces: p = tid + 512 t -> (half, row, 16-byte column)
    u32x4 ar[D][AP];
    auto load_a = [&](int it, u32x4 (&a)[AP]) {
#pragma unroll
        for (int t = 0; t < AP; ++t) {
            const int p = tid + 512 * t;
            const int half = p / (ROWS * 16), row = (p / 16) % ROWS, col = (p & 15) * 8;
            const int g = min(g0 + 2 * it + half, g1 - 1);
            a[t] = *(const u32x4*)(A + (size_t)(m0 + min(row, rows - 1)) * K + (size_t)g * QK + col);
        }
    };
    // rows past M hold copies of row M - 1 (their outputs are never stored)
    // and padding groups a clamped group (their scale is taken as 0)
    auto store_a = [&](int buf, const u32x4 (&a)[AP]) {
#pragma unroll
        for (int t = 0; t < AP; ++t) {
            const int p = tid + 512 * t;
            const int half = p / (ROWS * 16), row = (p / 16) % ROWS, col = (p & 15) * 8;
            *(u32x4*)&As[buf][half][row * QLD + col] = a[t];
        }
    };
    u32x4 wr[D][WPL];
    auto load_w = [&](int it, u32x4 (&q)[WPL]) {
        const int g = min(g0 + 2 * it + hh, g1 - 1);
        const u32x4* base = (const u32x4*)Wq + ((size_t)nbl * G + g) * (64 * WPL);
#pragma unroll
        for (int i = 0; i < WPL; ++i) q[i] = base[64 * i + lane];
    };

    floatx16 acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;

    uint32_t lo = 0x000F000Fu, hi = 0x00F000F0u, magic = FMT == QF_W8 ? 0x64646464u : 0x64006400u;
    asm volatile("" : "+v"(lo), "+v"(hi), "+v"(magic));   // keep the constants in VGPRs
    auto compute = [&](int buf, int it, const u32x4 (&q)[WPL]) {
        const uint16_t* ab = &As[buf][hh][(lane & 31) * QLD + 8 * (lane >> 5)];
        const int gi = 2 * it + hh;
        half2v sub = {(_Float16)1032.0f, (_Float16)1032.0f}, mhi = {(_Float16)-72.0f, (_Float16)-72.0f};
        if (FMT == QF_W4A) {
            const _Float16 z = (_Float16)(float)Zs[cb * QSMAX * 32 + min(gi, Gs - 1) * 32 + (lane & 31)];
            sub = (half2v){(_Float16)1024.0f + z, (_Float16)1024.0f + z};
            mhi = (half2v){(_Float16)-64.0f - z, (_Float16)-64.0f - z};
        }
        floatx16 tmp[MT];
#pragma unroll
        for (int st = 0; st < 8; ++st) {
            half8 b;
            if (FMT == QF_W8) b = dq_bytes(q[st >> 1][2 * (st & 1)], q[st >> 1][2 * (st & 1) + 1], magic);
            else b = dq_word(q[st >> 2][st & 3], lo, hi, magic, sub, mhi);
#pragma unroll
            for (int t = 0; t < MT; ++t) {
                const half8 a = *(const half8*)(ab + t * 32 * QLD + 16 * st);
                if (st == 0) {
                    floatx16 z;
#pragma unroll
                    for (int r = 0; r < 16; ++r) z[r] = 0.f;
                    tmp[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, z, 0, 0, 0);
                } else {
                    tmp[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, tmp[t], 0, 0, 0);
                }
            }
        }
        // a padding group (past the split) contributes nothing
        const float sv_ = h2f(Ss[cb * QSMAX * 32 + min(gi, Gs - 1) * 32 + (lane & 31)]);
        const float sc = gi < Gs ? sv_ : 0.f;
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[t][r] += sc * tmp[t][r];
    };

    // prologue: A and weights of the first D - 1 iterations in flight, A of iteration 0 in LDS
#pragma unroll
    for (int u = 0; u < D - 1; ++u) {
        load_a(min(u, nit - 1), ar[u]);
        load_w(min(u, nit - 1), wr[u]);
    }
    if (tid < 16 * Gs) *(u32x4*)&Ss[sb * QSMAX * 32 + sr * 8] = sv;
    if (FMT == QF_W4A && tid < 8 * Gs) *(u32x4*)&Zs[zb * QSMAX * 32 + zr * 16] = zv;
    store_a(0, ar[0]);
    lds_barrier();

    // iteration it uses ring slot it % D and LDS buffer it & 1; it requests
    // iteration it + D - 1 and stages the A tiles of it + 1
    for (int ib = 0; ib < nend; ib += D) {
#pragma unroll
        for (int u = 0; u < D; ++u) {
            const int it = ib + u;
            const int buf = it & 1;
            const int nx = (u + D - 1) % D;
            load_a(min(it + D - 1, nit - 1), ar[nx]);
            load_w(min(it + D - 1, nit - 1), wr[nx]);
            // keep the loads at the top of the iteration and this iteration's
            // math inside it (the scheduler otherwise sinks the loads and
            // hoists later dequantization, which shortens the prefetch)
            __builtin_amdgcn_sched_barrier(0);
            compute(buf, it, wr[u]);
            __builtin_amdgcn_sched_barrier(0);
            store_a(buf ^ 1, ar[(u + 1) % D]);
            lds_barrier();
        }
    }

    // ---- k-half 1 hands its sums to k-half 0 through LDS (the A buffers are free)
    float* xs = (float*)&As[0][0][0];                  // [4 blocks][MT][16][64 lanes]
    if (hh == 1) {
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) xs[((cb * MT + t) * 16 + r) * 64 + lane] = acc[t][r];
    }
    lds_barrier();
    if constexpr (SW) {
        // the up blocks hand their sums to the gate blocks of the same features
        static_assert((4 + 2) * MT * 16 * 64 * 4 <= sizeof(As), "SwiGLU exchange does not fit the A buffers");
        float* ys = xs + 4 * MT * 16 * 64;             // [2 up blocks][MT][16][64 lanes]
        if (hh == 0) {
#pragma unroll
            for (int t = 0; t < MT; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    acc[t][r] += xs[((cb * MT + t) * 16 + r) * 64 + lane];
                    if (cb >= 2) ys[(((cb - 2) * MT + t) * 16 + r) * 64 + lane] = acc[t][r];
                }
        }
        lds_barrier();
        if (hh == 1 || cb >= 2) return;
        const int F = N / 2, feat = nb * 32 + (lane & 31);
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + t * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (row >= M) continue;
                const float g = acc[t][r], u = ys[((cb * MT + t) * 16 + r) * 64 + lane];
                const float v = g / (1.f + __expf(-g)) * u;
                const size_t oi = (size_t)row * F + feat;
                if (out_t == ACT_F16) store_act<_Float16>(out, oi, v);
                else if (out_t == ACT_BF16) store_act<uint16_t>(out, oi, v);
                else store_act<float>(out, oi, v);
            }
        return;
    }
    if (hh == 1 || nb >= nblk) return;
    const int col = nb * 32 + (lane & 31);
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float v = acc[t][r] + xs[((cb * MT + t) * 16 + r) * 64 + lane];
            const int row = m0 + t * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (row >= M) continue;
            if (S == 1) {
                float* cp = C + (size_t)row * ldc + col;
                *cp = mode == GEMM_ADD ? *cp + v : v;
            } else {
                P[((size_t)s * M + row) * N + col] = v;
            }
        }
}

// split count: the smallest divisor S of G with at most QSMAX groups per
// split that gives at least Q4_MIN_WGS work-groups (else the largest valid)
#ifndef Q4_MIN_WGS
#define Q4_MIN_WGS 192
#endif

int q4_plan(int M, int N, int K)
{
    const int G = K / QK, msup = (M + 63) / 64, tiles = (N / 32 + 3) / 4;
    int best = -1;
    for (int S = 1; S <= G; ++S) {
        if (G % S || G / S > QSMAX) continue;
        best = S;
        if (tiles * S * msup >= Q4_MIN_WGS) return S;
    }
    return best;
}

template <int MT, int FMT, bool SW>
void q4_launch_d(int D, dim3 grid, hipStream_t st, const uint16_t* A, const uint32_t* Wq, const uint16_t* Sc,
                 const uint8_t* Z, float* C, float* P, int M, int N, int K, int ldc, int mode, int S, int msup,
                 int total, void* out, int out_t)
{
    if (D == 2)
        k_gemm_q4<MT, 2, FMT, SW><<<grid, 512, 0, st>>>(A, Wq, Sc, Z, C, P, M, N, K, ldc, mode, S, msup, total, out, out_t);
    else if (D == 3)
        k_gemm_q4<MT, 3, FMT, SW><<<grid, 512, 0, st>>>(A, Wq, Sc, Z, C, P, M, N, K, ldc, mode, S, msup, total, out, out_t);
    else
        k_gemm_q4<MT, 4, FMT, SW><<<grid, 512, 0, st>>>(A, Wq, Sc, Z, C, P, M, N, K, ldc, mode, S, msup, total, out, out_t);
}

template <int MT, bool SW>
void q4_launch_f(int fmt, int D, dim3 grid, hipStream_t st, const uint16_t* A, const uint32_t* Wq, const uint16_t* Sc,
                 const uint8_t* Z, float* C, float* P, int M, int N, int K, int ldc, int mode, int S, int msup,
                 int total, void* out = nullptr, int out_t = 0)
{
    if (fmt == QF_W4A)
        q4_launch_d<MT, QF_W4A, SW>(D, grid, st, A, Wq, Sc, Z, C, P, M, N, K, ldc, mode, S, msup, total, out, out_t);
    else if (fmt == QF_W8)
        q4_launch_d<MT, QF_W8, SW>(D, grid, st, A, Wq, Sc, Z, C, P, M, N, K, ldc, mode, S, msup, total, out, out_t);
    else
        q4_launch_d<MT, QF_W4, SW>(D, grid, st, A, Wq, Sc, Z, C, P, M, N, K, ldc, mode, S, msup, total, out, out_t);
}

// ring depth (iterations in flight + 1), chosen so the padding to a multiple
// of D wastes no iteration where possible
int q4_ring_depth(int nit) { return nit % 4 == 0 ? 4 : (nit % 3 == 0 ? 3 : (nit >= 4 ? 4 : (nit == 3 ? 3 : 2))); }

}  // namespace

int gemm_q4_k_ok(int K) { return K % QK == 0 && q4_plan(64, QCOLS, K) > 0; }

size_t gemm_q4_part_floats(int M, int N, int K)
{
    const int S = q4_plan(M, N, K);
    return S > 1 ? (size_t)S * M * N : 0;
}

int launch_gemm_q4(const uint16_t* A, const uint32_t* Wq, const uint16_t* Sc, const uint8_t* Z, int fmt, float* C,
                   float* part, size_t part_cap, int M, int N, int K, int ldc, gemm_mode mode, hipStream_t st)
{
    if (K % QK || N % 32 || M < 1 || fmt < QF_W4 || fmt > QF_W8 || (fmt == QF_W4A && !Z)) return -1;
    const int S = q4_plan(M, N, K);
    if (S < 1 || (S > 1 && (size_t)S * M * N > part_cap)) return -1;
    const int G = K / QK, nit = (G / S + 1) / 2;
    const int D = q4_ring_depth(nit);
    const int msup = (M + 63) / 64;
    const int total = (N / 32 + 3) / 4 * S * msup;
    dim3 grid((total + 7) / 8 * 8);
    if (M <= 32) q4_launch_f<1, false>(fmt, D, grid, st, A, Wq, Sc, Z, C, part, M, N, K, ldc, mode, S, msup, total);
    else q4_launch_f<2, false>(fmt, D, grid, st, A, Wq, Sc, Z, C, part, M, N, K, ldc, mode, S, msup, total);
    return S;
}

int launch_gemm_q4_swiglu(const uint16_t* A, const uint32_t* Wq, const uint16_t* Sc, const uint8_t* Z, int fmt,
                          void* out, act_t out_t, int M, int F, int K, hipStream_t st)
{
    // one split: every group of K must fit the work-group's scale staging
    if (K % QK || F % 64 || K / QK > QSMAX || M < 1 || fmt < QF_W4 || fmt > QF_W8 || (fmt == QF_W4A && !Z)) return 0;
    const int G = K / QK, nit = (G + 1) / 2;
    const int D = q4_ring_depth(nit);
    const int msup = (M + 63) / 64;
    const int total = F / 64 * msup;
    dim3 grid((total + 7) / 8 * 8);
    if (M <= 32)
        q4_launch_f<1, true>(fmt, D, grid, st, A, Wq, Sc, Z, nullptr, nullptr, M, 2 * F, K, 0, 0, 1, msup, total, out,
                             (int)out_t);
    else
        q4_launch_f<2, true>(fmt, D, grid, st, A, Wq, Sc, Z, nullptr, nullptr, M, 2 * F, K, 0, 0, 1, msup, total, out,
                             (int)out_t);
    return 1;
}
