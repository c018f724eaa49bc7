// kernels_q4.hip -- the drafter's weight-only quantized projections:
// C[M][N] (+)= A[M][K] Wq^T with A in fp16, RTN weights in groups of 128
// along K with one fp16 scale per (column, group) (Sec. 4.1), fp32
// accumulation.  Formats: int4 symmetric (the default), int4 asymmetric with
// a zero point per (column, group) (App. B.2) and int8 symmetric (the W8
// drafter of App. B.3).  Drafting runs one token per sequence, so M is the
// live batch (64 in the benchmark workloads) and each weight is streamed from
// HBM once per m-tile of 64 rows.
//
// Packed int4 layout (written by the drafter refresh): for column block
// nb = n / 32 and group g = k / 128 of a [N][K] matrix, G = K / 128, lane
// l in 0..63 stands for column 32 nb + (l & 31) and k-half h = l >> 5.  For
// k-step s in 0..7 (16 k each) lane l owns the uint32 word with the 8 codes
// k = 128 g + 16 s + 8 h + e, e = 0..7; code e sits in the nibble at bit
// 4 (e / 2) + 16 (e % 2), stored as q + 8 (symmetric) or q (asymmetric).
// The word of (nb, g, l, s) is at index (((nb G + g) 2 + s / 4) 64 + l) 4 +
// s % 4, so a wave reads one group of its block with two fully contiguous
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
// Work-group: 8 waves (two per SIMD), 256 columns: wave w owns column block
// 8 t + w of tile t and walks the K range of its split group by group.  The
// group's A tile (the m-tile's rows x 128 k, fp16) is brought into LDS by
// global_load_lds_dwordx4 (no registers, no LDS stores), one group per stage
// of a D-stage ring, and read back as MFMA A fragments; 16-byte chunk c of
// row r sits at position c ^ (r & 15), so the fragment reads (16 rows at one
// chunk per phase) are free of bank conflicts.  Each wave streams its own
// weights from HBM (non-temporal loads: each weight is read once) into a
// ring of D register sets.  Group g + D - 1 is
// requested right after the barrier that opens group g.  Inside a group the
// A fragments and dequantized weights of k-step s + 1 are formed while the
// MFMAs of step s run, and the previous group's sums are scaled into the
// accumulators while the first MFMAs of the next group run (two alternating
// sets of per-group sums).  The scales (and zero points) of the work-group's
// columns over its split are staged in LDS once, before the ring starts.
// Split-K partials go to P[s][M][N] for the consumer kernel to sum; the
// gate/up projection without a split can instead form SiLU(g) u in its
// epilogue (waves 0-3 hold the gate blocks, waves 4-7 the up blocks of the
// same 128 features, exchanged through LDS).
#include "common.h"
#include "kernels.h"

namespace {

constexpr int QK = 128;             // k per group
constexpr int QGSMAX = 40;          // most groups one split may cover (scales staged in LDS)
constexpr int QWAVES = 8;           // waves per work-group, one 32-column block each
constexpr int QCOLS = 32 * QWAVES;  // columns per work-group
constexpr int QRING = 4;            // groups in flight (stages of the A ring, register sets of the weight ring)

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


__device__ __forceinline__ void lds_dma16(const void* src, uint32_t lds_byte)
{
    asm volatile("global_load_lds_dwordx4 %0, off" : : "v"(src), "{m0}"(lds_byte) : "memory");
}

// s_waitcnt vmcnt(N); the DMA loads above are invisible to the compiler's
// own wait counting, so the kernel waits for its A stages itself
template <int N>
__device__ __forceinline__ void wait_vm()
{
    static_assert(N >= 0 && N < 64, "vmcnt field is 6 bits");
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// MT m-tiles of 32 rows; FMT drafter format; SW SwiGLU epilogue (S == 1)
template <int MT, int FMT, bool SW>
__global__ void __launch_bounds__(64 * QWAVES) k_gemm_q4(const uint16_t* __restrict__ A, const uint32_t* __restrict__ Wq,
                                                         const uint16_t* __restrict__ Sc, const uint8_t* __restrict__ Zp,
                                                         float* __restrict__ C, float* __restrict__ P, int M, int N,
                                                         int K, int ldc, int mode, int S, int msup, int total,
                                                         void* __restrict__ out, int out_t)
{
    constexpr int D = QRING;
    constexpr int ROWS = 32 * MT;
    constexpr int STG = ROWS * 2 * QK;                 // bytes of one A stage (one group)
    constexpr int NA = STG / 1024 / QWAVES;            // DMA instructions per wave per stage
    constexpr int WPL = FMT == QF_W8 ? 4 : 2;          // 16-byte weight pieces per lane per group
    static_assert(NA >= 1 && (D - 2) * (NA + WPL) < 64, "vmcnt range");
    static_assert(D % 2 == 0, "the per-group sums alternate between two sets");
    __shared__ __attribute__((aligned(1024))) uint8_t sa[D * STG];
    __shared__ __attribute__((aligned(16))) uint16_t ss[QWAVES * QGSMAX * 32];
    __shared__ __attribute__((aligned(16))) uint8_t zs[FMT == QF_W4A ? QWAVES * QGSMAX * 32 : 16];
    const uint32_t sbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)sa;

    const int per_xcd = gridDim.x >> 3;                // gridDim.x is a multiple of 8
    const int w = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (w >= total) return;
    const int ms = w % msup, rest = w / msup;
    const int s = rest % S, tile = rest / S;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: keeps per-wave math scalar
    const int m0 = ms * ROWS;
    const int G = K / QK, Gs = G / S, g0 = s * Gs;
    const int rows = min(M - m0, ROWS);
    const int nblk = N / 32;
    // column block of wave slot c: consecutive blocks, or (SwiGLU) the gate
    // blocks 4 t .. 4 t + 3 for c < 4 and the up blocks of the same features
    auto blk_of = [&](int c) { return SW ? (c < 4 ? tile * 4 + c : nblk / 2 + tile * 4 + c - 4) : tile * QWAVES + c; };
    const int nb = blk_of(wv);                         // stores only if < nblk
    const int nbl = min(nb, nblk - 1);                 // block it loads

    // scales (and zero points) of the work-group's blocks over the split:
    // block slot c's Gs * 32 entries at ss[c * Gs * 32 ..]
    for (int p = tid; p < QWAVES * Gs * 4; p += 64 * QWAVES) {
        const int c = p / (Gs * 4), r = p - c * (Gs * 4);
        *(u32x4*)&ss[c * Gs * 32 + r * 8] = *(const u32x4*)(Sc + ((size_t)min(blk_of(c), nblk - 1) * G + g0) * 32 + r * 8);
    }
    if (FMT == QF_W4A)
        for (int p = tid; p < QWAVES * Gs * 2; p += 64 * QWAVES) {
            const int c = p / (Gs * 2), r = p - c * (Gs * 2);
            *(u32x4*)&zs[c * Gs * 32 + r * 16] = *(const u32x4*)(Zp + ((size_t)min(blk_of(c), nblk - 1) * G + g0) * 32 + r * 16);
        }

    // this thread's A pieces: instruction q of the wave covers chunks
    // (wv NA + q) 64 + lane of the stage; rows past M repeat row M - 1 (their
    // outputs are never stored)
    const uint16_t* asrc[NA];
    uint32_t adst[NA];
#pragma unroll
    for (int q = 0; q < NA; ++q) {
        const int ch = (wv * NA + q) * 64 + lane;
        const int r = ch >> 4, pos = ch & 15;
        asrc[q] = A + (size_t)(m0 + min(r, rows - 1)) * K + (size_t)g0 * QK + (pos ^ (r & 15)) * 8;
        adst[q] = (wv * NA + q) * 1024;
    }
    const u32x4* wbase = (const u32x4*)Wq + ((size_t)nbl * G + g0) * (64 * WPL) + lane;

    // group gi of the split (clamped past its end: the ring runs a few
    // iterations further; their sums are scaled by 0)
    auto issue = [&](int gi, u32x4 (&wr)[WPL]) {
        const int g = min(gi, Gs - 1);
        const uint32_t stg = sbase + (gi % D) * STG;
#pragma unroll
        for (int q = 0; q < NA; ++q) lds_dma16(asrc[q] + (size_t)g * QK, stg + adst[q]);
#pragma unroll
        for (int i = 0; i < WPL; ++i) wr[i] = __builtin_nontemporal_load(wbase + (size_t)g * (64 * WPL) + 64 * i);
    };

    floatx16 acc[MT], tmp[2][MT];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) { acc[t][r] = 0.f; tmp[1][t][r] = 0.f; }

    u32x4 wr[D][WPL];
#pragma unroll
    for (int u = 0; u < D - 1; ++u) issue(u, wr[u]);

    uint32_t lo = 0x000F000Fu, hi = 0x00F000F0u, magic = FMT == QF_W8 ? 0x64646464u : 0x64006400u;
    asm volatile("" : "+v"(lo), "+v"(hi), "+v"(magic));   // keep the constants in VGPRs
    float scp = 0.f;                                   // scale of the previous group (0 before the first)
    const int nend = (Gs + D - 1) / D * D;
    for (int ib = 0; ib < nend; ib += D) {
#pragma unroll
        for (int u = 0; u < D; ++u) {
            const int gi = ib + u;
            const int cur = u & 1, prv = cur ^ 1;
            wait_vm<(D - 2) * (NA + WPL)>();            // this thread's pieces of group gi are in
            lds_barrier();                             // everyone's are, and stage gi - 1 is no longer read
            issue(gi + D - 1, wr[(u + D - 1) % D]);
            const uint8_t* stg = sa + (gi % D) * STG;
            const int gc = min(gi, Gs - 1);
            half2v sub = {(_Float16)1032.0f, (_Float16)1032.0f}, mhi = {(_Float16)-72.0f, (_Float16)-72.0f};
            if (FMT == QF_W4A) {
                const _Float16 z = (_Float16)(float)zs[wv * Gs * 32 + gc * 32 + (lane & 31)];
                sub = (half2v){(_Float16)1024.0f + z, (_Float16)1024.0f + z};
                mhi = (half2v){(_Float16)-64.0f - z, (_Float16)-64.0f - z};
            }
            auto lda = [&](int st, half8 (&af)[MT]) {
#pragma unroll
                for (int t = 0; t < MT; ++t) {
                    const int r = 32 * t + (lane & 31), c = 2 * st + (lane >> 5);
                    af[t] = *(const half8*)(stg + r * (2 * QK) + ((c ^ (r & 15)) << 4));
                }
            };
            auto dqb = [&](int st) {
                if (FMT == QF_W8) return dq_bytes(wr[u][st >> 1][2 * (st & 1)], wr[u][st >> 1][2 * (st & 1) + 1], magic);
                return dq_word(wr[u][st >> 2][st & 3], lo, hi, magic, sub, mhi);
            };
            half8 afc[MT], afn[MT], bqc, bqn;
            lda(0, afc);
            bqc = dqb(0);
#pragma unroll
            for (int st = 0; st < 8; ++st) {
                if (st < 7) { lda(st + 1, afn); bqn = dqb(st + 1); }
#pragma unroll
                for (int t = 0; t < MT; ++t) {
                    if (st == 0) {
                        floatx16 z;
#pragma unroll
                        for (int r = 0; r < 16; ++r) z[r] = 0.f;
                        tmp[cur][t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(afc[t], bqc, z, 0, 0, 0);
                    } else {
                        tmp[cur][t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(afc[t], bqc, tmp[cur][t], 0, 0, 0);
                    }
                }
                if (st == 0) {
                    // the previous group's sums, scaled, while this group's first MFMAs run
#pragma unroll
                    for (int t = 0; t < MT; ++t)
#pragma unroll
                        for (int r = 0; r < 16; ++r) acc[t][r] += scp * tmp[prv][t][r];
                }
#pragma unroll
                for (int t = 0; t < MT; ++t) afc[t] = afn[t];
                bqc = bqn;
            }
            const float sv = h2f(ss[wv * Gs * 32 + gc * 32 + (lane & 31)]);
            scp = gi < Gs ? sv : 0.f;
        }
    }
    {
        const int prv = (nend - 1) & 1;
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[t][r] += scp * tmp[prv][t][r];
    }
    wait_vm<0>();                                      // the ring's last (clamped) DMA pieces have landed
    if constexpr (SW) {
        // the up waves hand their sums to the gate waves of the same features
        static_assert(4 * MT * 16 * 64 * 4 <= D * STG, "SwiGLU exchange does not fit the A ring");
        float* xs = (float*)sa;                        // [4 up waves][MT][16][64 lanes]
        lds_barrier();                                 // every wave is done reading the A ring
        if (wv >= 4) {
#pragma unroll
            for (int t = 0; t < MT; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) xs[(((wv - 4) * MT + t) * 16 + r) * 64 + lane] = acc[t][r];
        }
        lds_barrier();
        if (wv >= 4 || nb >= nblk) return;
        const int F = N / 2, feat = nb * 32 + (lane & 31);
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + t * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (row >= M) continue;
                const float g = acc[t][r], u = xs[((wv * MT + t) * 16 + r) * 64 + lane];
                const float v = g / (1.f + __expf(-g)) * u;
                const size_t oi = (size_t)row * F + feat;
                if (out_t == ACT_F16) store_act<_Float16>(out, oi, v);
                else if (out_t == ACT_BF16) store_act<uint16_t>(out, oi, v);
                else store_act<float>(out, oi, v);
            }
        return;
    }
    if (nb >= nblk) return;
    const int col = nb * 32 + (lane & 31);
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = m0 + t * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (row >= M) continue;
            const float v = acc[t][r];
            if (S == 1) {
                float* cp = C + (size_t)row * ldc + col;
                *cp = mode == GEMM_ADD ? *cp + v : v;
            } else {
                P[((size_t)s * M + row) * N + col] = v;
            }
        }
}

// split count: the smallest divisor S of G with at most QGSMAX groups per
// split that gives at least Q4_MIN_WGS work-groups, else the largest such S
// up to 64 (partials stay at most 64 M N floats).  Half the CUs is enough:
// a split's partials are read back by the consumer kernel (a norm, RoPE, the
// SwiGLU), so fewer splits with more groups each give the shorter step (at
// the 32B shape and M = 64 the output and down projections take 8 splits
// instead of 16 and 12; measured 0.6-1.1% less time per SD step)
#ifndef Q4_MIN_WGS
#define Q4_MIN_WGS 128
#endif

int q4_plan(int M, int N, int K)
{
    const int G = K / QK, msup = (M + 63) / 64, tiles = (N / 32 + QWAVES - 1) / QWAVES;
    int best = -1;
    for (int S = 1; S <= G && S <= 64; ++S) {
        if (G % S || G / S > QGSMAX) continue;
        best = S;
        if (tiles * S * msup >= Q4_MIN_WGS) return S;
    }
    return best;
}

template <int MT, bool SW>
void q4_launch(int fmt, dim3 grid, hipStream_t st, const uint16_t* A, const uint32_t* Wq, const uint16_t* Sc,
               const uint8_t* Z, float* C, float* P, int M, int N, int K, int ldc, int mode, int S, int msup, int total,
               void* out = nullptr, int out_t = 0)
{
    const dim3 blk(64 * QWAVES);
    if (fmt == QF_W4A)
        k_gemm_q4<MT, QF_W4A, SW><<<grid, blk, 0, st>>>(A, Wq, Sc, Z, C, P, M, N, K, ldc, mode, S, msup, total, out, out_t);
    else if (fmt == QF_W8)
        k_gemm_q4<MT, QF_W8, SW><<<grid, blk, 0, st>>>(A, Wq, Sc, Z, C, P, M, N, K, ldc, mode, S, msup, total, out, out_t);
    else
        k_gemm_q4<MT, QF_W4, SW><<<grid, blk, 0, st>>>(A, Wq, Sc, Z, C, P, M, N, K, ldc, mode, S, msup, total, out, out_t);
}

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
    const int msup = (M + 63) / 64;
    const int total = (N / 32 + QWAVES - 1) / QWAVES * S * msup;
    dim3 grid((total + 7) / 8 * 8);
    if (M <= 32) q4_launch<1, false>(fmt, grid, st, A, Wq, Sc, Z, C, part, M, N, K, ldc, mode, S, msup, total);
    else q4_launch<2, false>(fmt, grid, st, A, Wq, Sc, Z, C, part, M, N, K, ldc, mode, S, msup, total);
    return S;
}

int launch_gemm_q4_swiglu(const uint16_t* A, const uint32_t* Wq, const uint16_t* Sc, const uint8_t* Z, int fmt,
                          void* out, act_t out_t, int M, int F, int K, hipStream_t st)
{
    // only where the plain projection would run without a split, so that the
    // fused and the separate forms sum the same products in the same order
    if (K % QK || F % 128 || M < 1 || fmt < QF_W4 || fmt > QF_W8 || (fmt == QF_W4A && !Z)) return 0;
    if (q4_plan(M, 2 * F, K) != 1) return 0;
    const int msup = (M + 63) / 64;
    const int total = F / 128 * msup;
    dim3 grid((total + 7) / 8 * 8);
    if (M <= 32)
        q4_launch<1, true>(fmt, grid, st, A, Wq, Sc, Z, nullptr, nullptr, M, 2 * F, K, 0, 0, 1, msup, total, out,
                           (int)out_t);
    else
        q4_launch<2, true>(fmt, grid, st, A, Wq, Sc, Z, nullptr, nullptr, M, 2 * F, K, 0, 0, 1, msup, total, out,
                           (int)out_t);
    return 1;
}
