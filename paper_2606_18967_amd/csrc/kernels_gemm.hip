// kernels_gemm.hip -- the bf16 projections: C[M][N] (fp32) = or += A[M][K] W^T.
//
// Weights are row-major [N][K] (K contiguous), activations [M][K].
//   - gemm_dma64 (M <= 64, N a multiple of 256): 64-row tiles with both
//     operands brought into LDS by DMA through a three-stage ring; see
//     k_gemm_dma64.  gemm_stream (M <= 64, other N): weights streamed from
//     HBM into registers, v_mfma_f32_16x16x32_bf16; see k_gemm_stream.
//   - gemm_tiled (M > 64, the verify forward): both operands through LDS.
//   - gemm_f32 / gemm_q4_f32: plain VALU versions for fp32 models (the int4
//     one reads the packed layout of kernels_q4.hip).
#include "common.h"
#include "kernels.h"

namespace {

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
        lds_barrier();
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
        lds_barrier();
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

__device__ __forceinline__ float f16_bits_to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }

// ------------------------------------------------------------------ weight-streaming bf16 MFMA GEMM
// C[M][N] = A[M][K] W^T for decode-shaped M (up to 64 rows per m-tile; the
// AR step and the draft LM head).  A work-group covers a 64-row m-tile,
// 64*NBW columns (NBW 16-column blocks per wave, 4 waves) and a range of K
// split into chunks of 128.  The A chunk is staged in LDS (double-buffered)
// and shared by the four waves; each wave streams its weight columns from
// HBM straight into registers through a ring of RD register sets (RD - 1
// chunks in flight), so every weight byte is read once per m-tile.  Lane l
// covers k = 128g + 32j + 8(l/16) + 0..7 of chunk g in k-step j
// (v_mfma_f32_16x16x32_bf16): each load instruction reads 64 contiguous
// bytes of 16 weight rows; A is read from LDS in the same k order.  With several K splits
// the partial sums go to P[s][M][N] for the consumer (or k_splitk_reduce).
// Work items are laid out so that consecutive ones (the m-tiles of one
// column tile) land on the same XCD and share its L2.
constexpr int SK = 128;          // k per chunk
constexpr int ALD = SK + 8;      // LDS row stride in 2-byte elements
constexpr int SM = 64;           // rows per m-tile

template <int NBW, int MT, int NW>
__global__ void __launch_bounds__(64 * NW) k_gemm_stream(const uint16_t* __restrict__ A, const uint16_t* __restrict__ Wt,
                                                     float* __restrict__ C, float* __restrict__ P, int M, int N, int K,
                                                     int ldc, int mode, int S, int msup, int total)
{
    constexpr int RD = NW == 8 ? 4 : 3;   // register sets in the load ring (deeper where the registers allow)
    __shared__ __attribute__((aligned(16))) uint16_t As[2][SM * ALD];
    const int per_xcd = gridDim.x >> 3;                     // gridDim.x is a multiple of 8
    const int w = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (w >= total) return;
    const int ms = w % msup, rest = w / msup;
    const int s = rest % S, tile = rest / S;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int m0 = ms * SM;
    const int G = K / SK, Gs = G / S, g0 = s * Gs, g1 = g0 + Gs;
    const int nb0 = (tile * NW + wv) * NBW;
    const int rows = min(M - m0, MT * 16);                  // rows staged (others stay zero)
    // each work item walks its chunks from a different starting offset: in
    // lockstep they would all read the same 256-byte column of the weight
    // rows at once and crowd a few HBM channels
    const int rot = (tile * 5 + s) % Gs;
    auto phys = [&](int g) { const int i = g - g0 + rot; return g0 + (i >= Gs ? i - Gs : i); };

    // A tiles travel through a ring of register sets too (same depth as the
    // weights): the tile of chunk c + 1 is requested RD - 2 chunks before it
    // is stored to LDS
    constexpr int AP = 1024 / (64 * NW);                  // 16-byte A pieces per thread per chunk
    u32x4 ar[RD][AP];
    auto load_a = [&](int g, u32x4 (&a)[AP]) {
#pragma unroll
        for (int t = 0; t < AP; ++t) {
            const int pidx = tid + t * 64 * NW;
            const int row = pidx >> 4, col = (pidx & 15) * 8;
            a[t] = *(const u32x4*)(A + (size_t)(m0 + min(row, rows - 1)) * K + (size_t)phys(g) * SK + col);
        }
    };
    // a tile of a chunk past the split (valid false) is stored as zeros, so
    // the padded iterations of the main loop add nothing
    auto store_a = [&](int buf, const u32x4 (&a)[AP], bool valid) {
#pragma unroll
        for (int t = 0; t < AP; ++t) {
            const int pidx = tid + t * 64 * NW;
            const int row = pidx >> 4, col = (pidx & 15) * 8;
            if (row < MT * 16)
                *(u32x4*)(&As[buf][row * ALD + col]) = (valid && row < rows) ? a[t] : (u32x4){0u, 0u, 0u, 0u};
        }
    };
    u32x4 wr[RD][NBW][4];
    auto load_w = [&](int g, u32x4 (&wq)[NBW][4]) {
#pragma unroll
        for (int i = 0; i < NBW; ++i) {
            const uint16_t* wp = Wt + (size_t)((nb0 + i) * 16 + (lane & 15)) * K + (size_t)phys(g) * SK + 8 * (lane >> 4);
#pragma unroll
            for (int j = 0; j < 4; ++j) wq[i][j] = *(const u32x4*)(wp + 32 * j);   // j, j + 1 share a 128-byte line: cached
        }
    };

    floatx4 acc[NBW][MT];
#pragma unroll
    for (int i = 0; i < NBW; ++i)
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[i][t] = (floatx4){0.f, 0.f, 0.f, 0.f};

    auto compute = [&](int buf, const u32x4 (&wq)[NBW][4]) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint16_t* ab = &As[buf][(lane & 15) * ALD + 32 * j + 8 * (lane >> 4)];
            u32x4 af[MT];
#pragma unroll
            for (int t = 0; t < MT; ++t) af[t] = *(const u32x4*)(ab + t * 16 * ALD);
#pragma unroll
            for (int i = 0; i < NBW; ++i) {
                const bf16x8 bb = __builtin_bit_cast(bf16x8, wq[i][j]);
#pragma unroll
                for (int t = 0; t < MT; ++t)
                    acc[i][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, af[t]), bb,
                                                                       acc[i][t], 0, 0, 0);
            }
        }
    };

    // prologue: A and weights of the first RD - 1 chunks in flight, A of chunk g0 in LDS
    // (chunk indices past the split are clamped: those loads are redundant but
    // unconditional, which keeps the compiler's wait counts exact)
#pragma unroll
    for (int u = 0; u < RD - 1; ++u) {
        load_a(min(g0 + u, g1 - 1), ar[u]);
        load_w(min(g0 + u, g1 - 1), wr[u]);
    }
    store_a(0, ar[0], true);
    lds_barrier();

    // chunk c uses ring slot u = (c - g0) % RD and LDS buffer (c - g0) & 1; it
    // requests chunk c + RD - 1 (A before weights, so waiting for an A tile
    // leaves the newer loads in flight) and stores the A tile of c + 1.  The
    // chunk count is rounded up to a multiple of RD so the unrolled body has
    // no branches: a conditional chunk would make the compiler's wait counts
    // conservative at the merge and drain the whole ring every chunk.
    const int gend = g0 + (Gs + RD - 1) / RD * RD;
    for (int gb = g0; gb < gend; gb += RD) {
#pragma unroll
        for (int u = 0; u < RD; ++u) {
            const int c = gb + u;
            const int buf = (gb - g0 + u) & 1;
            const int nx = (u + RD - 1) % RD;
            load_a(min(c + RD - 1, g1 - 1), ar[nx]);
            load_w(min(c + RD - 1, g1 - 1), wr[nx]);
            compute(buf, wr[u]);
            store_a(buf ^ 1, ar[(u + 1) % RD], c + 1 < g1);
            lds_barrier();
        }
    }

    // ---- epilogue
#pragma unroll
    for (int i = 0; i < NBW; ++i) {
        const int col = (nb0 + i) * 16 + (lane & 15);
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = m0 + t * 16 + (lane >> 4) * 4 + r;
                if (row >= M) continue;
                if (S == 1) {
                    float* cp = C + (size_t)row * ldc + col;
                    *cp = mode == GEMM_ADD ? *cp + acc[i][t][r] : acc[i][t][r];
                } else {
                    P[((size_t)s * M + row) * N + col] = acc[i][t][r];
                }
            }
    }
}

// ------------------------------------------------------------------ tiled bf16 MFMA GEMM (M > 64)
// C[M][N] = A[M][K] W^T with both operands staged through LDS.  Block tile
// (32*MTW) x 128, four waves in a 2 x 2 grid, each wave (16*MTW) x 64 =
// MTW x 4 MFMA tiles of v_mfma_f32_16x16x32_bf16.  K advances in stages of 64
// with double-buffered LDS and the global loads of stage k + 2 in flight while
// stage k is multiplied.  LDS rows are padded to 72 elements (bank-conflict
// free 16-byte fragment reads).  Split-K partials as in k_gemm_stream.
constexpr int TBK = 64, TLD = TBK + 8, TBN = 128;

template <int MTW>
__global__ void __launch_bounds__(256) k_gemm_tiled(const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
                                                    float* __restrict__ C, float* __restrict__ P, int M, int N, int K,
                                                    int ldc, int mode, int S, int mtiles, int total)
{
    constexpr int BM = 32 * MTW;
    constexpr int AP = MTW;      // 16-byte A pieces per thread per stage (BM*8/256)
    constexpr int WP = 4;        // 16-byte W pieces per thread per stage (128*8/256)
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * TLD];
    __shared__ __attribute__((aligned(16))) uint16_t Ws[2][TBN * TLD];
    const int per_xcd = gridDim.x >> 3;
    const int w = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (w >= total) return;
    const int mt = w % mtiles, rest = w / mtiles;
    const int s = rest % S, nt = rest / S;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1;
    const int m0 = mt * BM, n0 = nt * TBN;
    const int KS = K / TBK, Ks = KS / S, k0 = s * Ks, k1 = k0 + Ks;
    const int rows = min(M - m0, BM);

    u32x4 ra[2][AP], rw[2][WP];
    auto load = [&](int kb, u32x4 (&a)[AP], u32x4 (&b)[WP]) {
#pragma unroll
        for (int t = 0; t < AP; ++t) {
            const int pidx = tid + t * 256, row = pidx >> 3, col = (pidx & 7) * 8;
            a[t] = *(const u32x4*)(A + (size_t)(m0 + min(row, rows - 1)) * K + (size_t)kb * TBK + col);
        }
#pragma unroll
        for (int t = 0; t < WP; ++t) {
            const int pidx = tid + t * 256, row = pidx >> 3, col = (pidx & 7) * 8;
            b[t] = *(const u32x4*)(W + (size_t)(n0 + row) * K + (size_t)kb * TBK + col);
        }
    };
    auto store = [&](int buf, const u32x4 (&a)[AP], const u32x4 (&b)[WP]) {
#pragma unroll
        for (int t = 0; t < AP; ++t) {
            const int pidx = tid + t * 256, row = pidx >> 3, col = (pidx & 7) * 8;
            *(u32x4*)(&As[buf][row * TLD + col]) = row < rows ? a[t] : (u32x4){0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int t = 0; t < WP; ++t) {
            const int pidx = tid + t * 256, row = pidx >> 3, col = (pidx & 7) * 8;
            *(u32x4*)(&Ws[buf][row * TLD + col]) = b[t];
        }
    };

    floatx4 acc[MTW][4];
#pragma unroll
    for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = (floatx4){0.f, 0.f, 0.f, 0.f};

    load(k0, ra[0], rw[0]);
    if (k0 + 1 < k1) load(k0 + 1, ra[1], rw[1]);
    store(0, ra[0], rw[0]);
    lds_barrier();
    for (int kb = k0; kb < k1; kb += 2) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int k = kb + u;
            if (k < k1) {
                const int buf = (k - k0) & 1;
                if (k + 2 < k1) load(k + 2, ra[u], rw[u]);      // slot u is free: stage k is in LDS
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const int kk = ks * 32 + (lane >> 4) * 8;
                    u32x4 af[MTW], bw[4];
#pragma unroll
                    for (int i = 0; i < MTW; ++i)
                        af[i] = *(const u32x4*)(&As[buf][(wm * 16 * MTW + 16 * i + (lane & 15)) * TLD + kk]);
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        bw[j] = *(const u32x4*)(&Ws[buf][(wn * 64 + 16 * j + (lane & 15)) * TLD + kk]);
#pragma unroll
                    for (int i = 0; i < MTW; ++i)
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, af[i]),
                                                                               __builtin_bit_cast(bf16x8, bw[j]),
                                                                               acc[i][j], 0, 0, 0);
                }
                if (k + 1 < k1) store(buf ^ 1, ra[u ^ 1], rw[u ^ 1]);
                lds_barrier();
            }
        }
    }
#pragma unroll
    for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = n0 + wn * 64 + 16 * j + (lane & 15);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = m0 + wm * 16 * MTW + 16 * i + (lane >> 4) * 4 + r;
                if (row >= M) continue;
                if (S == 1) {
                    float* cp = C + (size_t)row * ldc + col;
                    *cp = mode == GEMM_ADD ? *cp + acc[i][j][r] : acc[i][j][r];
                } else {
                    P[((size_t)s * M + row) * N + col] = acc[i][j][r];
                }
            }
        }
}

// The same tiling on v_mfma_f32_32x32x16_bf16 (MTW even): each wave's
// (16 MTW) x 64 tile is MTW/2 x 2 blocks of 32 x 32; lane l reads row or
// column l % 32 and k 8 (l / 32) + 0..7 of each 16-k step.
// SW: the SwiGLU epilogue.  W is [2F][K], gate rows then up rows; column tile
// t loads gate rows 64t..64t+63 (waves wn = 0) and up rows F + 64t.. (wn = 1),
// runs without split-K and writes out[m][f] = SiLU(g) u (type out_t).
template <int MTW, bool SW>
__global__ void __launch_bounds__(256) k_gemm_t32(const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
                                                    float* __restrict__ C, float* __restrict__ P, int M, int N, int K,
                                                    int ldc, int mode, int S, int mtiles, int total,
                                                    void* __restrict__ out, int out_t)
{
    constexpr int BM = 32 * MTW;
    constexpr int AP = MTW;      // 16-byte A pieces per thread per stage (BM*8/256)
    constexpr int WP = 4;        // 16-byte W pieces per thread per stage (128*8/256)
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * TLD];
    __shared__ __attribute__((aligned(16))) uint16_t Ws[2][TBN * TLD];
    const int per_xcd = gridDim.x >> 3;
    const int w = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (w >= total) return;
    const int mt = w % mtiles, rest = w / mtiles;
    const int s = rest % S, nt = rest / S;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1;
    const int m0 = mt * BM, n0 = nt * TBN;
    const int KS = K / TBK, Ks = KS / S, k0 = s * Ks, k1 = k0 + Ks;
    const int rows = min(M - m0, BM);

    u32x4 ra[2][AP], rw[2][WP];
    auto load = [&](int kb, u32x4 (&a)[AP], u32x4 (&b)[WP]) {
#pragma unroll
        for (int t = 0; t < AP; ++t) {
            const int pidx = tid + t * 256, row = pidx >> 3, col = (pidx & 7) * 8;
            a[t] = *(const u32x4*)(A + (size_t)(m0 + min(row, rows - 1)) * K + (size_t)kb * TBK + col);
        }
#pragma unroll
        for (int t = 0; t < WP; ++t) {
            const int pidx = tid + t * 256, row = pidx >> 3, col = (pidx & 7) * 8;
            const int wrow = SW ? (row < 64 ? nt * 64 + row : N / 2 + nt * 64 + row - 64) : n0 + row;
            b[t] = *(const u32x4*)(W + (size_t)wrow * K + (size_t)kb * TBK + col);
        }
    };
    auto store = [&](int buf, const u32x4 (&a)[AP], const u32x4 (&b)[WP]) {
#pragma unroll
        for (int t = 0; t < AP; ++t) {
            const int pidx = tid + t * 256, row = pidx >> 3, col = (pidx & 7) * 8;
            *(u32x4*)(&As[buf][row * TLD + col]) = row < rows ? a[t] : (u32x4){0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int t = 0; t < WP; ++t) {
            const int pidx = tid + t * 256, row = pidx >> 3, col = (pidx & 7) * 8;
            *(u32x4*)(&Ws[buf][row * TLD + col]) = b[t];
        }
    };

    floatx16 acc[MTW / 2][2];
#pragma unroll
    for (int i = 0; i < MTW / 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    load(k0, ra[0], rw[0]);
    if (k0 + 1 < k1) load(k0 + 1, ra[1], rw[1]);
    store(0, ra[0], rw[0]);
    lds_barrier();
    for (int kb = k0; kb < k1; kb += 2) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int k = kb + u;
            if (k < k1) {
                const int buf = (k - k0) & 1;
                if (k + 2 < k1) load(k + 2, ra[u], rw[u]);      // slot u is free: stage k is in LDS
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const int kk = ks * 16 + (lane >> 5) * 8;
                    u32x4 af[MTW / 2], bw[2];
#pragma unroll
                    for (int i = 0; i < MTW / 2; ++i)
                        af[i] = *(const u32x4*)(&As[buf][(wm * 16 * MTW + 32 * i + (lane & 31)) * TLD + kk]);
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        bw[j] = *(const u32x4*)(&Ws[buf][(wn * 64 + 32 * j + (lane & 31)) * TLD + kk]);
#pragma unroll
                    for (int i = 0; i < MTW / 2; ++i)
#pragma unroll
                        for (int j = 0; j < 2; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[i]),
                                                                               __builtin_bit_cast(bf16x8, bw[j]),
                                                                               acc[i][j], 0, 0, 0);
                }
                if (k + 1 < k1) store(buf ^ 1, ra[u ^ 1], rw[u ^ 1]);
                lds_barrier();
            }
        }
    }
    if constexpr (SW) {
        // the up half hands its products to the gate half of the same features
        static_assert(2 * (MTW / 2) * 2 * 16 * 64 * 4 <= sizeof(As), "SwiGLU exchange does not fit the A buffers");
        float* ys = (float*)&As[0][0];                 // [wm][i][j][r][64 lanes]
        auto yi = [&](int i, int j, int r) { return (((wm * (MTW / 2) + i) * 2 + j) * 16 + r) * 64 + lane; };
        if (wn == 1) {
#pragma unroll
            for (int i = 0; i < MTW / 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) ys[yi(i, j, r)] = acc[i][j][r];
        }
        lds_barrier();
        if (wn == 1) return;
        const int F = N / 2;
#pragma unroll
        for (int i = 0; i < MTW / 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int feat = nt * 64 + 32 * j + (lane & 31);
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = m0 + wm * 16 * MTW + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                    if (row >= M) continue;
                    const float g = acc[i][j][r], u = ys[yi(i, j, r)];
                    const float v = g / (1.f + __expf(-g)) * u;
                    const size_t oi = (size_t)row * F + feat;
                    if (out_t == ACT_F16) store_act<_Float16>(out, oi, v);
                    else if (out_t == ACT_BF16) store_act<uint16_t>(out, oi, v);
                    else store_act<float>(out, oi, v);
                }
            }
        return;
    }
#pragma unroll
    for (int i = 0; i < MTW / 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int col = n0 + wn * 64 + 32 * j + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm * 16 * MTW + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (row >= M) continue;
                if (S == 1) {
                    float* cp = C + (size_t)row * ldc + col;
                    *cp = mode == GEMM_ADD ? *cp + acc[i][j][r] : acc[i][j][r];
                } else {
                    P[((size_t)s * M + row) * N + col] = acc[i][j][r];
                }
            }
        }
}

// ------------------------------------------------------------------ 320-row tiles fed by LDS DMA
// The 320-row tile of k_gemm_t32 (wave tile 160 x 64, v_mfma_f32_32x32x16_bf16,
// the same MFMA operands in the same k order, so the same fp32 sums) with the
// operands brought into LDS by global_load_lds_dwordx4: each instruction puts
// 64 lanes x 16 bytes straight into 1 KB of LDS, so no registers stage the
// tiles and the waves issue no LDS stores.  K advances in stages of 64 through
// two LDS buffers: stage k + 1 is requested right after the barrier that opens
// stage k.  A stage holds 128-byte rows (64 k) of the A and W tiles; the
// 16-byte chunk c of row r sits at position c ^ sw(r), sw(r) = (r ^ r / 8) % 8,
// which keeps the fragment reads (rows r..r+7 or r..r+15 at one chunk) free of
// bank conflicts; a DMA lane therefore fetches chunk pos ^ sw(r) of its row.
// WN = 2: 320 x 128 tiles, 4 waves; WN = 4: 320 x 256 tiles, 8 waves (half the
// activation re-reads per weight byte, for launches with a full wave of tiles).
// SW: the SwiGLU epilogue; the tile takes 32 WN features, and wave column
// wn's two 32-column blocks are the gate rows and the up rows of the same 32
// features, so SiLU(g) u is formed in registers (no split-K there).  With S
// K splits the partial sums go to P[s][M][N] as in k_gemm_t32.
constexpr int DBK = 64, DRB = DBK * 2;                  // k per stage, bytes per tile row

__device__ __forceinline__ void lds_dma16(const void* src, uint32_t lds_byte)
{
    asm volatile("global_load_lds_dwordx4 %0, off" : : "v"(src), "{m0}"(lds_byte) : "memory");
}

// the same for data read once (weights): non-temporal
__device__ __forceinline__ void lds_dma16_nt(const void* src, uint32_t lds_byte)
{
    asm volatile("global_load_lds_dwordx4 %0, off nt" : : "v"(src), "{m0}"(lds_byte) : "memory");
}

// s_waitcnt vmcnt(N) with the other counters left free (gfx9 field layout)
template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt field is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ int dma_sw(int r) { return (r ^ (r >> 3)) & 7; }

template <int WN, bool SW>
__global__ void __launch_bounds__(128 * WN) k_gemm_dma(const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
                                                       float* __restrict__ C, float* __restrict__ P, int M, int N, int K,
                                                       int ldc, int mode, int S, int mtiles, int total,
                                                       void* __restrict__ out, int out_t)
{
    constexpr int MTW = 10, BM = 32 * MTW, BN = 64 * WN, NWAVE = 2 * WN;
    constexpr int NA = BM / 8, NI = NA + BN / 8;               // 1 KB pieces (8 rows) per stage
    constexpr int STG = (BM + BN) * DRB;
    constexpr int CNT = NI / NWAVE;                            // pieces per wave per stage
    static_assert(NI % NWAVE == 0, "every wave issues the same number of pieces");
    constexpr int FT = 32 * WN;                                // features per tile of the SwiGLU form
    __shared__ __attribute__((aligned(1024))) uint8_t sm[2 * STG];
    const uint32_t sbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)sm;
    const int per_xcd = gridDim.x >> 3;
    const int w = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (w >= total) return;
    const int mt = w % mtiles, rest = w / mtiles;
    const int s = rest % S, nt = rest / S;
    const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wv / WN, wn = wv % WN;
    const int m0 = mt * BM, n0 = nt * BN;
    const int Ks = K / DBK / S, k0 = s * Ks;
    const int rows = min(M - m0, BM);

    // this lane's source row and chunk for each of its pieces
    const uint16_t* src[CNT];
    uint32_t dst[CNT];
#pragma unroll
    for (int q = 0; q < CNT; ++q) {
        const int t = wv + q * NWAVE, rl = lane >> 3, pos = lane & 7;
        if (t < NA) {
            const int row = 8 * t + rl;
            src[q] = A + (size_t)(m0 + min(row, rows - 1)) * K + (size_t)k0 * DBK + 8 * (pos ^ dma_sw(row));
            dst[q] = t * 1024;
        } else {
            const int row = 8 * (t - NA) + rl;
            int wrow = n0 + row;
            if constexpr (SW) {
                const int f = nt * FT + (row >> 6) * 32 + (row & 31);   // wave column row/64, block (row/32)%2
                wrow = ((row >> 5) & 1) ? N / 2 + f : f;
            }
            src[q] = W + (size_t)wrow * K + (size_t)k0 * DBK + 8 * (pos ^ dma_sw(row));
            dst[q] = BM * DRB + (t - NA) * 1024;
        }
    }
    auto issue = [&](int buf, int kb) {
#pragma unroll
        for (int q = 0; q < CNT; ++q) {
            if (wv + q * NWAVE < NA) lds_dma16(src[q] + (size_t)kb * DBK, sbase + buf * STG + dst[q]);
            else lds_dma16_nt(src[q] + (size_t)kb * DBK, sbase + buf * STG + dst[q]);
        }
    };

    floatx16 acc[MTW / 2][2];
#pragma unroll
    for (int i = 0; i < MTW / 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    issue(0, 0);
    for (int kb = 0; kb < Ks; ++kb) {
        wait_vmcnt<0>();                    // this wave's pieces of stage kb are in LDS
        lds_barrier();                      // everyone's are, and stage kb - 1 is no longer read
        if (kb + 1 < Ks) issue((kb + 1) & 1, kb + 1);
        const uint8_t* sa = sm + (kb & 1) * STG;
        const uint8_t* sw = sa + BM * DRB;
#pragma unroll
        for (int ks = 0; ks < DBK / 16; ++ks) {
            const int c = 2 * ks + (lane >> 5);
            u32x4 af[MTW / 2], bw[2];
#pragma unroll
            for (int i = 0; i < MTW / 2; ++i) {
                const int r = wm * 16 * MTW + 32 * i + (lane & 31);
                af[i] = *(const u32x4*)(sa + r * DRB + ((c ^ dma_sw(r)) << 4));
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int r = wn * 64 + 32 * j + (lane & 31);
                bw[j] = *(const u32x4*)(sw + r * DRB + ((c ^ dma_sw(r)) << 4));
            }
#pragma unroll
            for (int i = 0; i < MTW / 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[i]),
                                                                       __builtin_bit_cast(bf16x8, bw[j]), acc[i][j],
                                                                       0, 0, 0);
        }
    }
    if constexpr (SW) {
        const int F = N / 2, feat = nt * FT + wn * 32 + (lane & 31);
#pragma unroll
        for (int i = 0; i < MTW / 2; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm * 16 * MTW + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (row >= M) continue;
                const float g = acc[i][0][r], u = acc[i][1][r];
                const float v = g / (1.f + __expf(-g)) * u;
                const size_t oi = (size_t)row * F + feat;
                if (out_t == ACT_F16) store_act<_Float16>(out, oi, v);
                else if (out_t == ACT_BF16) store_act<uint16_t>(out, oi, v);
                else store_act<float>(out, oi, v);
            }
        return;
    }
#pragma unroll
    for (int i = 0; i < MTW / 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int col = n0 + wn * 64 + 32 * j + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm * 16 * MTW + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (row >= M) continue;
                if (S == 1) {
                    float* cp = C + (size_t)row * ldc + col;
                    *cp = mode == GEMM_ADD ? *cp + acc[i][j][r] : acc[i][j][r];
                } else {
                    P[((size_t)s * M + row) * N + col] = acc[i][j][r];
                }
            }
        }
}

// ------------------------------------------------------------------ 64-row tiles fed by LDS DMA
// The decode-shaped GEMM (M <= 64: the AR step's projections, the draft LM
// head) as a 64 x 256 tile of the DMA-fed kernel above: eight waves, each a
// 32 x 64 block of v_mfma_f32_32x32x16_bf16, operands brought into LDS by
// global_load_lds_dwordx4 in whole 128-byte lines.  At 64 rows the tile
// computes little per stage, so the ring is three stages deep (two in
// flight while one is multiplied; 120 KB of LDS).  Streaming the weights
// straight into registers in the MFMA layout (k_gemm_stream) reads 64 bytes
// from each of 16 rows 10 KB apart per instruction and reaches 2.3-4.3 TB/s
// at the 32B shape's projections; this tile reaches 3.7-6.0 TB/s (gate/up
// 137 -> 95 us, down 85 -> 49 us, LM head 368 -> 309 us at M = 64).  Rows past
// M repeat row M - 1 (never stored); split-K partials as in k_gemm_dma.  SW:
// the SwiGLU epilogue of k_gemm_dma (a tile of 128 features; wave column
// wn's two 32-column blocks are the gate and the up rows of the same 32
// features), used where the gate/up projection runs unsplit.
constexpr int D64R = 3;                                 // LDS ring stages

template <bool SW>
__global__ void __launch_bounds__(512) k_gemm_dma64(const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
                                                    float* __restrict__ C, float* __restrict__ P, int M, int N, int K,
                                                    int ldc, int mode, int S, int total, void* __restrict__ out,
                                                    int out_t)
{
    constexpr int BM = 64, BN = 256, NWAVE = 8, NB = D64R;
    constexpr int NA = BM / 8, NI = NA + BN / 8;            // 1 KB pieces (8 rows of 128 B) per stage
    constexpr int STG = (BM + BN) * DRB;
    constexpr int CNT = NI / NWAVE;
    static_assert(NI % NWAVE == 0 && NB == 3, "five pieces per wave, waits written for three stages");
    __shared__ __attribute__((aligned(1024))) uint8_t sm[NB * STG];
    const uint32_t sbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)sm;
    const int per_xcd = gridDim.x >> 3;                     // gridDim.x is a multiple of 8
    const int w = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (w >= total) return;
    const int s = w % S, nt = w / S;
    const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wv >> 2, wn = wv & 3;
    const int n0 = nt * BN;
    const int Ks = K / DBK / S, k0 = s * Ks;

    const uint16_t* src[CNT];
    uint32_t dst[CNT];
#pragma unroll
    for (int q = 0; q < CNT; ++q) {
        const int t = wv + q * NWAVE, rl = lane >> 3, pos = lane & 7;
        if (t < NA) {
            const int row = 8 * t + rl;
            src[q] = A + (size_t)min(row, M - 1) * K + (size_t)k0 * DBK + 8 * (pos ^ dma_sw(row));
            dst[q] = t * 1024;
        } else {
            const int row = 8 * (t - NA) + rl;
            int wrow = n0 + row;
            if constexpr (SW) {
                const int f = nt * (BN / 2) + (row >> 6) * 32 + (row & 31);   // wave column row/64, block (row/32)%2
                wrow = ((row >> 5) & 1) ? N / 2 + f : f;
            }
            src[q] = W + (size_t)wrow * K + (size_t)k0 * DBK + 8 * (pos ^ dma_sw(row));
            dst[q] = BM * DRB + (t - NA) * 1024;
        }
    }
    auto issue = [&](int buf, int kb) {
#pragma unroll
        for (int q = 0; q < CNT; ++q) {
            if (wv + q * NWAVE < NA) lds_dma16(src[q] + (size_t)kb * DBK, sbase + buf * STG + dst[q]);
            else lds_dma16_nt(src[q] + (size_t)kb * DBK, sbase + buf * STG + dst[q]);
        }
    };

    floatx16 acc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;

    issue(0, 0);
    if (Ks > 1) issue(1, 1);
    for (int kb = 0; kb < Ks; ++kb) {
        // this wave's pieces of stage kb are in once those of the (at most one) later stage are all that is outstanding
        if (kb + 1 < Ks) wait_vmcnt<CNT>();
        else wait_vmcnt<0>();
        lds_barrier();                      // everyone's are, and stage kb - 1 is no longer read
        if (kb + 2 < Ks) issue((kb + 2) % NB, kb + 2);
        const uint8_t* sa = sm + (kb % NB) * STG;
        const uint8_t* sw = sa + BM * DRB;
#pragma unroll
        for (int ks = 0; ks < DBK / 16; ++ks) {
            const int c = 2 * ks + (lane >> 5);
            const int ra = wm * 32 + (lane & 31);
            const u32x4 af = *(const u32x4*)(sa + ra * DRB + ((c ^ dma_sw(ra)) << 4));
            u32x4 bw[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int r = wn * 64 + 32 * j + (lane & 31);
                bw[j] = *(const u32x4*)(sw + r * DRB + ((c ^ dma_sw(r)) << 4));
            }
#pragma unroll
            for (int j = 0; j < 2; ++j)
                acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af),
                                                                 __builtin_bit_cast(bf16x8, bw[j]), acc[j], 0, 0, 0);
        }
    }
    if constexpr (SW) {
        const int F = N / 2, feat = nt * (BN / 2) + wn * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (row >= M) continue;
            const float g = acc[0][r], u = acc[1][r];
            const float v = g / (1.f + __expf(-g)) * u;
            const size_t oi = (size_t)row * F + feat;
            if (out_t == ACT_F16) store_act<_Float16>(out, oi, v);
            else if (out_t == ACT_BF16) store_act<uint16_t>(out, oi, v);
            else store_act<float>(out, oi, v);
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int col = n0 + wn * 64 + 32 * j + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (row >= M) continue;
            if (S == 1) {
                float* cp = C + (size_t)row * ldc + col;
                *cp = mode == GEMM_ADD ? *cp + acc[j][r] : acc[j][r];
            } else {
                P[((size_t)s * M + row) * N + col] = acc[j][r];
            }
        }
    }
}

// C[m][n] (+)= sum_s P[s][m][n]
__global__ void __launch_bounds__(256) k_splitk_reduce(const float* __restrict__ P, float* __restrict__ C, int M, int N,
                                                       int ldc, int S, int mode)
{
    size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
    size_t MN = (size_t)M * N;
    if (idx >= MN) return;
    const float v = add_splits(0.f, P, S, MN, idx);
    int row = (int)(idx / N), col = (int)(idx % N);
    float* cp = C + (size_t)row * ldc + col;
    *cp = mode == GEMM_ADD ? *cp + v : v;
}

// ------------------------------------------------------------------ int4 x fp32 VALU
// code of weight (n, k) in the packed layout of kernels_q4.hip
// the stored code of weight (n, k) in the packed layout of format fmt
// (kernels_q4.hip), before the zero point is taken off
__device__ __forceinline__ int q_stored(const uint32_t* Wq, int fmt, int G, int n, int k)
{
    const int nb = n >> 5, g = k >> 7, kk = k & 127;
    const int st = kk >> 4, h = (kk >> 3) & 1, e = kk & 7;
    const int l = (n & 31) + 32 * h;
    if (fmt == QF_W8) {
        const int j = 2 * st + (e >> 2);
        const uint32_t word = Wq[((((size_t)nb * G + g) * 4 + (j >> 2)) * 64 + l) * 4 + (j & 3)];
        return (int)((word >> (8 * (e & 3))) & 255u);
    }
    const uint32_t word = Wq[((((size_t)nb * G + g) * 2 + (st >> 2)) * 64 + l) * 4 + (st & 3)];
    return (int)((word >> (4 * (e >> 1) + 16 * (e & 1))) & 15u);
}

__global__ void __launch_bounds__(256) k_gemm_q4_f32(const float* __restrict__ A, const uint32_t* __restrict__ Wq,
                                                     const uint16_t* __restrict__ Sc, const uint8_t* __restrict__ Z,
                                                     int fmt, float* __restrict__ C, int M, int N, int K, int ldc,
                                                     int mode)
{
    int n = blockIdx.x * 64 + (threadIdx.x & 63);
    int m = blockIdx.y * 4 + (threadIdx.x >> 6);
    if (m >= M || n >= N) return;
    int G = K / 128;
    const float* ar = A + (size_t)m * K;
    float acc = 0.f;
    for (int g = 0; g < G; ++g) {
        const size_t si = ((size_t)(n >> 5) * G + g) * 32 + (n & 31);
        const int z = fmt == QF_W8 ? 128 : (fmt == QF_W4A ? (int)Z[si] : 8);
        float part = 0.f;
        for (int k = g * 128; k < g * 128 + 128; ++k) part += ar[k] * (float)(q_stored(Wq, fmt, G, n, k) - z);
        acc += f16_bits_to_f32(Sc[si]) * part;
    }
    float* cp = C + (size_t)m * ldc + n;
    *cp = mode == GEMM_ADD ? *cp + acc : acc;
}

}  // namespace

// Split-K is used until the launch has GEMM_SPLIT_TARGET work-groups, with at
// most GEMM_MAX_SPLIT splits and at least two chunks per split.
#ifndef GEMM_SPLIT_TARGET
#define GEMM_SPLIT_TARGET 256
#endif
#ifndef GEMM_MAX_SPLIT
#define GEMM_MAX_SPLIT 8
#endif

void gemm_plan(int M, int N, int K, int* nbw, int* S)
{
    *nbw = (N % 128 == 0) ? 2 : 1;
    int tiles = N / (64 * *nbw);
    int msup = (M + SM - 1) / SM;
    int G = K / SK;
    int s = 1;
    while (tiles * s * msup < GEMM_SPLIT_TARGET && G % (2 * s) == 0 && G / (2 * s) >= 2 && 2 * s <= GEMM_MAX_SPLIT)
        s *= 2;
    *S = s;
}

// bf16 GEMMs with more than 64 rows use the tiled kernel (N % 128 == 0).
static bool use_tiled(int M, int N, int K) { return M > 64 && N % TBN == 0 && K % TBK == 0; }

// Tile height of the LDS-tiled kernels, in units of 32 rows: the height with
// the fewest padded rows ceil(M / BM) BM, ties going to the taller tile, since
// every m-tile reads the whole weight matrix again.  Heights 320, 256, 192 and
// 128 rows are k_gemm_t32<10|8|6|4> (32x32x16 MFMAs), 160 rows k_gemm_tiled<5>
// (16x16x32).  At M = 320 (64 sequences, gamma = 4) one 320-row tile reads each
// weight tile once: -15% on the four projections of a layer against two 160-
// or three 128-row tiles.
static int tiled_mtw(int M)
{
    static const int cand[] = {10, 8, 6, 5, 4};
    int best = 4;
    long best_rows = -1;
    for (int m : cand) {
        const long rows = (long)((M + 32 * m - 1) / (32 * m)) * 32 * m;
        if (best_rows < 0 || rows < best_rows) best = m, best_rows = rows;
    }
    return best;
}

// The height every form of the tiled GEMM takes.  Past 320 rows the 320-row
// tiles fed by LDS DMA win even where they pad: fewer passes over the weights
// at a higher rate per pass (measured at N = 28672, K = 4096: 142 against
// 158 us at M = 330, 144 against 228 us at M = 448; 894 against 537 TFLOP/s
// at 8192^3).  Up to 320 rows the tightest height stays (at 96-256 rows the
// shorter tiles are faster).
static int gemm_mtw(int M) { return M > 320 ? 10 : tiled_mtw(M); }

#ifndef TILED_SPLIT_TARGET
#define TILED_SPLIT_TARGET 192
#endif

static void tiled_plan(int M, int N, int K, int* mtw, int* S)
{
    *mtw = gemm_mtw(M);
    int mtiles = (M + 32 * *mtw - 1) / (32 * *mtw);
    int tiles = N / TBN * mtiles;
    int KS = K / TBK;
    int s = 1;
    while (tiles * s < TILED_SPLIT_TARGET && KS % (2 * s) == 0 && KS / (2 * s) >= 4 && 2 * s <= GEMM_MAX_SPLIT) s *= 2;
    *S = s;
}

// 320-row tiles: without a K split where 320 x 256 tiles (eight waves, half
// the activation bytes per weight byte of 320 x 128) or else 320 x 128 tiles
// give DMA_SPLIT_TARGET work-groups; otherwise 320 x 256 tiles (where N
// allows) and the smallest split S of the K / 64 stages (at least two per
// split, at most DMA_MAX_SPLIT) that gives that many.  The register-staged
// tiles and the SwiGLU form take the same S, so every form sums the same
// products in the same order.
#ifndef DMA_SPLIT_TARGET
#define DMA_SPLIT_TARGET 192
#endif
#ifndef DMA_MAX_SPLIT
#define DMA_MAX_SPLIT 32
#endif

static void dma_plan(int M, int N, int K, int* wn, int* S)
{
    const int mtiles = (M + 319) / 320;
    *S = 1;
    if (N % 256 == 0 && N / 256 * mtiles >= DMA_SPLIT_TARGET) { *wn = 4; return; }
    if (N / 128 * mtiles >= DMA_SPLIT_TARGET) { *wn = 2; return; }
    *wn = N % 256 == 0 ? 4 : 2;
    const int tiles = N / (64 * *wn) * mtiles;
    const int KB = K / 64;
    for (int s = 1; s <= DMA_MAX_SPLIT && 2 * s <= KB; ++s) {
        if (KB % s) continue;
        *S = s;
        if (tiles * s >= DMA_SPLIT_TARGET) break;
    }
}

// the 64-row DMA tiles: N a multiple of 256, K of 64 (at least two stages)
static bool use_dma64(int M, int N, int K) { return M <= 64 && N % 256 == 0 && K % DBK == 0 && K >= 2 * DBK; }

#ifndef DMA64_SPLIT_TARGET
#define DMA64_SPLIT_TARGET 192
#endif

// split count of the 64-row tiles: the smallest divisor S of the K / 64
// stages (at least two stages per split, at most 32 splits) giving
// DMA64_SPLIT_TARGET work-groups, else the largest such S
static int dma64_split(int N, int K)
{
    const int tiles = N / 256, KB = K / DBK;
    int S = 1;
    for (int s = 1; s <= 32 && 2 * s <= KB; ++s) {
        if (KB % s) continue;
        S = s;
        if (tiles * s >= DMA64_SPLIT_TARGET) break;
    }
    return S;
}

size_t gemm_part_floats(int M, int N, int K)
{
    int nbw, S;
    gemm_plan(M, N, K, &nbw, &S);
    if (use_dma64(M, N, K)) {
        const int S64 = dma64_split(N, K);
        S = S64 > S ? S64 : S;
    }
    if (use_tiled(M, N, K)) {
        int mtw, St;
        tiled_plan(M, N, K, &mtw, &St);
        if (mtw == 10) {
            int wn;
            dma_plan(M, N, K, &wn, &St);
        }
        S = St > S ? St : S;
    }
    return S > 1 ? (size_t)S * M * N : 0;
}

template <int NBW, int NW>
static void stream_mt(int MT, dim3 grid, hipStream_t s, const uint16_t* A, const uint16_t* W, float* C, float* P, int M,
                      int N, int K, int ldc, int mode, int S, int msup, int total)
{
    constexpr int T = 64 * NW;
    switch (MT) {
        case 1: k_gemm_stream<NBW, 1, NW><<<grid, T, 0, s>>>(A, W, C, P, M, N, K, ldc, mode, S, msup, total); break;
        case 2: k_gemm_stream<NBW, 2, NW><<<grid, T, 0, s>>>(A, W, C, P, M, N, K, ldc, mode, S, msup, total); break;
        case 3: k_gemm_stream<NBW, 3, NW><<<grid, T, 0, s>>>(A, W, C, P, M, N, K, ldc, mode, S, msup, total); break;
        default: k_gemm_stream<NBW, 4, NW><<<grid, T, 0, s>>>(A, W, C, P, M, N, K, ldc, mode, S, msup, total); break;
    }
}

int launch_gemm_bf16(const uint16_t* A, const uint16_t* W, float* C, float* part, size_t part_cap, int M, int N, int K,
                     int ldc, gemm_mode mode, bool defer_reduce, hipStream_t s, bool lds_dma)
{
    if (use_tiled(M, N, K)) {
        int mtw, S, wn = 2;
        tiled_plan(M, N, K, &mtw, &S);
        if (mtw == 10) dma_plan(M, N, K, &wn, &S);
        if (S > 1 && (size_t)S * M * N > part_cap) S = 1;
        int mtiles = (M + 32 * mtw - 1) / (32 * mtw);
        if (lds_dma && mtw == 10) {
            // 320-row tiles: the DMA-fed kernel
            const int total = N / (64 * wn) * mtiles * S;
            dim3 grid((total + 7) / 8 * 8);
            if (wn == 4)
                k_gemm_dma<4, false><<<grid, 512, 0, s>>>(A, W, C, part, M, N, K, ldc, mode, S, mtiles, total, nullptr, 0);
            else
                k_gemm_dma<2, false><<<grid, 256, 0, s>>>(A, W, C, part, M, N, K, ldc, mode, S, mtiles, total, nullptr, 0);
            if (S > 1 && !defer_reduce) {
                size_t MN = (size_t)M * N;
                k_splitk_reduce<<<(unsigned)((MN + 255) / 256), 256, 0, s>>>(part, C, M, N, ldc, S, mode);
            }
            return S;
        }
        int total = N / TBN * mtiles * S;
        dim3 grid((total + 7) / 8 * 8);
        switch (mtw) {
            case 10: k_gemm_t32<10, false><<<grid, 256, 0, s>>>(A, W, C, part, M, N, K, ldc, mode, S, mtiles, total, nullptr, 0); break;
            case 8: k_gemm_t32<8, false><<<grid, 256, 0, s>>>(A, W, C, part, M, N, K, ldc, mode, S, mtiles, total, nullptr, 0); break;
            case 6: k_gemm_t32<6, false><<<grid, 256, 0, s>>>(A, W, C, part, M, N, K, ldc, mode, S, mtiles, total, nullptr, 0); break;
            case 5: k_gemm_tiled<5><<<grid, 256, 0, s>>>(A, W, C, part, M, N, K, ldc, mode, S, mtiles, total); break;
            default: k_gemm_t32<4, false><<<grid, 256, 0, s>>>(A, W, C, part, M, N, K, ldc, mode, S, mtiles, total, nullptr, 0); break;
        }
        if (S > 1 && !defer_reduce) {
            size_t MN = (size_t)M * N;
            k_splitk_reduce<<<(unsigned)((MN + 255) / 256), 256, 0, s>>>(part, C, M, N, ldc, S, mode);
        }
        return S;
    }
    if (use_dma64(M, N, K)) {
        int S = dma64_split(N, K);
        if (S > 1 && (size_t)S * M * N > part_cap) S = 1;   // workspace too small: no split
        const int total = N / 256 * S;
        k_gemm_dma64<false><<<dim3((total + 7) / 8 * 8), 512, 0, s>>>(A, W, C, part, M, N, K, ldc, mode, S, total,
                                                                       nullptr, 0);
        if (S > 1 && !defer_reduce) {
            size_t MN = (size_t)M * N;
            k_splitk_reduce<<<(unsigned)((MN + 255) / 256), 256, 0, s>>>(part, C, M, N, ldc, S, mode);
        }
        return S;
    }
    int nbw, S;
    gemm_plan(M, N, K, &nbw, &S);
    if (S > 1 && (size_t)S * M * N > part_cap) S = 1;   // workspace too small: no split
    int msup = (M + SM - 1) / SM;
    int MT = msup > 1 ? 4 : (M + 15) / 16;
    // 8-wave work-groups (twice the columns, one A tile for twice the waves)
    // when 4-wave ones would not all be resident at once (two per CU): the
    // draft LM head then runs in a single wave of work-groups
    const bool wide = nbw == 2 && N % 256 == 0 && (N / 128) * S * msup > 512;
    int tiles = N / (64 * nbw * (wide ? 2 : 1));
    int total = tiles * S * msup;
    dim3 grid((total + 7) / 8 * 8);
    if (wide) stream_mt<2, 8>(MT, grid, s, A, W, C, part, M, N, K, ldc, mode, S, msup, total);
    else if (nbw == 2) stream_mt<2, 4>(MT, grid, s, A, W, C, part, M, N, K, ldc, mode, S, msup, total);
    else stream_mt<1, 4>(MT, grid, s, A, W, C, part, M, N, K, ldc, mode, S, msup, total);
    if (S > 1 && !defer_reduce) {
        size_t MN = (size_t)M * N;
        k_splitk_reduce<<<(unsigned)((MN + 255) / 256), 256, 0, s>>>(part, C, M, N, ldc, S, mode);
    }
    return S;
}

int launch_gemm_bf16_swiglu(const uint16_t* A, const uint16_t* W, void* out, act_t out_t, int M, int F, int K,
                            hipStream_t s, bool lds_dma)
{
    if (use_dma64(M, 2 * F, K) && F % 128 == 0) {
        // 64-row tiles: fused only where the plain projection runs unsplit
        if (dma64_split(2 * F, K) != 1) return 0;
        const int total = F / 128;
        k_gemm_dma64<true><<<dim3((total + 7) / 8 * 8), 512, 0, s>>>(A, W, nullptr, nullptr, M, 2 * F, K, 0, 0, 1,
                                                                      total, out, (int)out_t);
        return 1;
    }
    if (!use_tiled(M, 2 * F, K) || F % 64) return 0;
    const int mtw = gemm_mtw(M);
    if (mtw == 5) return 0;                              // the 16x16x32 kernel has no SwiGLU epilogue
    const int mtiles = (M + 32 * mtw - 1) / (32 * mtw);
    const int total = F / 64 * mtiles;
    dim3 grid((total + 7) / 8 * 8);
    const int N = 2 * F;
    if (mtw == 10) {
        // fused only where the plain projection would run unsplit (the same
        // products summed in the same order either way)
        int wn, S;
        dma_plan(M, N, K, &wn, &S);
        if (S != 1) return 0;
        if (lds_dma) {
            const int tot = F / (32 * wn) * mtiles;
            dim3 g((tot + 7) / 8 * 8);
            if (wn == 4)
                k_gemm_dma<4, true><<<g, 512, 0, s>>>(A, W, nullptr, nullptr, M, N, K, 0, 0, 1, mtiles, tot, out, out_t);
            else
                k_gemm_dma<2, true><<<g, 256, 0, s>>>(A, W, nullptr, nullptr, M, N, K, 0, 0, 1, mtiles, tot, out, out_t);
            return 1;
        }
    }
    switch (mtw) {
        case 10: k_gemm_t32<10, true><<<grid, 256, 0, s>>>(A, W, nullptr, nullptr, M, N, K, 0, 0, 1, mtiles, total, out, out_t); break;
        case 8: k_gemm_t32<8, true><<<grid, 256, 0, s>>>(A, W, nullptr, nullptr, M, N, K, 0, 0, 1, mtiles, total, out, out_t); break;
        case 6: k_gemm_t32<6, true><<<grid, 256, 0, s>>>(A, W, nullptr, nullptr, M, N, K, 0, 0, 1, mtiles, total, out, out_t); break;
        default: k_gemm_t32<4, true><<<grid, 256, 0, s>>>(A, W, nullptr, nullptr, M, N, K, 0, 0, 1, mtiles, total, out, out_t); break;
    }
    return 1;
}

void launch_gemm_f32(const float* A, const float* W, float* C, int M, int N, int K, int ldc, gemm_mode mode,
                     hipStream_t s)
{
    dim3 grid(N / FT, (M + FT - 1) / FT);
    k_gemm_f32<<<grid, 256, 0, s>>>(A, W, C, M, N, K, ldc, mode);
}

void launch_gemm_q4_f32(const float* A, const uint32_t* Wq, const uint16_t* Sc, const uint8_t* Z, int fmt, float* C,
                        int M, int N, int K, int ldc, gemm_mode mode, hipStream_t s)
{
    dim3 grid((N + 63) / 64, (M + 3) / 4);
    k_gemm_q4_f32<<<grid, 256, 0, s>>>(A, Wq, Sc, Z, fmt, C, M, N, K, ldc, mode);
}
