// kernels_model.hip -- decoder glue kernels: embedding gather, RMSNorm,
// RoPE + KV-cache write, decode attention, SwiGLU, KV length bookkeeping.
//
// Row convention of every forward call: row r = b*n + i is token i of
// sequence b, at absolute position kv_len[slots[b]] + off + i.
#include <hip/hip_ext.h>
#include "common.h"
#include "kernels.h"

namespace {

// physical page holding logical page lp of a slot's positions, or -1 when the
// block table has no valid page there (kv_geom, kernels.h)
__device__ __forceinline__ long long kv_page(const kv_geom& g, int slot, int lp)
{
    if (!g.bt) return slot;
    if (lp < 0 || lp >= g.mpp) return -1;
    const int pg = g.bt[(size_t)slot * g.mpp + lp];
    return pg >= 0 && pg < g.n_pages ? pg : -1;
}


typedef short v4s __attribute__((ext_vector_type(4)));
typedef short v8s __attribute__((ext_vector_type(8)));

__device__ __forceinline__ bool row_geom(const rows_t& r, int row, int* b, int* i, int* slot, int* pos)
{
    *b = row / r.n;
    *i = row - *b * r.n;
    *slot = r.slots[*b];
    if (*slot < 0 || *slot >= r.max_slots) return false;
    *pos = r.kv_len[*slot] + r.off + *i;
    return *pos >= 0 && *pos < r.max_ctx;
}


// four consecutive outputs (idx % 4 == 0) in one store
template <typename T>
__device__ __forceinline__ void store_act4(void* out, size_t idx, float4 v);
template <> __device__ __forceinline__ void store_act4<float>(void* out, size_t idx, float4 v) { *(float4*)((float*)out + idx) = v; }
template <> __device__ __forceinline__ void store_act4<uint16_t>(void* out, size_t idx, float4 v)
{
    *(uint2*)((uint16_t*)out + idx) = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
}
template <> __device__ __forceinline__ void store_act4<_Float16>(void* out, size_t idx, float4 v)
{
    const half2v a = {(_Float16)v.x, (_Float16)v.y}, b = {(_Float16)v.z, (_Float16)v.w};
    *(uint2*)((_Float16*)out + idx) = make_uint2(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b));
}

// ------------------------------------------------------------------ embed + rmsnorm
// Inputs that come out of a split-K projection are read as the sum of the
// partial products P[s][row][col] (s < S, S > 1); with S <= 1 the producer
// wrote its output directly.

// four consecutive elements of a weight row as floats (H % 4 == 0)
template <typename T> __device__ __forceinline__ float4 load4(const T* p);
template <> __device__ __forceinline__ float4 load4<float>(const float* p) { return *(const float4*)p; }
template <> __device__ __forceinline__ float4 load4<uint16_t>(const uint16_t* p)
{
    const uint2 v = *(const uint2*)p;
    return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u), __uint_as_float(v.y << 16),
                       __uint_as_float(v.y & 0xffff0000u));
}

// h[row] = E[token(row)];  out[row] = RMSNorm(h[row]) * gain
template <typename T, typename O>
__global__ void __launch_bounds__(1024) k_embed_rmsnorm(rows_t r, const int32_t* tokA, int sA, const int32_t* tokB,
                                                        int sB, const T* E, int H, int V, float* h, const T* gain,
                                                        float eps, void* out)
{
    __shared__ float red[16];
    const int row = blockIdx.x;
    const int b = row / r.n, i = row - b * r.n;
    const bool pad = r.lim && i >= r.lim[b];            // a padding row: embedded as token 0, never cached
    const int tok = pad ? 0 : (i == 0) ? tokA[(size_t)b * sA] : tokB[(size_t)b * sB + i - 1];
    const bool ok = tok >= 0 && tok < V;
    if (!ok && threadIdx.x == 0) flag_error(r.err, ERR_TOKEN);
    const T* er = E + (size_t)(ok ? tok : 0) * H;
    float* hr = h + (size_t)row * H;
    float ss = 0.f;
    for (int k4 = threadIdx.x * 4; k4 < H; k4 += blockDim.x * 4) {
        float4 x = load4<T>(er + k4);
        if (!ok) x = make_float4(0.f, 0.f, 0.f, 0.f);
        *(float4*)(hr + k4) = x;
        ss += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
    }
    ss = block_sum(ss, red);
    const float inv = rsqrtf(ss / (float)H + eps);
    for (int k4 = threadIdx.x * 4; k4 < H; k4 += blockDim.x * 4) {
        const float4 x = *(const float4*)(hr + k4);
        const float4 g = load4<T>(gain + k4);
        store_act4<O>(out, (size_t)row * H + k4, make_float4(x.x * inv * g.x, x.y * inv * g.y, x.z * inv * g.z, x.w * inv * g.w));
    }
}

// h[row] += sum_s P[s][row] (S > 1);  out[row] = RMSNorm(h[row]) * gain.
// Thread t holds the float4s t + j blockDim (j < NPT) of its row in registers:
// the residual, the split-K partials and the gain are all requested before any
// store, so a row costs one memory round trip and the block sum (a short row
// batch runs on few CUs and is bound by that latency, not by its bytes).
template <typename G, typename O, int NPT>
__global__ void __launch_bounds__(1024) k_add_rmsnorm(float* h, const float* P, int S, int R, int H, const G* gain,
                                                     float eps, void* out)
{
    __shared__ float red[16];
    const int row = blockIdx.x;
    float* hr = h + (size_t)row * H;
    const size_t RH = (size_t)R * H;
    // a thread's float4s past the row end read the last one (in bounds) and are dropped
    int kc[NPT];
    float4 x[NPT], g[NPT];
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
        kc[j] = min((int)(threadIdx.x + j * blockDim.x) * 4, H - 4);
        x[j] = *(const float4*)(hr + kc[j]);
        g[j] = load4<G>(gain + kc[j]);
    }
    // the partials of all NPT float4s in batches of SB splits, each batch's
    // loads together (a select, not a branch, drops the clamped repeats past
    // S, so that no load is deferred into a branch of its own)
    constexpr int SB = NPT <= 2 ? 8 : 16 / NPT;
    const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = 0; S > 1 && s0 < S; s0 += SB) {
        float4 p[NPT][SB];
#pragma unroll
        for (int j = 0; j < NPT; ++j)
#pragma unroll
            for (int u = 0; u < SB; ++u)
                p[j][u] = *(const float4*)(P + (size_t)min(s0 + u, S - 1) * RH + (size_t)row * H + kc[j]);
#pragma unroll
        for (int j = 0; j < NPT; ++j)
#pragma unroll
            for (int u = 0; u < SB; ++u) x[j] = add4(x[j], s0 + u < S ? p[j][u] : z4);
    }
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
        const int k4 = (threadIdx.x + j * blockDim.x) * 4;
        if (k4 < H) {
            if (S > 1) *(float4*)(hr + k4) = x[j];
            ss += x[j].x * x[j].x + x[j].y * x[j].y + x[j].z * x[j].z + x[j].w * x[j].w;
        }
    }
    ss = block_sum(ss, red);
    const float inv = rsqrtf(ss / (float)H + eps);
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
        const int k4 = (threadIdx.x + j * blockDim.x) * 4;
        if (k4 < H)
            store_act4<O>(out, (size_t)row * H + k4,
                          make_float4(x[j].x * inv * g[j].x, x[j].y * inv * g[j].y, x[j].z * inv * g[j].z,
                                      x[j].w * inv * g[j].w));
    }
}

__device__ __forceinline__ float sum_parts(const float* src, const float* P, int S, size_t RN, size_t idx)
{
    if (S <= 1) return src[idx];
    return add_splits(0.f, P, S, RN, idx);
}

// rotate-half RoPE of the column pair (a, c) = (x_k, x_{k + d/2}) with (cos, sin) = cs
__device__ __forceinline__ float2 rope_rot(float a, float c, float2 cs)
{
    return make_float2(a * cs.x - c * cs.y, a * cs.y + c * cs.x);
}

// element offset of (layer, KV head) inside a cache page (kv_geom)
__device__ __forceinline__ long long hbase_of(const kv_geom& g, int layer, int kvh)
{
    return (long long)layer * g.LS + (long long)kvh * g.HS;
}

// ------------------------------------------------------------------ rope + kv write
// qkv row = [q (n_q*d) | k (n_kv*d) | v (n_kv*d)], fp32: n_q + 2 n_kv head
// units of d columns.  RoPE rotate-half with the (cos, sin) table
// rope[pos][d/2].  q_out gets the rotated queries (fp32); the rotated keys and
// the values go to the cache at the row's position.  Work-group (row, group
// of upw head units); each thread takes one (unit, k) pair, columns k and
// k + d/2 of the unit.
template <typename T>
__global__ void __launch_bounds__(256) k_rope_kv(rows_t r, const float* qkv, const float* P, int S, const float2* rope,
                                                 int n_q, int n_kv, int d, T* kc, T* vc, kv_geom g, int layer,
                                                 float* q_out, int upw)
{
    const int row = blockIdx.x;
    int b, i, slot, pos;
    const bool ok = row_geom(r, row, &b, &i, &slot, &pos);
    const int hd = d / 2, units = n_q + 2 * n_kv;
    const int u0 = blockIdx.y * upw, nu = min(upw, units - u0);
    const size_t RN = (size_t)r.B * r.n * units * d;
    const size_t base_idx = (size_t)row * units * d;
    float* qo = q_out + (size_t)row * n_q * d;
    const bool pad = r.lim && (row % r.n) >= r.lim[row / r.n];   // padding rows are not cached
    if (!ok || pad) {
        if (!pad && threadIdx.x == 0 && blockIdx.y == 0) {
            const bool bad_slot = slot < 0 || slot >= r.max_slots;
            flag_error(r.err, bad_slot ? ERR_SLOT : ERR_CTX);
        }
        for (int t = threadIdx.x; t < nu * d; t += blockDim.x) {
            const int u = u0 + t / d;
            if (u < n_q) qo[(size_t)u * d + t % d] = 0.f;
        }
        return;
    }
    const float2* rp = rope + (size_t)pos * hd;
    // this row's K/V position: page, then layer and offset in the page
    const long long pg = kv_page(g, slot, pos / g.P);
    if (pg < 0 && threadIdx.x == 0 && blockIdx.y == 0) flag_error(r.err, ERR_PAGE);
    const long long cbase = pg * g.PS + layer * g.LS + (long long)(pos % g.P) * d;
    for (int t = threadIdx.x; t < nu * hd; t += blockDim.x) {
        const int u = u0 + t / hd, k = t - (t / hd) * hd;
        const size_t c0 = base_idx + (size_t)u * d + k;
        const float a = sum_parts(qkv, P, S, RN, c0), c = sum_parts(qkv, P, S, RN, c0 + hd);
        if (u < n_q + n_kv) {
            const float2 rot = rope_rot(a, c, rp[k]);
            const float x0 = rot.x, x1 = rot.y;
            if (u < n_q) {
                qo[(size_t)u * d + k] = x0;
                qo[(size_t)u * d + k + hd] = x1;
            } else if (pg >= 0) {
                const size_t o = cbase + (u - n_q) * g.HS;
                elem<T>::store(kc, o + k, x0);
                elem<T>::store(kc, o + k + hd, x1);
            }
        } else if (pg >= 0) {
            const size_t o = cbase + (u - n_q - n_kv) * g.HS;
            elem<T>::store(vc, o + k, a);
            elem<T>::store(vc, o + k + hd, c);
        }
    }
}

// ------------------------------------------------------------------ attention
// Split-context decode attention (flash-decoding style), fp32 arithmetic.
// Work-group (b, kv head, chunk c) covers context positions [c*CH, (c+1)*CH)
// of that sequence; query row (i, head h) of the sequence attends positions
// [0, kv_len + off + i] (causal inside the block of new tokens).  Each
// work-group writes (m, l, o[d]) per query row and head; k_attn_combine
// merges the chunks.  D/8 lanes share one position, 8 dims per lane.
constexpr int ATT_CH = 256;
constexpr int ATT_RG = 4;   // query rows per pass

template <typename T, int D>
__global__ void __launch_bounds__(256) k_attn_partial(rows_t r, const float* q, int n_q, int n_kv,
                                                      const T* kc, const T* vc, kv_geom kg, int layer, float* part,
                                                      int max_chunks)
{
    constexpr int LPP = D / 8;          // lanes per position
    constexpr int PPW = WAVE / LPP;     // positions per wave-step
    constexpr int NPG = 4 * PPW;        // position groups per work-group
    __shared__ float s_m[NPG][ATT_RG];
    __shared__ float s_l[NPG][ATT_RG];
    __shared__ float s_o[NPG][ATT_RG][D];

    int b = blockIdx.x / n_kv, kvh = blockIdx.x - b * n_kv;
    int c = blockIdx.y;
    int slot = r.slots[b];
    if (slot < 0 || slot >= r.max_slots) return;   // flagged by k_rope_kv
    int basepos = r.kv_len[slot] + r.off;
    int ctx = basepos + r.n;
    if (ctx > r.max_ctx) ctx = r.max_ctx;
    int p0 = c * ATT_CH;
    if (p0 >= ctx) return;
    int p1 = min(p0 + ATT_CH, ctx);

    int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int pg = lane / LPP;                 // position group within the wave
    int dd = (lane % LPP) * 8;
    int G = n_q / n_kv;
    int QR = G * r.n;
    float scale = rsqrtf((float)D);
    const long long hbase = layer * kg.LS + kvh * kg.HS;      // + page * PS + (p % P) * D

    for (int rg0 = 0; rg0 < QR; rg0 += ATT_RG) {
        float qv[ATT_RG][8], m[ATT_RG], l[ATT_RG], o[ATT_RG][8];
        int lim[ATT_RG];
#pragma unroll
        for (int rr = 0; rr < ATT_RG; ++rr) {
            int qr = rg0 + rr;
            bool live = qr < QR;
            int g = live ? qr / r.n : 0, i = live ? qr - g * r.n : 0;
            int hq = kvh * G + g;
            const float* qp = q + ((size_t)(b * r.n + i) * n_q + hq) * D + dd;
#pragma unroll
            for (int e = 0; e < 8; ++e) { qv[rr][e] = live ? qp[e] * scale : 0.f; o[rr][e] = 0.f; }
            m[rr] = -INFINITY; l[rr] = 0.f;
            lim[rr] = live ? basepos + i : -1;   // last visible position
        }
        for (int pb = p0 + w * PPW; pb < p1; pb += NPG) {
            int p = pb + pg;
            bool pv = p < p1;
            float kf[8], vf[8];
            long long page = pv ? kv_page(kg, slot, p / kg.P) : 0;
            if (page < 0) {
                if ((lane % LPP) == 0) flag_error(r.err, ERR_PAGE);
                pv = false;
            }
            if (pv) {
                const size_t o = page * kg.PS + hbase + (long long)(p % kg.P) * D + dd;
#pragma unroll
                for (int e = 0; e < 8; ++e) { kf[e] = elem<T>::load(kc, o + e); vf[e] = elem<T>::load(vc, o + e); }
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) { kf[e] = 0.f; vf[e] = 0.f; }
            }
#pragma unroll
            for (int rr = 0; rr < ATT_RG; ++rr) {
                float s = 0.f;
#pragma unroll
                for (int e = 0; e < 8; ++e) s += qv[rr][e] * kf[e];
#pragma unroll
                for (int ofs = LPP / 2; ofs > 0; ofs >>= 1) s += __shfl_xor(s, ofs, WAVE);
                if (pv && p <= lim[rr]) {
                    float mn = fmaxf(m[rr], s);
                    float corr = __expf(m[rr] - mn);
                    float pe = __expf(s - mn);
                    l[rr] = l[rr] * corr + pe;
#pragma unroll
                    for (int e = 0; e < 8; ++e) o[rr][e] = o[rr][e] * corr + pe * vf[e];
                    m[rr] = mn;
                }
            }
        }
        // merge the NPG position groups through LDS
        int gidx = w * PPW + pg;
        if ((lane % LPP) == 0) {
#pragma unroll
            for (int rr = 0; rr < ATT_RG; ++rr) { s_m[gidx][rr] = m[rr]; s_l[gidx][rr] = l[rr]; }
        }
#pragma unroll
        for (int rr = 0; rr < ATT_RG; ++rr)
#pragma unroll
            for (int e = 0; e < 8; ++e) s_o[gidx][rr][dd + e] = o[rr][e];
        __syncthreads();
        for (int t = threadIdx.x; t < ATT_RG * D; t += blockDim.x) {
            int rr = t / D, k = t - rr * D;
            int qr = rg0 + rr;
            if (qr >= QR) continue;
            float mm = -INFINITY;
            for (int gq = 0; gq < NPG; ++gq) mm = fmaxf(mm, s_m[gq][rr]);
            float ls = 0.f, os = 0.f;
            if (mm > -INFINITY) {
                for (int gq = 0; gq < NPG; ++gq) {
                    float f = s_m[gq][rr] > -INFINITY ? __expf(s_m[gq][rr] - mm) : 0.f;
                    ls += s_l[gq][rr] * f;
                    os += s_o[gq][rr][k] * f;
                }
            }
            int g = qr / r.n, i = qr - g * r.n;
            int hq = kvh * G + g;
            float* pp = part + (((size_t)(b * r.n + i) * n_q + hq) * max_chunks + c) * (D + 2);
            if (k == 0) { pp[0] = mm; pp[1] = ls; }
            pp[2 + k] = os;
        }
        __syncthreads();
    }
}

// MFMA attention for a bf16 cache.  Work-group (b, kv head, chunk, query-row
// slice z): a sequence's context is split evenly into ceil(ctx / ch) chunks
// and each wave takes a quarter of its chunk in blocks of 32 positions.  Per
// block:
//   S^T = K Q^T with v_mfma_f32_16x16x32_bf16: K rows straight from global
//   memory (lane l: position l%16 of a 16-row tile, dims 8*(4ks + l/16)+0..7),
//   Q^T pre-scaled by log2(e)/sqrt(d).  Lane l then holds the scores of query
//   row l%16 at positions 4*(l/16) + r and 16 + 4*(l/16) + r (r = 0..3), which
//   is exactly the B operand layout of the next product, so P never leaves
//   registers.
//   O^T += V^T P^T: V is staged row-major in a wave-private LDS tile (row
//   stride d + 8) and read back transposed with ds_read_b64_tr_b16.
//   The next block's K and V are loaded while the current one computes (with
//   two query tiles, the other wave on the SIMD covers the loads instead).
// The online softmax runs per query row in base 2 with lazy rescaling (the
// reference max of a row moves only when the block max exceeds it by more
// than 8, bounding the exp2 terms by 256); the four waves are merged
// through LDS and the chunk result (m in natural-log units, l, o[d]) goes to
// the same partial buffer k_attn_combine reads.
// Chunk length of the MFMA kernel, chosen per launch: enough chunks per
// sequence for about ATT_TARGET_WGS work-groups in all (two per CU), each at
// least ATT_MIN_CHUNK positions, so a large batch streams a whole context per
// work-group and a small one still fills the GPU.
#ifndef ATT_INTERLEAVE
#define ATT_INTERLEAVE 1
#endif
// K and V are read once per launch: non-temporal loads (cache policy bit 1,
// nt on this target) stream them past the caches, which HBM serves faster
// (7.2 against 6.4 TB/s for plain 16-byte streaming loads measured on this part)
#ifndef ATT_NT
#define ATT_NT 2
#endif
#ifndef ATT_TARGET_WGS
#define ATT_TARGET_WGS 512
#endif
#ifndef ATT_MIN_CHUNK
#define ATT_MIN_CHUNK 512
#endif

// two waves per SIMD where the registers allow it without spills (one query
// tile; two tiles with a single K/V register set); three or four tiles run one
// wave per SIMD
//
// RoPE and the cache write of the new rows are part of the kernel: from the
// QKV projection's output (qkv_src, kernels.h) each work-group forms its
// rotated query rows and writes its KV head's new K (rotated) and V rows of
// its context range to the cache before its waves read them (each
// work-group of the head covering new positions writes those it reads;
// query-row slices of one chunk write the same values), and it raises the
// slot, position and page flags for them.
template <int D, int MQ, bool PAGED>
__global__ void __launch_bounds__(256, MQ <= 2 ? 2 : 1) k_attn_mfma(rows_t r, int n_q, int n_kv, const uint16_t* kc,
                                                   const uint16_t* vc, kv_geom kg, int layer, float* part, int max_chunks, int ch,
                                                   void* out, int out_t, qkv_src qs)
{
    constexpr int KS = D / 32;      // k-steps over the head dim
    constexpr int NBD = D / 16;     // 16-wide blocks of the head dim
    constexpr int LDV = D + 8;      // LDS row stride (elements)
    constexpr int CPP = D / 8;      // 16-byte pieces per cached position
    __shared__ __attribute__((aligned(16))) uint16_t Vs[4][32 * LDV];
    __shared__ float s_ml[4][2][16];

    const int b = blockIdx.x / n_kv, kvh = blockIdx.x - b * n_kv;
    const int c = blockIdx.y, z = blockIdx.z;
    // wave-uniform by construction; readfirstlane lets the compiler keep them
    // (and the buffer resources built from them) in scalar registers
    const int slot = __builtin_amdgcn_readfirstlane(r.slots[b]);
    if (slot < 0 || slot >= r.max_slots) {         // flagged once per sequence; a direct output is zeroed
        if (c == 0 && z == 0 && kvh == 0 && threadIdx.x == 0) flag_error(r.err, ERR_SLOT);
        const int G = n_q / n_kv;
        for (int idx = threadIdx.x; out && idx < 16 * MQ * D; idx += 256) {
            const int qrow = z * 16 * MQ + idx / D, d = idx % D;
            if (qrow >= G * r.n) continue;
            const int g = qrow / r.n, i = qrow - g * r.n;
            const size_t oi = ((size_t)(b * r.n + i) * n_q + kvh * G + g) * D + d;
            if (out_t == ACT_F16) store_act<_Float16>(out, oi, 0.f);
            else if (out_t == ACT_BF16) store_act<uint16_t>(out, oi, 0.f);
            else store_act<float>(out, oi, 0.f);
        }
        return;
    }
    const int basepos = __builtin_amdgcn_readfirstlane(r.kv_len[slot]) + r.off;
    int ctx = basepos + r.n;
    if (ctx > r.max_ctx) ctx = r.max_ctx;
    // rows (b, i >= nlive) are padding: neither cached nor flagged
    const int nlive = r.lim ? min(r.n, max(__builtin_amdgcn_readfirstlane(r.lim[b]), 0)) : r.n;
    if (c == 0 && z == 0 && kvh == 0 && threadIdx.x == 0 && nlive > 0 &&
        (basepos < 0 || basepos + nlive > r.max_ctx))
        flag_error(r.err, ERR_CTX);                 // a live row's position outside [0, max_ctx)
    // the sequence's ceil(ctx / ch) chunks (the count k_attn_combine reads)
    // split its context evenly, in multiples of 32 positions
    const int nch = (ctx + ch - 1) / ch;
    const int clen = ((ctx + nch - 1) / nch + 31) & ~31;
    const int p0 = c * clen;
    if (p0 >= ctx) return;
    const int p1 = min(p0 + clen, ctx);
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int cq = lane >> 4, lr = lane & 15;
    const int G = n_q / n_kv, QR = G * r.n;
    const int qbase = z * 16 * MQ;
    const int units = n_q + 2 * n_kv;                          // head units of a projection row
    const size_t RN = (size_t)r.B * r.n * units * D;           // elements of one split

    const float qscale = 1.4426950408889634f * rsqrtf((float)D);

    // Q^T fragments (B operand of S^T = K Q^T), read from LDS after the
    // pass below has formed the rotated query rows
    bf16x8 qf[MQ][KS];
    int lim[MQ];

    const long long hbase = hbase_of(kg, layer, kvh);         // + page * PS (+ (p % P) * D)
    const uint16_t* K = kc + (PAGED ? 0 : slot * kg.PS) + hbase;
    const uint16_t* V = vc + (PAGED ? 0 : slot * kg.PS) + hbase;
    uint16_t* vs = Vs[w];

    float m[MQ], lsum[MQ];
    floatx4 o[MQ][NBD];
#pragma unroll
    for (int mt = 0; mt < MQ; ++mt) {
        m[mt] = -INFINITY;
        lsum[mt] = 0.f;
#pragma unroll
        for (int nb = 0; nb < NBD; ++nb) o[mt][nb] = (floatx4){0.f, 0.f, 0.f, 0.f};
    }

#if ATT_INTERLEAVE
    // the four waves take the chunk's 32-position blocks in turn, so the
    // work-group reads K and V as two contiguous streams
    const int wq0 = p0 + 32 * w, wq1 = p1, wstep = 128;
#else
    const int wlen = ((clen + 3) / 4 + 31) & ~31;                  // positions per wave
    const int wq0 = p0 + w * wlen, wq1 = min(wq0 + wlen, p1), wstep = 32;
#endif
    // K fragments of the two 16-position tiles and the V block of the block at
    // blk, through buffer resources limited to the cached positions: reads at
    // or past ctx return 0 without touching memory.  Positions past the wave's
    // range get -inf scores below, so their P is 0.  The dense cache has one
    // resource per sequence; the paged one a resource per page (a block of 32
    // positions never straddles pages), none (0 records) for a missing page.
    __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc((void*)K, 0, ctx * D * 2, 0x00020000);
    __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc((void*)V, 0, ctx * D * 2, 0x00020000);
    const int koff = (lr * D + 8 * cq) * 2;                         // + (16 pt) D 2 + 64 ks
    const int voff = ((lane / CPP) * D + (lane % CPP) * 8) * 2;     // + t (64 / CPP) D 2
    // Paged cache: the pages of the wave's blocks wq0 + k wstep for k in
    // [kw, kw + 128), lane l holding those of k = kw + l and kw + 64 + l
    // (-1: missing), loaded together when a block leaves the window, which
    // also raises ERR_PAGE for a missing page of the wave's range.  A block
    // then finds its page with a lane read: a table load or a flag store per
    // block would make the compiler wait for every load in flight (they
    // complete in order) before the next block's loads go out.
    int pgw[2] = {-1, -1}, kw = -(1 << 20);
    int sb = 0;                                                     // scalar offset of the block
    // the resources and offset of block blk, then its K and its V loads
    auto kv_setup = [&](int blk) {
        sb = __builtin_amdgcn_readfirstlane(blk * D * 2);
        if constexpr (PAGED) {
            const int lp = __builtin_amdgcn_readfirstlane(blk / kg.P), in0 = lp * kg.P;
            const int k = __builtin_amdgcn_readfirstlane((blk - wq0) / wstep);
            if (k < kw || k >= kw + 128) {
                kw = k;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int bj = wq0 + (k + 64 * h + lane) * wstep;
                    pgw[h] = (int)kv_page(kg, slot, bj / kg.P);
                    if (pgw[h] < 0 && bj < wq1)     // a global, not a generic, store: see above
                        ((volatile __attribute__((address_space(1))) uint32_t*)r.err)[ERR_PAGE] = 1u;
                }
            }
            const int j = k - kw;
            // two lane reads and a scalar select: a vector select would need a
            // temporary register, which may be one a load in flight still writes
            const int pa = __builtin_amdgcn_readlane(pgw[0], j & 63), pb = __builtin_amdgcn_readlane(pgw[1], j & 63);
            const int pg = j < 64 ? pa : pb;
            const int nrec = pg < 0 ? 0 : max(0, min(kg.P, ctx - in0)) * D * 2;
            const long long po = (pg < 0 ? 0 : pg) * kg.PS;
            krs = __builtin_amdgcn_make_buffer_rsrc((void*)(K + po), 0, nrec, 0x00020000);
            vrs = __builtin_amdgcn_make_buffer_rsrc((void*)(V + po), 0, nrec, 0x00020000);
            sb = __builtin_amdgcn_readfirstlane((blk - in0) * D * 2);
        }
    };
    // no block: resources of zero records, whose loads return zeros without
    // touching memory (so that a wave's loads need not sit in a branch)
    auto kv_none = [&] {
        sb = 0;
        krs = __builtin_amdgcn_make_buffer_rsrc((void*)K, 0, 0, 0x00020000);
        vrs = __builtin_amdgcn_make_buffer_rsrc((void*)V, 0, 0, 0x00020000);
    };
    auto issue_k = [&](u32x4 (&kf)[2][KS]) {
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                kf[pt][ks] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                           krs, koff + (16 * pt * D + 32 * ks) * 2, sb, ATT_NT));
    };
    auto issue_v = [&](u32x4 (&vv)[CPP / 2]) {
#pragma unroll
        for (int t = 0; t < CPP / 2; ++t)
            vv[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                  vrs, voff + t * (64 / CPP) * D * 2, sb, ATT_NT));
    };
    auto load_kv = [&](int blk, u32x4 (&kf)[2][KS], u32x4 (&vv)[CPP / 2]) {
        kv_setup(blk);
        issue_k(kf);
        issue_v(vv);
    };
    // lane l's pieces of the transposing LDS reads that build V^T fragments:
    // positions 4*(l/16) + (l%16)/4 (+16), dims 4*(l%4) of each 16-dim block
    const int trow = 4 * cq + (lr >> 2), tcol = 4 * (lr & 3);
    // after_k runs once the block's K fragments are consumed (after the last
    // tile's S^T products), after_v once its V is in LDS: a single register
    // set requests the next block's K and V there
    auto block = [&](int blk, const u32x4 (&kf)[2][KS], const u32x4 (&vv)[CPP / 2], auto after_k, auto after_v) {
        bf16x8 pf[MQ];
#pragma unroll
        for (int mt = 0; mt < MQ; ++mt) {
            floatx4 st[2];
#pragma unroll
            for (int pt = 0; pt < 2; ++pt) {
                st[pt] = (floatx4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    st[pt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kf[pt][ks]), qf[mt][ks],
                                                                     st[pt], 0, 0, 0);
            }
            if (mt == MQ - 1) after_k();
            float bm = -INFINITY;
#pragma unroll
            for (int pt = 0; pt < 2; ++pt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int pos = blk + 16 * pt + 4 * cq + i;
                    float sv = st[pt][i];
                    if (pos >= wq1 || pos > lim[mt]) sv = -INFINITY;
                    st[pt][i] = sv;
                    bm = fmaxf(bm, sv);
                }
            bm = fmaxf(bm, __shfl_xor(bm, 16, WAVE));
            bm = fmaxf(bm, __shfl_xor(bm, 32, WAVE));
            // lazy rescaling: a row moves its reference max (and rescales its
            // sums) only when the block max exceeds it by more than 8, so the
            // exp2 terms stay <= 256; the result is the same softmax
            const bool need = bm > m[mt] + 8.f;
            if (__builtin_amdgcn_ballot_w64(need)) {
                const float mn = need ? bm : m[mt];
                const float corr = m[mt] == -INFINITY ? 0.f : exp2f(m[mt] - mn);
                m[mt] = mn;
                lsum[mt] *= corr;
#pragma unroll
                for (int nb = 0; nb < NBD; ++nb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) o[mt][nb][i] *= corr;
            }
            const float mn = m[mt];
            float pv[8];
#pragma unroll
            for (int pt = 0; pt < 2; ++pt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float x = st[pt][i];
                    pv[pt * 4 + i] = x == -INFINITY ? 0.f : exp2f(x - mn);
                    lsum[mt] += pv[pt * 4 + i];
                }
            pf[mt] = __builtin_bit_cast(bf16x8, (u32x4){pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]),
                                                        pack_bf16x2(pv[4], pv[5]), pack_bf16x2(pv[6], pv[7])});
        }
        // V block -> wave-private LDS tile (row-major, padded)
#pragma unroll
        for (int t = 0; t < CPP / 2; ++t) {
            const int piece = t * 64 + lane;
            const int pos = piece / CPP, ch = piece - pos * CPP;
            *(u32x4*)(vs + pos * LDV + ch * 8) = vv[t];
        }
        after_v();
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // O^T += V^T P^T; V^T fragments from two transposing reads: lane l gets
        // dim 16 nb + l%16 at positions 4(l/16) + 0..3 and 16 + 4(l/16) + 0..3,
        // the k order of pf
#pragma unroll
        for (int nb = 0; nb < NBD; ++nb) {
            const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) v4s*)(vs + trow * LDV + 16 * nb + tcol));
            const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) v4s*)(vs + (16 + trow) * LDV + 16 * nb + tcol));
            const bf16x8 vt = __builtin_bit_cast(bf16x8, (v8s){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
#pragma unroll
            for (int mt = 0; mt < MQ; ++mt) o[mt][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vt, pf[mt], o[mt][nb], 0, 0, 0);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };

    // two register sets: the next block's K and V load while this one computes
    u32x4 kf0[2][KS], kf1[2][KS], vv0[CPP / 2], vv1[CPP / 2];
    // a wave whose first block holds no new row loads it during the pass below
    const bool early = wq0 + 32 <= basepos;
    if (early) load_kv(wq0, kf0, vv0);
    // one pass of the work-group over (a) its 16 MQ query rows, rotated,
    // scaled and rounded to bf16 into LDS (the V tiles' space, unused until the
    // first block) and (b) its KV head's new rows [n0, p1), K rotated and V,
    // stored to the cache.  A task is 4 columns and their RoPE partners D/2
    // further; a thread's task loads go out together, so the pass costs a
    // memory round trip or two before the K/V stream starts.
    uint16_t* qst = &Vs[0][0];                                  // [16 MQ][D]
    static_assert(16 * MQ * D <= 4 * 32 * LDV, "query rows fit the V tiles");
    {
        constexpr int QG = D / 8;                               // 4-column groups of a half row
        const int n0 = max(p0, basepos), nkv = max(p1 - n0, 0);
        // tasks: the tile's live query rows, then the new K/V rows, then the
        // tile's rows past QR (zeros, no loads), so the loading tasks come first
        const int nlr = max(min(16 * MQ, QR - qbase), 0);
        const int nlq = nlr * QG, nkt = nkv * 2 * QG, ntask = 16 * MQ * QG + nkt;
        const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
        // columns ci and ci + D/2 of the projection output
        auto sum4x2 = [&](size_t ci, float4& a, float4& c) {
            a = z4;
            c = z4;
            if (qs.S <= 1) {
                a = *(const float4*)(qs.qkv + ci);
                c = *(const float4*)(qs.qkv + ci + D / 2);
            } else {
                add_splits2(a, c, qs.P, qs.S, RN, ci, ci + D / 2);
            }
        };
        // columns (a, c) -> (a cos - c sin, a sin + c cos) times scl, for 4 columns
        auto rot4 = [&](float4 a, float4 c, const float2* rp, float scl, float4& lo, float4& hi) {
            const float4 c01 = *(const float4*)rp, c23 = *(const float4*)(rp + 2);
            const float2 r0 = rope_rot(a.x, c.x, make_float2(c01.x, c01.y));
            const float2 r1 = rope_rot(a.y, c.y, make_float2(c01.z, c01.w));
            const float2 r2 = rope_rot(a.z, c.z, make_float2(c23.x, c23.y));
            const float2 r3 = rope_rot(a.w, c.w, make_float2(c23.z, c23.w));
            lo = make_float4(r0.x * scl, r1.x * scl, r2.x * scl, r3.x * scl);
            hi = make_float4(r0.y * scl, r1.y * scl, r2.y * scl, r3.y * scl);
        };
        auto put4 = [](uint16_t* d, float4 v) { *(uint2*)d = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w)); };
        for (int t = threadIdx.x; t < ntask; t += 256) {
            if (t < nlq || t >= nlq + nkt) {
                const int tq = t < nlq ? t : t - nkt;           // query-row task: row rr of the tile
                const int rr = tq / QG, gq = tq - rr * QG, qrow = qbase + rr;
                float4 lo = z4, hi = z4;
                if (qrow < QR) {
                    const int g = qrow / r.n, i = qrow - g * r.n, pos = basepos + i;
                    // rows k_rope_kv does not rotate (padding, outside [0, max_ctx)) keep q = 0, as it writes
                    if (i < nlive && pos >= 0 && pos < r.max_ctx) {
                        const size_t ci = ((size_t)(b * r.n + i) * units + kvh * G + g) * D + 4 * gq;
                        float4 a, c;
                        sum4x2(ci, a, c);
                        rot4(a, c, qs.rope + (size_t)pos * (D / 2) + 4 * gq, qscale, lo, hi);
                    }
                }
                put4(qst + rr * D + 4 * gq, lo);
                put4(qst + rr * D + D / 2 + 4 * gq, hi);
            } else {
                const int tt = t - nlq, j = tt / (2 * QG), rem = tt - j * (2 * QG);
                const bool isv = rem >= QG;
                const int gq = isv ? rem - QG : rem, i = n0 - basepos + j, pos = basepos + i;
                if (i >= nlive) continue;                       // padding rows are not cached
                const long long pg = kv_page(kg, slot, pos / kg.P);
                if (pg < 0) {
                    if (gq == 0) flag_error(r.err, ERR_PAGE);
                    continue;
                }
                const size_t ci = ((size_t)(b * r.n + i) * units + n_q + (isv ? n_kv : 0) + kvh) * D + 4 * gq;
                float4 lo, hi;
                sum4x2(ci, lo, hi);
                if (!isv) rot4(lo, hi, qs.rope + (size_t)pos * (D / 2) + 4 * gq, 1.f, lo, hi);
                uint16_t* dst = (uint16_t*)(isv ? vc : kc) + pg * kg.PS + hbase_of(kg, layer, kvh) + (long long)(pos % kg.P) * D;
                put4(dst + 4 * gq, lo);
                put4(dst + D / 2 + 4 * gq, hi);
            }
        }
        if (nkv > 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the new rows are stored before any wave reads them
        __syncthreads();                                        // and the query rows are in LDS
    }
    if (!early) load_kv(wq0, kf0, vv0);
    // the query fragments from LDS (rows past QR are zeros)
#pragma unroll
    for (int mt = 0; mt < MQ; ++mt) {
        const int qrow = qbase + 16 * mt + lr;
        const bool live = qrow < QR;
        const int i = (live ? qrow : 0) % r.n;
        lim[mt] = live ? basepos + i : -1;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            qf[mt][ks] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qst + (16 * mt + lr) * D + 8 * (4 * ks + cq)));
    }
    lds_barrier();                                              // every wave holds its q before the V tiles take the space

    if constexpr (MQ == 2 || MQ == 4) {
        // one register set: with two tiles 246 VGPRs instead of 366, so two
        // waves per SIMD and the other wave hides each block's loads; with four
        // tiles the second set would spill (the 32B verify at gamma 9 took 822
        // against 500 us per launch).  Three tiles keep both sets at one wave
        // per SIMD (384 against 425 us at gamma 7).
        // The next block's K loads go out once this block's S^T products have
        // read K, its V loads once this block's V is in LDS; after the wave's
        // last block they read nothing.  Issued in a branch, they would make
        // the compiler wait for them wherever the paths join.
        for (int blk = wq0; blk < wq1; blk += wstep) {
            const int nx = blk + wstep;
            block(
                blk, kf0, vv0,
                [&] {
                    if (nx < wq1) kv_setup(nx);
                    else kv_none();
                    issue_k(kf0);
                },
                [&] { issue_v(vv0); });
        }
    } else {
        const auto none = [] {};
        for (int blk = wq0; blk < wq1; blk += 2 * wstep) {
            load_kv(blk + wstep, kf1, vv1);
            block(blk, kf0, vv0, none, none);
            if (blk + wstep >= wq1) break;
            load_kv(blk + 2 * wstep, kf0, vv0);
            block(blk + wstep, kf1, vv1, none, none);
        }
    }
#pragma unroll
    for (int mt = 0; mt < MQ; ++mt) {
        lsum[mt] += __shfl_xor(lsum[mt], 16, WAVE);
        lsum[mt] += __shfl_xor(lsum[mt], 32, WAVE);
    }

    // merge the four waves, 16 query rows at a time, through the (now free) V tiles
    float* so = (float*)&Vs[0][0];   // [4 waves][16 rows][D]
    const float LN2 = 0.6931471805599453f;
    for (int mt = 0; mt < MQ; ++mt) {
        __syncthreads();
        if (cq == 0) { s_ml[w][0][lr] = m[mt]; s_ml[w][1][lr] = lsum[mt]; }
#pragma unroll
        for (int nb = 0; nb < NBD; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i) so[(w * 16 + lr) * D + 16 * nb + 4 * cq + i] = o[mt][nb][i];
        __syncthreads();
        for (int idx = threadIdx.x; idx < 16 * D; idx += 256) {
            const int qr = idx / D, d = idx - qr * D;
            const int qrow = qbase + 16 * mt + qr;
            if (qrow >= QR) continue;
            float mm = -INFINITY;
#pragma unroll
            for (int ww = 0; ww < 4; ++ww) mm = fmaxf(mm, s_ml[ww][0][qr]);
            float ls = 0.f, os = 0.f;
            if (mm > -INFINITY) {
#pragma unroll
                for (int ww = 0; ww < 4; ++ww) {
                    const float mw = s_ml[ww][0][qr];
                    const float f = mw > -INFINITY ? exp2f(mw - mm) : 0.f;
                    ls += s_ml[ww][1][qr] * f;
                    os += so[(ww * 16 + qr) * D + d] * f;
                }
            }
            const int g = qrow / r.n, i = qrow - g * r.n;
            if (out) {
                // a single chunk per sequence: the normalized output directly (what
                // k_attn_combine computes from one chunk)
                const size_t oi = ((size_t)(b * r.n + i) * n_q + kvh * G + g) * D + d;
                const float v = ls > 0.f ? os / ls : 0.f;
                if (out_t == ACT_F16) store_act<_Float16>(out, oi, v);
                else if (out_t == ACT_BF16) store_act<uint16_t>(out, oi, v);
                else store_act<float>(out, oi, v);
                continue;
            }
            float* pp = part + (((size_t)(b * r.n + i) * n_q + kvh * G + g) * max_chunks + c) * (D + 2);
            if (d == 0) { pp[0] = mm * LN2; pp[1] = ls; }
            pp[2 + d] = os;
        }
    }
}

template <typename O>
__global__ void k_attn_combine(rows_t r, int n_q, int D, const float* part, int max_chunks, int chunk, void* out)
{
    int row = blockIdx.x / n_q, hq = blockIdx.x - row * n_q;
    int b = row / r.n;
    int slot = r.slots[b];
    int ctx = 0;
    if (slot >= 0 && slot < r.max_slots) ctx = min(r.kv_len[slot] + r.off + r.n, r.max_ctx);
    int nch = (ctx + chunk - 1) / chunk;
    if (nch > max_chunks) nch = max_chunks;
    const float* pp = part + ((size_t)row * n_q + hq) * max_chunks * (D + 2);
    // chunks are merged in order, sixteen at a time: the loads of a batch go
    // out together (past the last chunk they repeat chunk nch - 1 and are not
    // used), and a later batch with a larger maximum rescales the sums so far.
    // Up to sixteen chunks this is one memory round trip and the same
    // arithmetic as taking the maximum first.
    constexpr int CB = 16;
    for (int k = threadIdx.x; k < D; k += blockDim.x) {
        float mm = -INFINITY, ls = 0.f, os = 0.f;
        for (int c0 = 0; c0 < nch; c0 += CB) {
            float cm[CB], cl[CB], co[CB];
#pragma unroll
            for (int u = 0; u < CB; ++u) {
                const float* pc = pp + (size_t)min(c0 + u, nch - 1) * (D + 2);
                cm[u] = pc[0];
                cl[u] = pc[1];
                co[u] = pc[2 + k];
            }
            float bm = mm;
#pragma unroll
            for (int u = 0; u < CB; ++u)
                if (c0 + u < nch && cl[u] > 0.f) bm = fmaxf(bm, cm[u]);
            if (bm > mm && mm > -INFINITY) {
                const float f = __expf(mm - bm);
                ls *= f;
                os *= f;
            }
            mm = bm;
#pragma unroll
            for (int u = 0; u < CB; ++u)
                if (c0 + u < nch && cl[u] > 0.f) {
                    const float f = __expf(cm[u] - mm);
                    ls += cl[u] * f;
                    os += co[u] * f;
                }
        }
        store_act<O>(out, ((size_t)row * n_q + hq) * D + k, ls > 0.f ? os / ls : 0.f);
    }
}

// ------------------------------------------------------------------ swiglu
// out[row][f] = SiLU(g) * u with (g, u) = gu[row][f], gu[row][F + f]
template <typename O>
__global__ void __launch_bounds__(256) k_silu_mul(const float* gu, const float* P, int S, int R, int F, void* out)
{
    const int row = blockIdx.x;
    const int f = (blockIdx.y * 256 + threadIdx.x) * 4;
    if (f >= F) return;
    const size_t RN = (size_t)R * 2 * F;
    const size_t gi = (size_t)row * 2 * F + f, ui = gi + F;
    float4 g, u;
    if (S <= 1) {
        g = *(const float4*)(gu + gi);
        u = *(const float4*)(gu + ui);
    } else {
        g = add_splits(make_float4(0.f, 0.f, 0.f, 0.f), P, S, RN, gi);
        u = add_splits(make_float4(0.f, 0.f, 0.f, 0.f), P, S, RN, ui);
    }
    const size_t o = (size_t)row * F + f;
    store_act<O>(out, o, g.x / (1.f + __expf(-g.x)) * u.x);
    store_act<O>(out, o + 1, g.y / (1.f + __expf(-g.y)) * u.y);
    store_act<O>(out, o + 2, g.z / (1.f + __expf(-g.z)) * u.z);
    store_act<O>(out, o + 3, g.w / (1.f + __expf(-g.w)) * u.w);
}

// ------------------------------------------------------------------ kv length
__global__ void k_kv_advance(int B, const int32_t* slots, const int32_t* inc, int inc_const,
                             int32_t* kv_len, int max_slots, uint32_t* err)
{
    int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    int s = slots[b];
    if (s < 0 || s >= max_slots) { flag_error(err, ERR_SLOT); return; }
    kv_len[s] += inc ? inc[b] : inc_const;
}

__global__ void k_prefill_lim(int B, const int32_t* len, int t0, int nc, int ld, int32_t* lim, uint32_t* err)
{
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    int n = len[b];
    if (n < 0 || n > ld) {
        flag_error(err, ERR_LEN);
        n = 0;
    }
    lim[b] = min(max(n - t0, 0), nc);
}

template <typename T>
__global__ void k_kv_poison(const int32_t* slots, const int32_t* kv_len, int span, T* kc, T* vc, kv_geom g,
                            int n_layers, int n_kv, int D, int max_slots, int max_ctx)
{
    int b = blockIdx.x;
    int s = slots[b];
    if (s < 0 || s >= max_slots) return;
    int p0 = kv_len[s];
    int p1 = min(p0 + span, max_ctx);
    if (p0 < 0) p0 = 0;
    int per = (p1 > p0 ? p1 - p0 : 0) * D;
    size_t total = (size_t)n_layers * n_kv * per;
    for (size_t t = threadIdx.x; t < total; t += blockDim.x) {
        size_t lh = t / per;
        int rem = (int)(t - lh * per);
        int l = (int)(lh / n_kv), h = (int)(lh - (size_t)l * n_kv);
        const int p = p0 + rem / D;
        const long long pg = kv_page(g, s, p / g.P);
        if (pg < 0) continue;
        size_t o = pg * g.PS + l * g.LS + h * g.HS + (long long)(p % g.P) * D + rem % D;
        elem<T>::store(kc, o, __int_as_float(0x7fc00000));
        elem<T>::store(vc, o, __int_as_float(0x7fc00000));
    }
}

}  // namespace

// ======================================================================= launchers
template <typename T>
static void embed_norm_t(const rows_t& r, const int32_t* tokA, int sA, const int32_t* tokB, int sB, const T* E, int H,
                         int V, float* h, const T* gain, float eps, void* out, act_t t, hipStream_t s)
{
    const int R = r.B * r.n;
    const int th = H >= 4096 ? 1024 : 256;
    if (t == ACT_F32) k_embed_rmsnorm<T, float><<<R, th, 0, s>>>(r, tokA, sA, tokB, sB, E, H, V, h, gain, eps, out);
    else if (t == ACT_BF16) k_embed_rmsnorm<T, uint16_t><<<R, th, 0, s>>>(r, tokA, sA, tokB, sB, E, H, V, h, gain, eps, out);
    else k_embed_rmsnorm<T, _Float16><<<R, th, 0, s>>>(r, tokA, sA, tokB, sB, E, H, V, h, gain, eps, out);
}

void launch_embed_rmsnorm(const rows_t& r, const int32_t* tokA, int sA, const int32_t* tokB, int sB, const void* E,
                          int w_f32, int H, int V, float* h, const void* gain, float eps, void* out, act_t out_t,
                          hipStream_t s)
{
    if (w_f32) embed_norm_t(r, tokA, sA, tokB, sB, (const float*)E, H, V, h, (const float*)gain, eps, out, out_t, s);
    else embed_norm_t(r, tokA, sA, tokB, sB, (const uint16_t*)E, H, V, h, (const uint16_t*)gain, eps, out, out_t, s);
}

template <typename G, int NPT>
static void add_rmsnorm_n(float* h, const float* P, int S, int R, int H, const G* g, float eps, void* out, act_t t,
                          hipStream_t s)
{
    const int th = ((H / 4 + NPT - 1) / NPT + 63) & ~63;      // <= 1024 by the caller's choice of NPT
    if (t == ACT_F32) k_add_rmsnorm<G, float, NPT><<<R, th, 0, s>>>(h, P, S, R, H, g, eps, out);
    else if (t == ACT_BF16) k_add_rmsnorm<G, uint16_t, NPT><<<R, th, 0, s>>>(h, P, S, R, H, g, eps, out);
    else k_add_rmsnorm<G, _Float16, NPT><<<R, th, 0, s>>>(h, P, S, R, H, g, eps, out);
}

// the fewest float4s per thread that cover the row with at most 1024 threads
// (hidden <= 32768, which the engine's configuration check guarantees)
template <typename G>
static void add_rmsnorm_t(float* h, const float* P, int S, int R, int H, const G* g, float eps, void* out, act_t t,
                          hipStream_t s)
{
    if (H <= 4 * 1024) add_rmsnorm_n<G, 1>(h, P, S, R, H, g, eps, out, t, s);
    else if (H <= 8 * 1024) add_rmsnorm_n<G, 2>(h, P, S, R, H, g, eps, out, t, s);
    else if (H <= 16 * 1024) add_rmsnorm_n<G, 4>(h, P, S, R, H, g, eps, out, t, s);
    else add_rmsnorm_n<G, 8>(h, P, S, R, H, g, eps, out, t, s);
}

void launch_add_rmsnorm(float* h, const float* P, int S, int R, int H, const void* gain, int g_f32, float eps,
                        void* out, act_t out_t, hipStream_t s)
{
    if (g_f32) add_rmsnorm_t(h, P, S, R, H, (const float*)gain, eps, out, out_t, s);
    else add_rmsnorm_t(h, P, S, R, H, (const uint16_t*)gain, eps, out, out_t, s);
}

void launch_rope_kv(const rows_t& r, const float* qkv, const float* P, int S, const float2* rope, int n_q,
                    const cache_t& c, int layer, float* q_out, hipStream_t s)
{
    const int R = r.B * r.n, units = n_q + 2 * c.n_kv;
    const int upw = 512 / c.head_dim;                       // head units per work-group: 256 threads, one pair each
    dim3 grid(R, (units + upw - 1) / upw);
    if (c.kv_f32)
        k_rope_kv<float><<<grid, 256, 0, s>>>(r, qkv, P, S, rope, n_q, c.n_kv, c.head_dim, (float*)c.k, (float*)c.v,
                                              c.g, layer, q_out, upw);
    else
        k_rope_kv<uint16_t><<<grid, 256, 0, s>>>(r, qkv, P, S, rope, n_q, c.n_kv, c.head_dim, (uint16_t*)c.k,
                                                 (uint16_t*)c.v, c.g, layer, q_out, upw);
}

int attention_chunk() { return ATT_CH < ATT_MIN_CHUNK ? ATT_CH : ATT_MIN_CHUNK; }

size_t attention_part_floats(int R, int n_q, int head_dim, int max_chunks)
{
    return (size_t)R * n_q * max_chunks * (head_dim + 2);
}

// a launch whose events (if any) are bound to the kernel's dispatch
template <typename F, typename... Args>
static void launch_ev(F kern, dim3 grid, dim3 block, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1, Args... args)
{
    if (ev0) hipExtLaunchKernelGGL(kern, grid, block, 0, s, ev0, ev1, 0, args...);
    else kern<<<grid, block, 0, s>>>(args...);
}

template <int D, bool PAGED>
static void attn_mfma_launch(int MQ, dim3 grid, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1, const rows_t& r,
                             int n_q, const cache_t& c, int layer, float* part, int mch, int ch, void* out, int out_t,
                             qkv_src qs)
{
    const uint16_t* kc = (const uint16_t*)c.k;
    const uint16_t* vc = (const uint16_t*)c.v;
    auto go = [&](auto kern) {
        launch_ev(kern, grid, dim3(256), s, ev0, ev1, r, n_q, c.n_kv, kc, vc, c.g, layer, part, mch, ch, out, out_t, qs);
    };
    switch (MQ) {
        case 1: go(k_attn_mfma<D, 1, PAGED>); break;
        case 2: go(k_attn_mfma<D, 2, PAGED>); break;
        case 3: go(k_attn_mfma<D, 3, PAGED>); break;
        default: go(k_attn_mfma<D, 4, PAGED>); break;
    }
}

template <typename T, int D>
static attn_split attn_t(const rows_t& r, const float* q, int n_q, const cache_t& c, int layer, float* part,
                         int max_chunks, void* out, act_t out_t, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1,
                         qkv_src qs)
{
    if constexpr (sizeof(T) == 2) {
        // bf16 cache: MFMA kernel.  max_chunks (the partial buffer's chunk
        // capacity) counts chunks of attention_chunk() <= ATT_MIN_CHUNK positions.
        const int QR = (n_q / c.n_kv) * r.n;
        const int MQ = QR > 48 ? 4 : (QR + 15) / 16;
        const int zs = (QR + 16 * MQ - 1) / (16 * MQ);
        const int per_chunk = r.B * c.n_kv * zs;                       // work-groups per chunk index
        const int want = (ATT_TARGET_WGS + per_chunk - 1) / per_chunk;   // chunks per sequence at capacity
        int ch = (r.max_ctx + want - 1) / want;
        ch = ((ch > ATT_MIN_CHUNK ? ch : ATT_MIN_CHUNK) + 31) & ~31;
        int mch = (r.max_ctx + ch - 1) / ch;
        if (mch > max_chunks) {                                          // cannot happen for ch >= attention_chunk()
            mch = max_chunks;
            ch = ((r.max_ctx + mch - 1) / mch + 31) & ~31;
        }
        dim3 grid(r.B * c.n_kv, mch, zs);
        // one chunk per sequence: the kernel writes the final output itself
        void* o = mch == 1 ? out : nullptr;
        if (c.g.bt) attn_mfma_launch<D, true>(MQ, grid, s, ev0, ev1, r, n_q, c, layer, part, mch, ch, o, out_t, qs);
        else attn_mfma_launch<D, false>(MQ, grid, s, ev0, ev1, r, n_q, c, layer, part, mch, ch, o, out_t, qs);
        return attn_split{mch, ch, o != nullptr};
    } else {
        dim3 grid(r.B * c.n_kv, max_chunks);
        launch_ev(k_attn_partial<T, D>, grid, dim3(256), s, ev0, ev1, r, q, n_q, c.n_kv, (const T*)c.k, (const T*)c.v,
                  c.g, layer, part, max_chunks);
        return attn_split{max_chunks, ATT_CH, false};
    }
}

attn_split launch_attention(const rows_t& r, qkv_src qs, float* q, int n_q, const cache_t& c, int layer, float* part,
                            int max_chunks, void* out, act_t out_t, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1)
{
    // the fp32 cache's kernel reads rotated queries: k_rope_kv writes them (and the new K/V rows) first
    if (c.kv_f32) launch_rope_kv(r, qs.qkv, qs.P, qs.S, qs.rope, n_q, c, layer, q, s);
    if (c.head_dim == 128) {
        if (c.kv_f32) return attn_t<float, 128>(r, q, n_q, c, layer, part, max_chunks, out, out_t, s, ev0, ev1, qs);
        return attn_t<uint16_t, 128>(r, q, n_q, c, layer, part, max_chunks, out, out_t, s, ev0, ev1, qs);
    }
    if (c.kv_f32) return attn_t<float, 64>(r, q, n_q, c, layer, part, max_chunks, out, out_t, s, ev0, ev1, qs);
    return attn_t<uint16_t, 64>(r, q, n_q, c, layer, part, max_chunks, out, out_t, s, ev0, ev1, qs);
}

void launch_attention_combine(const rows_t& r, int n_q, int head_dim, const float* part, attn_split sp, void* out,
                              act_t out_t, hipStream_t s)
{
    const int R = r.B * r.n, D = head_dim;
    if (out_t == ACT_F32) k_attn_combine<float><<<R * n_q, D, 0, s>>>(r, n_q, D, part, sp.chunks, sp.chunk, out);
    else if (out_t == ACT_BF16) k_attn_combine<uint16_t><<<R * n_q, D, 0, s>>>(r, n_q, D, part, sp.chunks, sp.chunk, out);
    else k_attn_combine<_Float16><<<R * n_q, D, 0, s>>>(r, n_q, D, part, sp.chunks, sp.chunk, out);
}

void launch_silu_mul(const float* gu, const float* P, int S, int R, int F, void* out, act_t out_t, hipStream_t s)
{
    dim3 grid(R, (F / 4 + 255) / 256);
    if (out_t == ACT_F32) k_silu_mul<float><<<grid, 256, 0, s>>>(gu, P, S, R, F, out);
    else if (out_t == ACT_BF16) k_silu_mul<uint16_t><<<grid, 256, 0, s>>>(gu, P, S, R, F, out);
    else k_silu_mul<_Float16><<<grid, 256, 0, s>>>(gu, P, S, R, F, out);
}

void launch_kv_advance(int B, const int32_t* slots, const int32_t* inc, int inc_const, int32_t* kv_len,
                       int max_slots, uint32_t* err, hipStream_t s)
{
    k_kv_advance<<<(B + 255) / 256, 256, 0, s>>>(B, slots, inc, inc_const, kv_len, max_slots, err);
}

void launch_prefill_lim(int B, const int32_t* len, int t0, int nc, int ld, int32_t* lim, uint32_t* err, hipStream_t s)
{
    k_prefill_lim<<<(B + 255) / 256, 256, 0, s>>>(B, len, t0, nc, ld, lim, err);
}

void launch_kv_poison(int B, const int32_t* slots, const int32_t* kv_len, int span, const cache_t& c,
                      int n_layers, int max_slots, int max_ctx, hipStream_t s)
{
    if (c.kv_f32)
        k_kv_poison<float><<<B, 256, 0, s>>>(slots, kv_len, span, (float*)c.k, (float*)c.v, c.g, n_layers, c.n_kv,
                                             c.head_dim, max_slots, max_ctx);
    else
        k_kv_poison<uint16_t><<<B, 256, 0, s>>>(slots, kv_len, span, (uint16_t*)c.k, (uint16_t*)c.v, c.g, n_layers,
                                                c.n_kv, c.head_dim, max_slots, max_ctx);
}
