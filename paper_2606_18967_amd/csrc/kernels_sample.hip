// kernels_sample.hip -- draft/AR sampling and speculative rejection sampling.
//
// Randomness: Philox-4x64-10 (Salmon et al., SC'11), key = (seed, step),
// counter = (block, position, slot, stream).  Each call yields four 64-bit
// words = eight uniforms (low 32-bit half first); a 32-bit half h maps to
// ((h >> 9) + 0.5) * 2^-23 in (0, 1).  Uniform i of a row is output i % 8 of
// block i / 8.
//
// Sampling x ~ softmax(l/T) is an exponential race (Gumbel-max):
// x = argmax_i [l_i/T - ln(-ln u_i)], ties to the lowest index.  The same pass
// yields max and log-sum-exp of l/T.
//
// Acceptance (the chain speculative sampling rule the paper builds on,
// Sec. 3.1 and App. D.1): d_j is accepted iff u_j <= p_j(d_j)/q_j(d_j); at the
// first rejection a token is drawn from norm(max(0, p_j - q_j)) (from p_j if
// that vanishes); if all gamma drafts pass, a bonus token is drawn from
// p_{gamma+1}.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int SCHUNK = 4096;            // vocabulary entries per work-group
constexpr int STHREADS = 256;
static_assert(SCHUNK % (8 * STHREADS) == 0, "a chunk is whole Philox blocks per thread");

struct philox_out { uint64_t w[4]; };

__device__ __forceinline__ philox_out philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                    uint64_t k0, uint64_t k1)
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        uint64_t lo0 = M0 * c0, hi0 = __umul64hi(M0, c0);
        uint64_t lo1 = M1 * c2, hi1 = __umul64hi(M1, c2);
        uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
        k0 += W0; k1 += W1;
    }
    philox_out o;
    o.w[0] = c0; o.w[1] = c1; o.w[2] = c2; o.w[3] = c3;
    return o;
}

__device__ __forceinline__ float u_of(uint32_t h) { return ((float)(h >> 9) + 0.5f) * (1.0f / 8388608.0f); }

__device__ __forceinline__ float uniform_at(rng_t rng, int stream, int slot, int pos, int idx)
{
    philox_out o = philox4x64_10((uint64_t)(idx >> 3), (uint64_t)(uint32_t)pos, (uint64_t)(uint32_t)slot,
                                 (uint64_t)stream, rng.seed, rng.step);
    uint64_t w = o.w[(idx & 7) >> 1];
    return u_of((idx & 1) ? (uint32_t)(w >> 32) : (uint32_t)w);
}

__device__ __forceinline__ float gumbel(float u) { return -logf(-logf(u)); }

// better (key, idx): larger key, ties to the lower index
__device__ __forceinline__ bool better(float ka, int ia, float kb, int ib)
{
    return ka > kb || (ka == kb && ia < ib);
}

struct race_t { float m, s, key; int idx; };

__device__ __forceinline__ void race_merge(race_t& a, const race_t& b)
{
    float m = fmaxf(a.m, b.m);
    float s = (a.s > 0.f ? a.s * __expf(a.m - m) : 0.f) + (b.s > 0.f ? b.s * __expf(b.m - m) : 0.f);
    a.m = m; a.s = s;
    if (better(b.key, b.idx, a.key, a.idx)) { a.key = b.key; a.idx = b.idx; }
}

__device__ race_t block_race(race_t v, race_t* sh)
{
    int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        race_t t;
        t.m = __shfl_xor(v.m, o, WAVE); t.s = __shfl_xor(v.s, o, WAVE);
        t.key = __shfl_xor(v.key, o, WAVE); t.idx = __shfl_xor(v.idx, o, WAVE);
        race_merge(v, t);
    }
    if (lane == 0) sh[w] = v;
    __syncthreads();
    race_t r = sh[0];
    for (int i = 1; i < (int)(blockDim.x >> 6); ++i) race_merge(r, sh[i]);
    return r;
}

// ------------------------------------------------------------------ token sampler
// partial[row][chunk] = (max, sumexp relative to max, best key, best idx)
__global__ void __launch_bounds__(STHREADS) k_sample_partial(rows_t r, const float* logits, long ld, int V,
                                                             float invT, rng_t rng, int pos_off, float* part,
                                                             int nch)
{
    __shared__ race_t sh[STHREADS / 64];
    int b = blockIdx.x, ch = blockIdx.y;
    int slot = r.slots[b];
    bool ok = slot >= 0 && slot < r.max_slots;
    int pos = ok ? r.kv_len[slot] + pos_off : 0;
    const float* lr = logits + (size_t)b * ld;
    // the thread's Philox blocks (8 consecutive entries each) in registers,
    // 16-byte loads where a block is whole and aligned; then max, sum of
    // exponentials and the race, with no data-dependent branch on the values
    constexpr int NB = SCHUNK / 8 / STHREADS;
    const int i0 = ch * SCHUNK;
    const bool vec = ((uintptr_t)lr & 15) == 0;
    float x[NB][8], key[NB][8];
#pragma unroll
    for (int bb = 0; bb < NB; ++bb) {
        const int blk = (i0 >> 3) + threadIdx.x + STHREADS * bb;
        const philox_out o = philox4x64_10((uint64_t)blk, (uint64_t)(uint32_t)pos, (uint64_t)(uint32_t)slot,
                                           (uint64_t)STREAM_TOKEN, rng.seed, rng.step);
        if (vec && blk * 8 + 8 <= V) {
            const float4 a = *(const float4*)(lr + blk * 8), c = *(const float4*)(lr + blk * 8 + 4);
            x[bb][0] = a.x; x[bb][1] = a.y; x[bb][2] = a.z; x[bb][3] = a.w;
            x[bb][4] = c.x; x[bb][5] = c.y; x[bb][6] = c.z; x[bb][7] = c.w;
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) x[bb][e] = blk * 8 + e < V ? lr[blk * 8 + e] : -INFINITY;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint64_t w = o.w[e >> 1];
            const float u = u_of((e & 1) ? (uint32_t)(w >> 32) : (uint32_t)w);
            const bool live = blk * 8 + e < V && blk * 8 + e < i0 + SCHUNK;
            x[bb][e] = live ? x[bb][e] * invT : -INFINITY;
            key[bb][e] = live ? x[bb][e] + gumbel(u) : -INFINITY;
        }
    }
    race_t v = {-INFINITY, 0.f, -INFINITY, 0x7fffffff};
#pragma unroll
    for (int bb = 0; bb < NB; ++bb)
#pragma unroll
        for (int e = 0; e < 8; ++e) v.m = fmaxf(v.m, x[bb][e]);
    if (v.m > -INFINITY) {
#pragma unroll
        for (int bb = 0; bb < NB; ++bb)
#pragma unroll
            for (int e = 0; e < 8; ++e) v.s += __expf(x[bb][e] - v.m);
    }
#pragma unroll
    for (int bb = 0; bb < NB; ++bb) {
        const int blk = (i0 >> 3) + threadIdx.x + STHREADS * bb;
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (better(key[bb][e], blk * 8 + e, v.key, v.idx)) { v.key = key[bb][e]; v.idx = blk * 8 + e; }
    }
    v = block_race(v, sh);
    if (threadIdx.x == 0) {
        float* p = part + ((size_t)b * nch + ch) * 4;
        p[0] = v.m; p[1] = v.s; p[2] = v.key; p[3] = __int_as_float(v.idx);
    }
}

// one wave per row: lane c merges chunks c, c + 64, ..., then a butterfly
__global__ void __launch_bounds__(64) k_sample_combine(rows_t r, const float* part, int nch, int32_t* tok,
                                                       int tok_stride, float* stats, int stats_stride)
{
    const int b = blockIdx.x, lane = threadIdx.x;
    const float* p = part + (size_t)b * nch * 4;
    race_t v = {-INFINITY, 0.f, -INFINITY, 0x7fffffff};
    for (int c = lane; c < nch; c += 64) {
        const race_t t = {p[c * 4], p[c * 4 + 1], p[c * 4 + 2], __float_as_int(p[c * 4 + 3])};
        race_merge(v, t);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        race_t t;
        t.m = __shfl_xor(v.m, o, WAVE); t.s = __shfl_xor(v.s, o, WAVE);
        t.key = __shfl_xor(v.key, o, WAVE); t.idx = __shfl_xor(v.idx, o, WAVE);
        race_merge(v, t);
    }
    if (lane == 0) {
        tok[(size_t)b * tok_stride] = v.idx;
        if (stats) {
            stats[(size_t)b * stats_stride] = v.m;
            stats[(size_t)b * stats_stride + 1] = v.m + logf(v.s);
        }
    }
}

// ------------------------------------------------------------------ row statistics
// partial (max, sumexp) of logits/T for rows of a [rows][V] block
// Each thread holds its SCHUNK / STHREADS entries in registers (16-byte loads
// when the chunk is whole and aligned), takes their max, then sums the
// exponentials with no data-dependent branch.
__global__ void __launch_bounds__(STHREADS) k_stats_partial(const float* logits, int V, float invT, float* part,
                                                            int nch)
{
    constexpr int PER = SCHUNK / STHREADS;
    __shared__ race_t sh[STHREADS / 64];
    const int row = blockIdx.x, ch = blockIdx.y;
    const float* lr = logits + (size_t)row * V;
    const int i0 = ch * SCHUNK;
    float x[PER];
    if (i0 + SCHUNK <= V && ((uintptr_t)(lr + i0) & 15) == 0) {
#pragma unroll
        for (int t = 0; t < PER / 4; ++t) {
            const float4 f = *(const float4*)(lr + i0 + 4 * (threadIdx.x + STHREADS * t));
            x[4 * t] = f.x * invT; x[4 * t + 1] = f.y * invT; x[4 * t + 2] = f.z * invT; x[4 * t + 3] = f.w * invT;
        }
    } else {
#pragma unroll
        for (int t = 0; t < PER; ++t) {
            const int i = i0 + threadIdx.x + STHREADS * t;
            x[t] = i < V ? lr[i] * invT : -INFINITY;
        }
    }
    float m = -INFINITY;
#pragma unroll
    for (int t = 0; t < PER; ++t) m = fmaxf(m, x[t]);
    float sum = 0.f;
    if (m > -INFINITY) {
#pragma unroll
        for (int t = 0; t < PER; ++t) sum += __expf(x[t] - m);
    }
    race_t v = {m, sum, -INFINITY, 0x7fffffff};
    v = block_race(v, sh);
    if (threadIdx.x == 0) { part[((size_t)row * nch + ch) * 2] = v.m; part[((size_t)row * nch + ch) * 2 + 1] = v.s; }
}

// work[b] = {mode (0 residual, 1 bonus), p row, lse_p, lse_q, position, n_emit}
constexpr int WK = 6;

// log-sum-exp of p row `row` from its chunk partials, reduced over one wave
// (lane c takes chunks c, c + 64, ...; the same butterfly order every time)
__device__ float wave_lse(const float* part, int row, int nch, int lane)
{
    const float* p = part + (size_t)row * nch * 2;
    float m = -INFINITY, s = 0.f;
    for (int c = lane; c < nch; c += 64) {
        const float mc = p[2 * c], sc = p[2 * c + 1];
        if (!(sc > 0.f)) continue;
        const float mn = fmaxf(m, mc);
        s = (s > 0.f ? s * __expf(m - mn) : 0.f) + sc * __expf(mc - mn);
        m = mn;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float mo = __shfl_xor(m, o, WAVE), so = __shfl_xor(s, o, WAVE);
        const float mn = fmaxf(m, mo);
        s = (s > 0.f ? s * __expf(m - mn) : 0.f) + (so > 0.f ? so * __expf(mo - mn) : 0.f);
        m = mn;
    }
    return m + logf(s);
}

// One wave per sequence.  Lane j - 1 tests draft j (j = 1..gamma) -- accept
// iff u_j <= p_j(d_j) / q_j(d_j) -- all at once; the first failing j is the
// rejection point (App. D.1).  work[b] then names the row of the final draw.
__global__ void __launch_bounds__(64) k_accept_decide(rows_t r, int gamma, int V, float invT, rng_t rng,
                                                      const int32_t* draft, const float* q_logits,
                                                      const float* q_stats, const float* p_logits,
                                                      const float* spart, int nch, int32_t* out_tok, int32_t* n_emit,
                                                      float* work)
{
    const int b = blockIdx.x, lane = threadIdx.x;
    const int slot = r.slots[b];
    float* wk = work + (size_t)b * WK;
    int32_t* ot = out_tok + (size_t)b * (gamma + 1);
    if (slot < 0 || slot >= r.max_slots) {
        if (lane == 0) {
            flag_error(r.err, ERR_SLOT);
            n_emit[b] = 0;
            wk[0] = -1.f;
        }
        for (int j = lane; j <= gamma; j += 64) ot[j] = -1;
        return;
    }
    const int kv = r.kv_len[slot];
    const int prow0 = b * (gamma + 1);
    // each lane t keeps the lse of p row t (t <= gamma); the bonus row's too
    float my_lse = 0.f, lse_bonus = 0.f;
    for (int t = 0; t <= gamma; ++t) {
        const float l = wave_lse(spart, prow0 + t, nch, lane);
        if (lane == t) my_lse = l;
        if (t == gamma) lse_bonus = l;
    }
    bool reject = false;
    int d = -1;
    if (lane < gamma) {
        const int j = lane + 1;
        d = draft[(size_t)b * gamma + lane];
        float ratio = 0.f;
        if (d >= 0 && d < V) {
            const float lp = p_logits[(size_t)(prow0 + lane) * V + d] * invT - my_lse;
            const float lq = q_logits[((size_t)b * gamma + lane) * V + d] * invT - q_stats[((size_t)b * gamma + lane) * 2 + 1];
            ratio = expf(lp - lq);
        } else {
            flag_error(r.err, ERR_TOKEN);
        }
        const float u = uniform_at(rng, STREAM_ACCEPT, slot, kv + j, 0);
        reject = !(u <= ratio);
    }
    const uint64_t rej = __builtin_amdgcn_ballot_w64(reject);
    const int jstar = rej ? (int)__builtin_ctzll(rej) + 1 : gamma + 1;
    const float lse_rej = __shfl(my_lse, (jstar - 1) & 63, WAVE);
    for (int t = lane; t <= gamma; t += 64) {
        if (t < jstar - 1) ot[t] = d;        // t < gamma here, so lane t holds d_t
        else if (t >= jstar) ot[t] = -1;
    }
    if (lane == 0) {
        if (jstar <= gamma) {
            wk[0] = 0.f; wk[1] = (float)(prow0 + jstar - 1); wk[2] = lse_rej;
            wk[3] = q_stats[((size_t)b * gamma + jstar - 1) * 2 + 1];
            wk[4] = (float)(kv + jstar);
        } else {
            wk[0] = 1.f; wk[1] = (float)(prow0 + gamma); wk[2] = lse_bonus; wk[3] = 0.f;
            wk[4] = (float)(kv + gamma + 1);
        }
        wk[5] = (float)jstar;
        n_emit[b] = jstar;
    }
}

// final draw: residual (mode 0) or bonus (mode 1); partial per (b, chunk) =
// (keyA, idxA, keyB, idxB) with A the residual race and B the race over p.
__global__ void __launch_bounds__(STHREADS) k_final_partial(rows_t r, int gamma, int V, float invT, rng_t rng,
                                                            const float* q_logits, const float* p_logits,
                                                            const float* work, float* part, int nch)
{
    __shared__ race_t sha[STHREADS / 64];
    __shared__ race_t shb[STHREADS / 64];
    int b = blockIdx.x, ch = blockIdx.y;
    const float* wk = work + (size_t)b * WK;
    if (wk[0] < 0.f) return;   // invalid slot
    int mode = (int)wk[0];
    int prow = (int)wk[1];
    float lsep = wk[2], lseq = wk[3];
    int pos = (int)wk[4];
    int jstar = (int)wk[5];
    int slot = r.slots[b];
    const float* lp = p_logits + (size_t)prow * V;
    const float* lq = q_logits + ((size_t)b * gamma + min(jstar, gamma) - 1) * V;   // read in mode 0 only
    int stream = mode == 0 ? STREAM_RESIDUAL : STREAM_TOKEN;
    // the thread's Philox blocks in registers (16-byte loads where a block is
    // whole and aligned), then both races; the mode is uniform per work-group
    constexpr int NB = SCHUNK / 8 / STHREADS;
    const int i0 = ch * SCHUNK;
    const bool vec = (((uintptr_t)lp | (uintptr_t)lq) & 15) == 0;
    float xp[NB][8], xq[NB][8];
#pragma unroll
    for (int bb = 0; bb < NB; ++bb) {
        const int base = ((i0 >> 3) + threadIdx.x + STHREADS * bb) * 8;
        if (vec && base + 8 <= V) {
            const float4 a = *(const float4*)(lp + base), c = *(const float4*)(lp + base + 4);
            xp[bb][0] = a.x; xp[bb][1] = a.y; xp[bb][2] = a.z; xp[bb][3] = a.w;
            xp[bb][4] = c.x; xp[bb][5] = c.y; xp[bb][6] = c.z; xp[bb][7] = c.w;
            if (mode == 0) {
                const float4 d = *(const float4*)(lq + base), f = *(const float4*)(lq + base + 4);
                xq[bb][0] = d.x; xq[bb][1] = d.y; xq[bb][2] = d.z; xq[bb][3] = d.w;
                xq[bb][4] = f.x; xq[bb][5] = f.y; xq[bb][6] = f.z; xq[bb][7] = f.w;
            }
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                xp[bb][e] = base + e < V ? lp[base + e] : 0.f;
                if (mode == 0) xq[bb][e] = base + e < V ? lq[base + e] : 0.f;
            }
        }
    }
    race_t va = {0.f, 0.f, -INFINITY, 0x7fffffff}, vb = va;
#pragma unroll
    for (int bb = 0; bb < NB; ++bb) {
        const int blk = (i0 >> 3) + threadIdx.x + STHREADS * bb;
        const philox_out o = philox4x64_10((uint64_t)blk, (uint64_t)(uint32_t)pos, (uint64_t)(uint32_t)slot,
                                           (uint64_t)stream, rng.seed, rng.step);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int i = blk * 8 + e;
            const uint64_t w = o.w[e >> 1];
            const float g = gumbel(u_of((e & 1) ? (uint32_t)(w >> 32) : (uint32_t)w));
            const float x = xp[bb][e] * invT;
            const float kb = i < V ? x + g : -INFINITY;
            float ka = kb;
            if (mode == 0) {
                const float rr = expf(x - lsep) - expf(xq[bb][e] * invT - lseq);
                ka = rr > 0.f && i < V ? logf(rr) + g : -INFINITY;
            }
            if (better(ka, i, va.key, va.idx)) { va.key = ka; va.idx = i; }
            if (better(kb, i, vb.key, vb.idx)) { vb.key = kb; vb.idx = i; }
        }
    }
    va = block_race(va, sha);
    vb = block_race(vb, shb);
    if (threadIdx.x == 0) {
        float* p = part + ((size_t)b * nch + ch) * 4;
        p[0] = va.key; p[1] = __int_as_float(va.idx); p[2] = vb.key; p[3] = __int_as_float(vb.idx);
    }
}

// one wave per sequence, as k_sample_combine
__global__ void __launch_bounds__(64) k_final_combine(int gamma, const float* work, const float* part, int nch,
                                                      int32_t* out_tok, int32_t* next_tok)
{
    const int b = blockIdx.x, lane = threadIdx.x;
    const float* wk = work + (size_t)b * WK;
    if (wk[0] < 0.f) {
        if (next_tok && lane == 0) next_tok[b] = -1;
        return;
    }
    const float* p = part + (size_t)b * nch * 4;
    float ka = -INFINITY, kb = -INFINITY;
    int ia = 0x7fffffff, ib = 0x7fffffff;
    for (int c = lane; c < nch; c += 64) {
        float k = p[c * 4]; int i = __float_as_int(p[c * 4 + 1]);
        if (better(k, i, ka, ia)) { ka = k; ia = i; }
        k = p[c * 4 + 2]; i = __float_as_int(p[c * 4 + 3]);
        if (better(k, i, kb, ib)) { kb = k; ib = i; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        float k = __shfl_xor(ka, o, WAVE); int i = __shfl_xor(ia, o, WAVE);
        if (better(k, i, ka, ia)) { ka = k; ia = i; }
        k = __shfl_xor(kb, o, WAVE); i = __shfl_xor(ib, o, WAVE);
        if (better(k, i, kb, ib)) { kb = k; ib = i; }
    }
    if (lane == 0) {
        const int y = ka > -INFINITY ? ia : ib;
        const int jstar = (int)wk[5];
        out_tok[(size_t)b * (gamma + 1) + jstar - 1] = y;
        if (next_tok) next_tok[b] = y;
    }
}

}  // namespace

int sample_chunks(int V) { return (V + SCHUNK - 1) / SCHUNK; }

size_t sample_part_floats(int rows, int V) { return (size_t)rows * sample_chunks(V) * 4; }

size_t accept_work_floats(int B, int gamma) { (void)gamma; return (size_t)B * WK; }

// launch_accept's part: (max, sumexp) per (p row, chunk), then the final
// draw's (keyA, idxA, keyB, idxB) per (sequence, chunk)
size_t accept_part_floats(int B, int gamma, int V)
{
    const size_t nch = (size_t)sample_chunks(V);
    return (size_t)B * (gamma + 1) * nch * 2 + (size_t)B * nch * 4;
}

void launch_sample(const rows_t& r, const float* logits, long ld, int V, float T, rng_t rng, int pos_off,
                   int32_t* tok, int tok_stride, float* stats, int stats_stride, float* part, hipStream_t s)
{
    int nch = sample_chunks(V);
    k_sample_partial<<<dim3(r.B, nch), STHREADS, 0, s>>>(r, logits, ld, V, 1.0f / T, rng, pos_off, part, nch);
    k_sample_combine<<<r.B, 64, 0, s>>>(r, part, nch, tok, tok_stride, stats, stats_stride);
}

void launch_accept(const rows_t& r, int gamma, int V, float T, rng_t rng, const int32_t* draft,
                   const float* q_logits, const float* q_stats, const float* p_logits, int32_t* out_tok,
                   int32_t* n_emit, int32_t* next_tok, float* part, float* work, hipStream_t s)
{
    int nch = sample_chunks(V);
    float invT = 1.0f / T;
    int prows = r.B * (gamma + 1);
    k_stats_partial<<<dim3(prows, nch), STHREADS, 0, s>>>(p_logits, V, invT, part, nch);
    k_accept_decide<<<r.B, 64, 0, s>>>(r, gamma, V, invT, rng, draft, q_logits, q_stats, p_logits, part, nch, out_tok,
                                       n_emit, work);
    float* fpart = part + (size_t)prows * nch * 2;
    k_final_partial<<<dim3(r.B, nch), STHREADS, 0, s>>>(r, gamma, V, invT, rng, q_logits, p_logits, work, fpart, nch);
    k_final_combine<<<r.B, 64, 0, s>>>(gamma, work, fpart, nch, out_tok, next_tok);
}
