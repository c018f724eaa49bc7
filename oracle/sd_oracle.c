/*
 * sd_oracle.c -- plain CPU oracle for quantized self-speculative decoding.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, the smoke check and the CPU-baseline
 * leg of the benchmark may load this library.  The product path (the HIP
 * library under paper_2606_18967_amd/) shares no source with it and never
 * calls it.
 *
 * Everything here is deliberately slow and direct:
 *   - model arithmetic (norms, projections, RoPE, attention, SwiGLU, LM head)
 *     is done in double precision, one token at a time, in the order the
 *     definitions are written;
 *   - decisions that turn floating point into integers (RTN codes, the
 *     exponential-race argmax, the accept test) are taken in fp32, the
 *     precision the device path takes them in;
 *   - random numbers come from Philox-4x64-10 (Salmon et al., SC'11), written
 *     from its published definition.
 *
 * Paper references: "EfficientRollout: System-Aware Self-Speculative Decoding
 * for RL Rollouts".  Sections are cited by number and label.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_API __attribute__((visibility("default")))

/* ------------------------------------------------------------------------ */
/* fp16 / bf16 scalar conversions (IEEE binary16 round-to-nearest-even).     */
/* ------------------------------------------------------------------------ */

static uint32_t f32_bits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float bits_f32(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* float -> binary16 bits, round to nearest even, with subnormals, inf, NaN. */
OR_API uint16_t or_f32_to_f16(float f)
{
    uint32_t x = f32_bits(f);
    uint16_t sign = (uint16_t)((x >> 16) & 0x8000u);
    uint32_t ax = x & 0x7fffffffu;
    if (ax >= 0x7f800000u) /* inf or NaN */
        return (uint16_t)(sign | 0x7c00u | (ax > 0x7f800000u ? 0x200u : 0u));
    /* Work with the exact value |f| = m * 2^e, then round to a multiple of
       the binary16 quantum for its binade. */
    double a = (double)bits_f32(ax);
    if (a == 0.0) return sign;
    int e;
    frexp(a, &e);                  /* a in [2^(e-1), 2^e) */
    int exp16 = e - 1;             /* unbiased exponent of a */
    if (exp16 < -14) exp16 = -14;  /* subnormal range shares the quantum 2^-24 */
    double quantum = ldexp(1.0, exp16 - 10);
    double q = a / quantum;        /* exact: a has <= 24 significant bits */
    double r = nearbyint(q);       /* default rounding mode: to nearest even */
    double v = r * quantum;
    if (v >= 65520.0) return (uint16_t)(sign | 0x7c00u); /* overflow to inf */
    /* encode v (exact binary16 value) */
    if (v < ldexp(1.0, -14)) {     /* subnormal */
        uint32_t mant = (uint32_t)(v / ldexp(1.0, -24));
        return (uint16_t)(sign | mant);
    }
    int ev;
    double fr = frexp(v, &ev);     /* v = fr * 2^ev, fr in [0.5,1) */
    uint32_t biased = (uint32_t)(ev - 1 + 15);
    uint32_t mant = (uint32_t)((fr * 2.0 - 1.0) * 1024.0);
    return (uint16_t)(sign | (biased << 10) | mant);
}

OR_API float or_f16_to_f32(uint16_t h)
{
    uint32_t sign = (h & 0x8000u) ? 1u : 0u;
    uint32_t ex = (h >> 10) & 0x1fu, mant = h & 0x3ffu;
    double v;
    if (ex == 0) v = ldexp((double)mant, -24);
    else if (ex == 31) v = mant ? NAN : INFINITY;
    else v = ldexp(1.0 + mant / 1024.0, (int)ex - 15);
    return (float)(sign ? -v : v);
}

static double bf16_to_f64(uint16_t b) { return (double)bits_f32(((uint32_t)b) << 16); }

/* ------------------------------------------------------------------------ */
/* Philox-4x64-10 and the uniform mapping.                                   */
/* ------------------------------------------------------------------------ */

OR_API void or_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    /* Round multipliers and Weyl key increments from Salmon et al. (2011). */
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
    uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        __uint128_t p0 = (__uint128_t)M0 * x0;
        __uint128_t p1 = (__uint128_t)M1 * x2;
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        uint64_t n0 = hi1 ^ x1 ^ k0;
        uint64_t n1 = lo1;
        uint64_t n2 = hi0 ^ x3 ^ k1;
        uint64_t n3 = lo0;
        x0 = n0; x1 = n1; x2 = n2; x3 = n3;
        k0 += W0; k1 += W1;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* Random streams (the last counter word). */
enum { OR_STREAM_TOKEN = 0, OR_STREAM_ACCEPT = 1, OR_STREAM_RESIDUAL = 2 };

/* The idx-th uniform of the row addressed by (stream, slot, pos):
   counter = (idx / 8, pos, slot, stream), key = (seed, step).  Output word
   w = (idx % 8) / 2 gives two uniforms, its low 32-bit half first.  A 32-bit
   half h maps to ((h >> 9) + 0.5) * 2^-23, which lies in (0, 1) and is exact
   in fp32. */
OR_API float or_uniform(uint64_t seed, uint64_t step, uint32_t stream,
                        uint32_t slot, uint32_t pos, uint32_t idx)
{
    uint64_t ctr[4] = { idx / 8u, pos, slot, stream };
    uint64_t key[2] = { seed, step };
    uint64_t out[4];
    or_philox4x64_10(ctr, key, out);
    uint64_t word = out[(idx % 8u) / 2u];
    uint32_t half = (idx % 2u) ? (uint32_t)(word >> 32) : (uint32_t)word;
    return ((float)(half >> 9) + 0.5f) * (1.0f / 8388608.0f);
}

/* Fill u[0..n) with the uniforms of one row (same mapping as or_uniform,
   one generator call per block of eight). */
OR_API void or_uniform_row(uint64_t seed, uint64_t step, uint32_t stream,
                           uint32_t slot, uint32_t pos, int n, float* u)
{
    uint64_t key[2] = { seed, step };
    for (int b = 0; 8 * b < n; ++b) {
        uint64_t ctr[4] = { (uint64_t)b, pos, slot, stream };
        uint64_t out[4];
        or_philox4x64_10(ctr, key, out);
        for (int e = 0; e < 8 && 8 * b + e < n; ++e) {
            uint64_t word = out[e / 2];
            uint32_t half = (e % 2) ? (uint32_t)(word >> 32) : (uint32_t)word;
            u[8 * b + e] = ((float)(half >> 9) + 0.5f) * (1.0f / 8388608.0f);
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Softmax statistics and the exponential-race sampler.                      */
/* Sampling x ~ softmax(l / T): by the Gumbel-max theorem,                   */
/*   x = argmax_i [ l_i / T - ln(-ln u_i) ],  u_i iid uniform(0,1).          */
/* Ties go to the lowest index.  Keys are formed in fp32.                    */
/* ------------------------------------------------------------------------ */

/* lse of the scaled row x_i = l_i * (1/T); returned as float, computed in
   double.  Also returns the max. */
OR_API void or_row_stats(const float* l, int V, float T, float* m_out, float* lse_out)
{
    float invT = 1.0f / T;
    double m = -INFINITY;
    for (int i = 0; i < V; ++i) { double x = (double)(l[i] * invT); if (x > m) m = x; }
    double s = 0.0;
    for (int i = 0; i < V; ++i) s += exp((double)(l[i] * invT) - m);
    *m_out = (float)m;
    *lse_out = (float)(m + log(s));
}

/* One draw by exponential race over the row, uniforms from (stream, slot,
   pos).  Returns the index; *gap_out gets the difference between the two
   largest keys (used by tests to spot near-ties). */
static int race_argmax(const float* key, int V, float* gap_out)
{
    int best = -1;
    float k1 = -INFINITY, k2 = -INFINITY;
    for (int i = 0; i < V; ++i) {
        float k = key[i];
        if (best < 0 || k > k1) { k2 = k1; k1 = k; best = i; }
        else if (k > k2) k2 = k;
    }
    if (gap_out) *gap_out = k1 - k2;
    return best;
}

OR_API int or_sample_row(const float* l, int V, float T, uint64_t seed, uint64_t step,
                         uint32_t stream, uint32_t slot, uint32_t pos, float* gap_out)
{
    float invT = 1.0f / T;
    float* key = (float*)malloc(sizeof(float) * (size_t)V);
    or_uniform_row(seed, step, stream, slot, pos, V, key);
    for (int i = 0; i < V; ++i) {
        float g = -logf(-logf(key[i]));
        key[i] = l[i] * invT + g;
    }
    int x = race_argmax(key, V, gap_out);
    free(key);
    return x;
}

/* ------------------------------------------------------------------------ */
/* Speculative rejection sampling for one sequence (Sec. 3.1 and App. D.1;   */
/* the chain rule of Leviathan et al. that the paper builds on).             */
/*                                                                           */
/*   p_j = softmax(lp_{j-1} / T)  (verify rows 0..gamma),                    */
/*   q_j = softmax(lq_j / T)      (draft rows 1..gamma, row j at j-1).       */
/*   for j = 1..gamma: accept d_j iff u^A_j <= p_j(d_j) / q_j(d_j).          */
/*   first rejection j*: emit y ~ norm(max(0, p_j* - q_j*)) (RESIDUAL        */
/*   stream); if no entry is positive, y ~ p_j* instead.                     */
/*   all accepted: emit a bonus y ~ p_{gamma+1} (TOKEN stream).              */
/* Positions: last token at kv_len; the j-th new token sits at kv_len + j.   */
/* Outputs: out_tok[0..n_emit), n_emit in [1, gamma+1].  Diagnostics (may be */
/* NULL): ratio[j-1] and u_acc[j-1] for each examined j (others NaN), and    */
/* the key gap of the final draw.                                            */
/* ------------------------------------------------------------------------ */

OR_API int or_accept_seq(int V, int gamma, float T,
                         const int32_t* draft_tok,  /* [gamma] */
                         const float* q_logits,     /* [gamma][V] */
                         const float* p_logits,     /* [gamma+1][V] */
                         uint64_t seed, uint64_t step, uint32_t slot, uint32_t kv_len,
                         int32_t* out_tok,          /* [gamma+1] */
                         float* ratio_out, float* u_out, float* gap_out)
{
    float invT = 1.0f / T;
    for (int j = 0; j < gamma; ++j) {
        if (ratio_out) ratio_out[j] = NAN;
        if (u_out) u_out[j] = NAN;
    }
    for (int j = 1; j <= gamma; ++j) {
        const float* lp = p_logits + (size_t)(j - 1) * V;
        const float* lq = q_logits + (size_t)(j - 1) * V;
        float mp, lsep, mq, lseq;
        or_row_stats(lp, V, T, &mp, &lsep);
        or_row_stats(lq, V, T, &mq, &lseq);
        int d = draft_tok[j - 1];
        float logp = lp[d] * invT - lsep;
        float logq = lq[d] * invT - lseq;
        float ratio = expf(logp - logq);
        uint32_t pos = kv_len + (uint32_t)j;
        float u = or_uniform(seed, step, OR_STREAM_ACCEPT, slot, pos, 0);
        if (ratio_out) ratio_out[j - 1] = ratio;
        if (u_out) u_out[j - 1] = u;
        if (u <= ratio) { out_tok[j - 1] = d; continue; }
        /* rejected at j: residual resample */
        float* key = (float*)malloc(sizeof(float) * (size_t)V);
        float* ur = (float*)malloc(sizeof(float) * (size_t)V);
        or_uniform_row(seed, step, OR_STREAM_RESIDUAL, slot, pos, V, ur);
        int any = 0;
        for (int i = 0; i < V; ++i) {
            float pi = expf(lp[i] * invT - lsep);
            float qi = expf(lq[i] * invT - lseq);
            float r = pi - qi;
            float g = -logf(-logf(ur[i]));
            if (r > 0.0f) { key[i] = logf(r) + g; any = 1; }
            else key[i] = -INFINITY;
        }
        if (!any) /* residual vanished numerically: draw from p_j */
            for (int i = 0; i < V; ++i) key[i] = lp[i] * invT - logf(-logf(ur[i]));
        out_tok[j - 1] = race_argmax(key, V, gap_out);
        free(key);
        free(ur);
        return j;
    }
    /* all accepted: bonus token from p_{gamma+1} */
    uint32_t pos = kv_len + (uint32_t)gamma + 1u;
    out_tok[gamma] = or_sample_row(p_logits + (size_t)gamma * V, V, T, seed, step,
                                   OR_STREAM_TOKEN, slot, pos, gap_out);
    return gamma + 1;
}

/* ------------------------------------------------------------------------ */
/* RTN weight quantization (Sec. 4.1; App. B.2 names the RTN form).          */
/* Symmetric int4 with groups of `group` consecutive weights along K within  */
/* each output row, binary16 scales:                                         */
/*   s = fp16(max|w_g| / 7),  q = clamp(rint(w / s), -8, 7),  w^ = s * q;    */
/*   s = 0 and q = 0 for an all-zero group.  fp32 arithmetic, RNE.           */
/* Also the asymmetric variant the paper mentions:                          */
/*   s = fp16((max - min) / 15), z = clamp(rint(-min / s), 0, 15),           */
/*   q = clamp(rint(w / s) + z, 0, 15), w^ = s * (q - z).                    */
/* And the 8-bit drafter of the W4-versus-W8 comparison (App. B.3, Table 4), */
/* symmetric like the 4-bit default:                                         */
/*   s = fp16(max|w_g| / 127), q = clamp(rint(w / s), -128, 127).            */
/* ------------------------------------------------------------------------ */

OR_API void or_quantize_rtn4(const float* w, int N, int K, int group,
                             int8_t* codes /* [N][K] */, uint16_t* scales /* [N][K/group] */)
{
    int G = K / group;
    for (int n = 0; n < N; ++n)
        for (int g = 0; g < G; ++g) {
            const float* wg = w + (size_t)n * K + (size_t)g * group;
            float amax = 0.0f;
            for (int i = 0; i < group; ++i) { float a = fabsf(wg[i]); if (a > amax) amax = a; }
            uint16_t sh = or_f32_to_f16(amax / 7.0f);
            float s = or_f16_to_f32(sh);
            scales[(size_t)n * G + g] = sh;
            int8_t* cg = codes + (size_t)n * K + (size_t)g * group;
            for (int i = 0; i < group; ++i) {
                int q = 0;
                if (s != 0.0f) {
                    float r = rintf(wg[i] / s);
                    q = r < -8.0f ? -8 : (r > 7.0f ? 7 : (int)r);
                }
                cg[i] = (int8_t)q;
            }
        }
}

OR_API void or_quantize_rtn4_asym(const float* w, int N, int K, int group,
                                  uint8_t* codes, uint16_t* scales, uint8_t* zeros)
{
    int G = K / group;
    for (int n = 0; n < N; ++n)
        for (int g = 0; g < G; ++g) {
            const float* wg = w + (size_t)n * K + (size_t)g * group;
            float lo = wg[0], hi = wg[0];
            for (int i = 1; i < group; ++i) { if (wg[i] < lo) lo = wg[i]; if (wg[i] > hi) hi = wg[i]; }
            uint16_t sh = or_f32_to_f16((hi - lo) / 15.0f);
            float s = or_f16_to_f32(sh);
            int z = 0;
            if (s != 0.0f) { float zr = rintf(-lo / s); z = zr < 0.0f ? 0 : (zr > 15.0f ? 15 : (int)zr); }
            scales[(size_t)n * G + g] = sh;
            zeros[(size_t)n * G + g] = (uint8_t)z;
            uint8_t* cg = codes + (size_t)n * K + (size_t)g * group;
            for (int i = 0; i < group; ++i) {
                int q = z;
                if (s != 0.0f) {
                    float r = rintf(wg[i] / s) + (float)z;
                    q = r < 0.0f ? 0 : (r > 15.0f ? 15 : (int)r);
                }
                cg[i] = (uint8_t)q;
            }
        }
}

OR_API void or_quantize_rtn8(const float* w, int N, int K, int group,
                             int8_t* codes /* [N][K] */, uint16_t* scales /* [N][K/group] */)
{
    int G = K / group;
    for (int n = 0; n < N; ++n)
        for (int g = 0; g < G; ++g) {
            const float* wg = w + (size_t)n * K + (size_t)g * group;
            float amax = 0.0f;
            for (int i = 0; i < group; ++i) { float a = fabsf(wg[i]); if (a > amax) amax = a; }
            uint16_t sh = or_f32_to_f16(amax / 127.0f);
            float s = or_f16_to_f32(sh);
            scales[(size_t)n * G + g] = sh;
            int8_t* cg = codes + (size_t)n * K + (size_t)g * group;
            for (int i = 0; i < group; ++i) {
                int q = 0;
                if (s != 0.0f) {
                    float r = rintf(wg[i] / s);
                    q = r < -128.0f ? -128 : (r > 127.0f ? 127 : (int)r);
                }
                cg[i] = (int8_t)q;
            }
        }
}

/* ------------------------------------------------------------------------ */
/* Decoder forward (Llama-style, the architecture the workloads use):        */
/*   a = RMSNorm(h) * g1;  q,k,v = a Wq^T, a Wk^T, a Wv^T;                  */
/*   RoPE (rotate-half) on q and k at the absolute position;                 */
/*   K,V written at that position; head i reads KV head floor(i*nkv/nq);     */
/*   softmax(q k^T / sqrt(d)) over positions [0, pos];  h += attn Wo^T;      */
/*   b = RMSNorm(h) * g2;  h += (SiLU(b Wg^T) * (b Wu^T)) Wd^T;             */
/*   logits = (RMSNorm(h) * gf) Wlm^T.                                       */
/* The drafter is the same network with Wq,Wk,Wv,Wo,Wg,Wu,Wd replaced by     */
/* their RTN dequantized values (Sec. 4.1: embedding, norms and LM head stay */
/* high precision; App. D.2).                                                */
/* Fused storage convention of the inputs: Wqkv rows = [Wq; Wk; Wv],         */
/* Wgu rows = [Wg; Wu].                                                       */
/* ------------------------------------------------------------------------ */

enum { OR_F32 = 0, OR_BF16 = 1, OR_Q4 = 2 };

typedef struct {
    int n_layers, hidden, n_q, n_kv, head_dim, ffn, vocab;
    float rms_eps, rope_theta;
} or_cfg;

typedef struct {
    int kind, N, K, group;
    const void* w;          /* OR_F32: float[N][K]; OR_BF16: uint16[N][K] */
    const int8_t* codes;    /* OR_Q4: int8[N][K] */
    const uint16_t* scales; /* OR_Q4: fp16[N][K/group] */
    const uint8_t* zeros;   /* OR_Q4: zero points [N][K/group], or NULL (symmetric) */
} or_lin;

typedef struct {
    or_cfg c;
    int wkind;               /* OR_F32 or OR_BF16 for embed/norms/lm head */
    const void* embed;       /* [V][H] */
    const void* final_norm;  /* [H] */
    or_lin lm;               /* [V][H] */
    const void** attn_norm;  /* [L] -> [H] */
    const void** ffn_norm;   /* [L] -> [H] */
    or_lin* qkv;             /* [L] */
    or_lin* o;               /* [L] */
    or_lin* gu;              /* [L] */
    or_lin* dn;              /* [L] */
} or_model;

static double vec_at(int kind, const void* p, size_t i)
{
    return kind == OR_BF16 ? bf16_to_f64(((const uint16_t*)p)[i]) : (double)((const float*)p)[i];
}

/* Row n of W as doubles (the quantized kind dequantizes s * (q - z) group by
   group, z = 0 for the symmetric formats). */
static void lin_row(const or_lin* L, size_t n, double* wrow)
{
    size_t K = (size_t)L->K;
    if (L->kind == OR_Q4) {
        size_t G = K / (size_t)L->group;
        for (size_t g = 0; g < G; ++g) {
            double s = (double)or_f16_to_f32(L->scales[n * G + g]);
            double z = L->zeros ? (double)L->zeros[n * G + g] : 0.0;
            for (size_t k = g * L->group; k < (g + 1) * L->group; ++k) wrow[k] = s * ((double)L->codes[n * K + k] - z);
        }
    } else if (L->kind == OR_BF16) {
        for (size_t k = 0; k < K; ++k) wrow[k] = bf16_to_f64(((const uint16_t*)L->w)[n * K + k]);
    } else {
        for (size_t k = 0; k < K; ++k) wrow[k] = (double)((const float*)L->w)[n * K + k];
    }
}

/* y[r] = sum_k x[k] * W[row0 + r][k] for r in [0, n) */
static void lin_rows(const or_lin* L, int row0, int r0, int r1, const double* x, double* y, double* wrow)
{
    for (int r = r0; r < r1; ++r) {
        lin_row(L, (size_t)(row0 + r), wrow);
        double acc = 0.0;
        for (int k = 0; k < L->K; ++k) acc += x[k] * wrow[k];
        y[r] = acc;
    }
}

static void lin_apply(const or_lin* L, int row0, int n, const double* x, double* y)
{
    if ((long)n * L->K <= (1L << 18)) {   /* small: one thread */
        double* wrow = (double*)malloc(sizeof(double) * (size_t)L->K);
        lin_rows(L, row0, 0, n, x, y, wrow);
        free(wrow);
        return;
    }
#pragma omp parallel
    {
        double* wrow = (double*)malloc(sizeof(double) * (size_t)L->K);
#pragma omp for schedule(static)
        for (int r = 0; r < n; ++r) lin_rows(L, row0, r, r + 1, x, y, wrow);
        free(wrow);
    }
}

static void rmsnorm(const double* h, int H, int gkind, const void* g, double eps, double* out)
{
    double ss = 0.0;
    for (int i = 0; i < H; ++i) ss += h[i] * h[i];
    double inv = 1.0 / sqrt(ss / H + eps);
    for (int i = 0; i < H; ++i) out[i] = h[i] * inv * vec_at(gkind, g, (size_t)i);
}

static void rope(double* x, int d, int pos, double theta)
{
    int half = d / 2;
    for (int i = 0; i < half; ++i) {
        double freq = pow(theta, -2.0 * i / d);
        double ang = pos * freq;
        double c = cos(ang), s = sin(ang);
        double a = x[i], b = x[i + half];
        x[i] = a * c - b * s;
        x[i + half] = a * s + b * c;
    }
}

OR_API or_model* or_model_new(const or_cfg* c, int wkind, const void* const* t)
{
    /* t: [embed, final_norm, lm_head, then per layer: attn_norm, wqkv, wo,
       ffn_norm, wgu, wdown] -- the same order the library binds. */
    or_model* m = (or_model*)calloc(1, sizeof(or_model));
    int L = c->n_layers, H = c->hidden, d = c->head_dim;
    m->c = *c;
    m->wkind = wkind;
    m->embed = t[0];
    m->final_norm = t[1];
    m->lm = (or_lin){ wkind, c->vocab, H, 0, t[2], 0, 0 };
    m->attn_norm = (const void**)calloc((size_t)L, sizeof(void*));
    m->ffn_norm = (const void**)calloc((size_t)L, sizeof(void*));
    m->qkv = (or_lin*)calloc((size_t)L, sizeof(or_lin));
    m->o = (or_lin*)calloc((size_t)L, sizeof(or_lin));
    m->gu = (or_lin*)calloc((size_t)L, sizeof(or_lin));
    m->dn = (or_lin*)calloc((size_t)L, sizeof(or_lin));
    for (int l = 0; l < L; ++l) {
        const void* const* tl = t + 3 + 6 * l;
        m->attn_norm[l] = tl[0];
        m->qkv[l] = (or_lin){ wkind, (c->n_q + 2 * c->n_kv) * d, H, 0, tl[1], 0, 0 };
        m->o[l] = (or_lin){ wkind, H, c->n_q * d, 0, tl[2], 0, 0 };
        m->ffn_norm[l] = tl[3];
        m->gu[l] = (or_lin){ wkind, 2 * c->ffn, H, 0, tl[4], 0, 0 };
        m->dn[l] = (or_lin){ wkind, H, c->ffn, 0, tl[5], 0, 0 };
    }
    return m;
}

/* Replace projection `which` (0 qkv, 1 o, 2 gu, 3 down) of layer l by int4
   codes + fp16 scales: this turns a copy of the target into the drafter. */
OR_API void or_model_set_q4(or_model* m, int l, int which, const int8_t* codes,
                            const uint16_t* scales, int group)
{
    or_lin* L = which == 0 ? &m->qkv[l] : which == 1 ? &m->o[l] : which == 2 ? &m->gu[l] : &m->dn[l];
    L->kind = OR_Q4; L->codes = codes; L->scales = scales; L->zeros = NULL; L->group = group;
}

/* The same for any RTN format: integer codes (int4, asymmetric int4 or int8),
   fp16 scales and, for the asymmetric format, zero points (else NULL). */
OR_API void or_model_set_quant(or_model* m, int l, int which, const int8_t* codes,
                               const uint16_t* scales, const uint8_t* zeros, int group)
{
    or_lin* L = which == 0 ? &m->qkv[l] : which == 1 ? &m->o[l] : which == 2 ? &m->gu[l] : &m->dn[l];
    L->kind = OR_Q4; L->codes = codes; L->scales = scales; L->zeros = zeros; L->group = group;
}

OR_API void or_model_free(or_model* m)
{
    if (!m) return;
    free(m->attn_norm); free(m->ffn_norm); free(m->qkv); free(m->o); free(m->gu); free(m->dn);
    free(m);
}

/* Per-sequence KV cache: k, v are double[L][n_kv][cap][head_dim]. */
static size_t kv_index(const or_cfg* c, int cap, int l, int h, int pos, int i)
{
    return (((size_t)l * c->n_kv + h) * cap + pos) * c->head_dim + i;
}

/* Run n tokens of one sequence through the model, the t-th token at
   absolute position start_pos + t; attention of token t covers positions
   [0, start_pos + t].  Writes K/V at those positions.  If logits is not
   NULL it receives float[n][V]. */
OR_API void or_forward_seq(const or_model* m, double* kc, double* vc, int cap,
                           const int32_t* tok, int start_pos, int n, float* logits)
{
    const or_cfg* c = &m->c;
    int H = c->hidden, d = c->head_dim, nq = c->n_q, nkv = c->n_kv, F = c->ffn, V = c->vocab;
    double* h = (double*)malloc(sizeof(double) * H);
    double* a = (double*)malloc(sizeof(double) * H);
    double* qkv = (double*)malloc(sizeof(double) * (size_t)(nq + 2 * nkv) * d);
    double* att = (double*)malloc(sizeof(double) * (size_t)nq * d);
    double* tmp = (double*)malloc(sizeof(double) * (size_t)(H > 2 * F ? H : 2 * F));
    double* act = (double*)malloc(sizeof(double) * (size_t)F);
    double* sc = (double*)malloc(sizeof(double) * (size_t)(start_pos + n));
    double* lg = (double*)malloc(sizeof(double) * (size_t)V);
    double scale = 1.0 / sqrt((double)d);
    for (int t = 0; t < n; ++t) {
        int pos = start_pos + t;
        for (int i = 0; i < H; ++i) h[i] = vec_at(m->wkind, m->embed, (size_t)tok[t] * H + i);
        for (int l = 0; l < c->n_layers; ++l) {
            rmsnorm(h, H, m->wkind, m->attn_norm[l], c->rms_eps, a);
            lin_apply(&m->qkv[l], 0, (nq + 2 * nkv) * d, a, qkv);
            double* q = qkv;
            double* k = qkv + (size_t)nq * d;
            double* v = k + (size_t)nkv * d;
            for (int hh = 0; hh < nq; ++hh) rope(q + (size_t)hh * d, d, pos, c->rope_theta);
            for (int hh = 0; hh < nkv; ++hh) {
                rope(k + (size_t)hh * d, d, pos, c->rope_theta);
                for (int i = 0; i < d; ++i) {
                    kc[kv_index(c, cap, l, hh, pos, i)] = k[(size_t)hh * d + i];
                    vc[kv_index(c, cap, l, hh, pos, i)] = v[(size_t)hh * d + i];
                }
            }
            for (int hh = 0; hh < nq; ++hh) {
                int kh = hh * nkv / nq;
                double mx = -INFINITY;
                for (int p = 0; p <= pos; ++p) {
                    double s = 0.0;
                    for (int i = 0; i < d; ++i) s += q[(size_t)hh * d + i] * kc[kv_index(c, cap, l, kh, p, i)];
                    sc[p] = s * scale;
                    if (sc[p] > mx) mx = sc[p];
                }
                double den = 0.0;
                for (int p = 0; p <= pos; ++p) { sc[p] = exp(sc[p] - mx); den += sc[p]; }
                for (int i = 0; i < d; ++i) {
                    double o = 0.0;
                    for (int p = 0; p <= pos; ++p) o += sc[p] * vc[kv_index(c, cap, l, kh, p, i)];
                    att[(size_t)hh * d + i] = o / den;
                }
            }
            lin_apply(&m->o[l], 0, H, att, tmp);
            for (int i = 0; i < H; ++i) h[i] += tmp[i];
            rmsnorm(h, H, m->wkind, m->ffn_norm[l], c->rms_eps, a);
            lin_apply(&m->gu[l], 0, 2 * F, a, tmp);
            for (int i = 0; i < F; ++i) {
                double g = tmp[i], u = tmp[F + i];
                act[i] = g / (1.0 + exp(-g)) * u;
            }
            lin_apply(&m->dn[l], 0, H, act, tmp);
            for (int i = 0; i < H; ++i) h[i] += tmp[i];
        }
        if (logits) {
            rmsnorm(h, H, m->wkind, m->final_norm, c->rms_eps, a);
            lin_apply(&m->lm, 0, V, a, lg);
            for (int i = 0; i < V; ++i) logits[(size_t)t * V + i] = (float)lg[i];
        }
    }
    free(h); free(a); free(qkv); free(att); free(tmp); free(act); free(sc); free(lg);
}

/* ------------------------------------------------------------------------ */
/* One SD iteration for one sequence (App. D.1, Algorithm 1's SD branch).    */
/* On entry the cache holds clean target KV for positions [0, kv_len) and    */
/* the last token (at position kv_len) is not cached.                        */
/*   draft:  for j = 1..gamma the drafter runs token x_{j-1} at position      */
/*           kv_len + j - 1 (x_0 = last_tok), writing provisional KV there,  */
/*           and samples d_j ~ q_j with the TOKEN stream at kv_len + j;      */
/*   verify: the target runs [last_tok, d_1..d_gamma] at positions kv_len..  */
/*           kv_len + gamma, overwriting that KV with clean values;          */
/*   accept: or_accept_seq;                                                  */
/*   rollback: the new length is kv_len + n_emit; KV at positions beyond it  */
/*           is discarded (here: left in place, never read).                 */
/* Returns n_emit.                                                           */
/* ------------------------------------------------------------------------ */

OR_API int or_sd_step_seq(const or_model* target, const or_model* drafter,
                          double* kc, double* vc, int cap, int kv_len, int32_t last_tok,
                          int gamma, float T, uint64_t seed, uint64_t step, uint32_t slot,
                          int32_t* draft_tok,  /* [gamma] */
                          float* q_logits,     /* [gamma][V] */
                          float* p_logits,     /* [gamma+1][V] */
                          int32_t* out_tok,    /* [gamma+1] */
                          float* draft_gap,    /* [gamma] key gaps of the draft draws, may be NULL */
                          float* ratio_out, float* u_out, float* final_gap)
{
    int V = target->c.vocab;
    int32_t x = last_tok;
    for (int j = 1; j <= gamma; ++j) {
        float* row = q_logits + (size_t)(j - 1) * V;
        or_forward_seq(drafter, kc, vc, cap, &x, kv_len + j - 1, 1, row);
        float gap;
        x = or_sample_row(row, V, T, seed, step, OR_STREAM_TOKEN, slot, (uint32_t)(kv_len + j), &gap);
        if (draft_gap) draft_gap[j - 1] = gap;
        draft_tok[j - 1] = x;
    }
    int32_t* vt = (int32_t*)malloc(sizeof(int32_t) * (size_t)(gamma + 1));
    vt[0] = last_tok;
    for (int j = 0; j < gamma; ++j) vt[j + 1] = draft_tok[j];
    or_forward_seq(target, kc, vc, cap, vt, kv_len, gamma + 1, p_logits);
    free(vt);
    return or_accept_seq(V, gamma, T, draft_tok, q_logits, p_logits, seed, step, slot,
                         (uint32_t)kv_len, out_tok, ratio_out, u_out, final_gap);
}

/* One AR step (the baseline and the toggle-off path): the target runs
   last_tok at position kv_len and the next token is drawn from p with the
   TOKEN stream at kv_len + 1. */
OR_API int32_t or_ar_step_seq(const or_model* target, double* kc, double* vc, int cap,
                              int kv_len, int32_t last_tok, float T, uint64_t seed,
                              uint64_t step, uint32_t slot, float* p_logits, float* gap)
{
    or_forward_seq(target, kc, vc, cap, &last_tok, kv_len, 1, p_logits);
    return or_sample_row(p_logits, target->c.vocab, T, seed, step, OR_STREAM_TOKEN, slot,
                         (uint32_t)(kv_len + 1), gap);
}

/* ------------------------------------------------------------------------ */
/* Block efficiency and the SD speedup model (Sec. 3.1, eq:sd_speedup).      */
/*   tau(alpha, gamma) = (1 - alpha^(gamma+1)) / (1 - alpha)                 */
/*   T_SD = gamma T_q + T_V;  speedup = tau T_p / T_SD.                      */
/* alpha from tau (App. E.2): invert tau(alpha, gamma) by bisection.         */
/* ------------------------------------------------------------------------ */

OR_API double or_tau_from_alpha(double alpha, int gamma)
{
    if (alpha == 1.0) return gamma + 1.0;
    return (1.0 - pow(alpha, gamma + 1)) / (1.0 - alpha);
}

OR_API double or_alpha_from_tau(double tau, int gamma)
{
    if (tau <= 1.0) return 0.0;
    if (tau >= gamma + 1.0) return 1.0;
    double lo = 0.0, hi = 1.0;
    for (int it = 0; it < 200; ++it) {
        double mid = 0.5 * (lo + hi);
        if (or_tau_from_alpha(mid, gamma) < tau) lo = mid; else hi = mid;
    }
    return 0.5 * (lo + hi);
}

OR_API double or_sd_speedup(double tau, double Tp, double Tq, double Tv, int gamma)
{
    return tau * Tp / (gamma * Tq + Tv);
}

/* ------------------------------------------------------------------------ */
/* Roofline cost model and toggle (Sec. 3.2 eq:roofline_basic, Sec. 4.2,     */
/* App. D.2):                                                                */
/*   M_T = (W_T + kappa_eff B S) / BW_eff                                    */
/*   M_D = (eta_D W_D + kappa_eff B S) / BW_eff                              */
/*   C   = B (C_dense + S C_attn) / F_eff                                    */
/*   T_p = max(M_T, C) + c_T B;  T_q = max(M_D, C) + c_D B;                  */
/*   T_V = max(M_T, (gamma+1) C) + c_V B                                     */
/*   pi_SD = 1[ tau T_p / (gamma T_q + T_V) >= 1 + eps ]                     */
/*   kappa_eff = rho_kappa * kappa_th,                                       */
/*   kappa_th = layers * 2 * kv_heads * head_dim * 2 bytes.                  */
/* Architecture-derived terms (our reading, the paper defines them in        */
/* words): W_T, W_D in bytes including embedding and LM head;                */
/* C_dense = 2 * (QKVO + FFN + LM-head parameters) FLOP per token;           */
/* C_attn  = 4 * layers * n_q * head_dim FLOP per token per context entry.   */
/* ------------------------------------------------------------------------ */

typedef struct {
    double W_T, W_D, kappa_th, C_dense, C_attn;   /* architecture terms */
    double BW_eff, F_eff, rho_kappa, eta_D, c_T, c_D, c_V;  /* calibrated */
} or_cost;

/* Architecture terms of a Llama-style decoder.  tbytes: bytes per target
   weight (2 for 16-bit); dbits: bits per quantized drafter weight (4 or 8);
   embedding + LM head (2 * V * H) stay at tbytes in the drafter.  Norm
   vectors are ignored (negligible). */
OR_API void or_cost_arch(int L, int H, int nq, int nkv, int d, int F, int V,
                         double tbytes, double dbits, double kvbytes, or_cost* out)
{
    double qkvo = (double)L * ((double)H * (nq + 2 * nkv) * d + (double)nq * d * H);
    double ffn = (double)L * 3.0 * H * F;
    double emb_lm = 2.0 * V * H;
    out->W_T = tbytes * (qkvo + ffn + emb_lm);
    out->W_D = dbits / 8.0 * (qkvo + ffn) + tbytes * emb_lm;
    out->kappa_th = (double)L * 2.0 * nkv * d * kvbytes;
    out->C_dense = 2.0 * (qkvo + ffn + (double)V * H);
    out->C_attn = 4.0 * L * nq * d;
}

OR_API void or_cost_times(const or_cost* c, double B, double S, int gamma,
                          double* Tp, double* Tq, double* Tv)
{
    double kv = c->rho_kappa * c->kappa_th * B * S;
    double MT = (c->W_T + kv) / c->BW_eff;
    double MD = (c->eta_D * c->W_D + kv) / c->BW_eff;
    double C = B * (c->C_dense + S * c->C_attn) / c->F_eff;
    *Tp = (MT > C ? MT : C) + c->c_T * B;
    *Tq = (MD > C ? MD : C) + c->c_D * B;
    double CV = (gamma + 1) * C;
    *Tv = (MT > CV ? MT : CV) + c->c_V * B;
}

OR_API int or_toggle(const or_cost* c, double B, double S, double tau, int gamma, double eps)
{
    double Tp, Tq, Tv;
    or_cost_times(c, B, S, gamma, &Tp, &Tq, &Tv);
    return tau * Tp / (gamma * Tq + Tv) >= 1.0 + eps;
}

/* ------------------------------------------------------------------------ */
/* Adaptive draft length (Sec. 4.3, Algorithm 1):                            */
/*   raise to next(gamma) if min of the last P taus >= 1 + gamma alpha_up    */
/*   and gamma < gamma_high; lower to prev(gamma) if max of the last P taus  */
/*   <= 1 + gamma alpha_down and gamma > gamma_low; else hold.               */
/* With fewer than P measurements the window is not full: hold (reading).   */
/* hist holds the taus in time order, the last entry being the newest.       */
/* ------------------------------------------------------------------------ */

OR_API int or_gamma_next(const int* set, int n_set, int gamma, const double* hist, int n_hist,
                         int P, double a_up, double a_down)
{
    int idx = -1;
    for (int i = 0; i < n_set; ++i) if (set[i] == gamma) idx = i;
    if (idx < 0 || n_hist < P || P <= 0) return gamma;
    double mn = INFINITY, mx = -INFINITY;
    for (int i = n_hist - P; i < n_hist; ++i) { if (hist[i] < mn) mn = hist[i]; if (hist[i] > mx) mx = hist[i]; }
    if (mn >= 1.0 + gamma * a_up && idx < n_set - 1) return set[idx + 1];
    if (mx <= 1.0 + gamma * a_down && idx > 0) return set[idx - 1];
    return gamma;
}

/* Sticky toggle state (Algorithm 1): once SD is on it stays on for the rest
   of the rollout.  Returns the new state. */
OR_API int or_toggle_sticky(const or_cost* c, double B, double S, double tau, int gamma,
                            double eps, int* sd_on)
{
    if (!*sd_on && or_toggle(c, B, S, tau, gamma, eps)) *sd_on = 1;
    return *sd_on;
}

/* ------------------------------------------------------------------------ */
/* Roofline decode-time breakdown of one single-token decode step (App. B.1, */
/* Table 3): each component costs max(FLOPs / F, bytes / BW).                */
/* out[0..3] = FFN, QKVO projections, attention (QK and PV over the cache),  */
/* LM head, in seconds.  Weights at wbytes per parameter, KV at kvbytes.     */
/* ------------------------------------------------------------------------ */

OR_API void or_decode_breakdown(int L, int H, int nq, int nkv, int d, int F, int V,
                                double wbytes, double kvbytes, double B, double S,
                                double flops, double bw, double* out)
{
    double p_ffn = (double)L * 3.0 * H * F;
    double p_qkvo = (double)L * ((double)H * (nq + 2 * nkv) * d + (double)nq * d * H);
    double p_lm = (double)V * H;
    double t[4];
    double P[3] = { p_ffn, p_qkvo, p_lm };
    for (int i = 0; i < 3; ++i) {
        double c = 2.0 * B * P[i] / flops, m = wbytes * P[i] / bw;
        t[i] = c > m ? c : m;
    }
    double kv_bytes = (double)L * 2.0 * nkv * d * kvbytes * B * S;
    double attn_flops = 4.0 * L * nq * d * B * S;
    double ca = attn_flops / flops, ma = kv_bytes / bw;
    out[0] = t[0]; out[1] = t[1]; out[2] = ca > ma ? ca : ma; out[3] = t[2];
}

/* Histogram helpers for the statistical pins (test support). */

/* n draws x ~ softmax(l/T) by exponential race, the t-th draw using the
   TOKEN stream of slot 0 at position t. */
OR_API void or_sample_hist(const float* l, int V, float T, uint64_t seed, uint64_t step,
                           int n, int64_t* counts)
{
    for (int t = 0; t < n; ++t) {
        int x = or_sample_row(l, V, T, seed, step, OR_STREAM_TOKEN, 0, (uint32_t)t, 0);
        counts[x]++;
    }
}

/* n single-token SD trials with gamma = 1 over fixed rows q, p1, p2: the
   draft d ~ q (TOKEN stream), then or_accept_seq.  counts[x] histograms the
   first emitted token; *n_acc counts accepted drafts. */
OR_API void or_accept_hist(const float* q, const float* p12, int V, float T, uint64_t seed,
                           uint64_t step, int n, int64_t* counts, int64_t* n_acc)
{
    int32_t out[2];
    for (int t = 0; t < n; ++t) {
        uint32_t kv_len = (uint32_t)(2 * t);
        int32_t d = or_sample_row(q, V, T, seed, step, OR_STREAM_TOKEN, 0, kv_len + 1u, 0);
        int ne = or_accept_seq(V, 1, T, &d, q, p12, seed, step, 0, kv_len, out, 0, 0, 0);
        counts[out[0]]++;
        if (ne == 2) (*n_acc)++;
    }
}

/* ------------------------------------------------------------------------ */
/* Threads of the parallel loops (timing of the oracle on one or all host    */
/* cores); n <= 0 restores every core.                                       */
/* ------------------------------------------------------------------------ */
OR_API void or_set_threads(int n)
{
    omp_set_num_threads(n > 0 ? n : omp_get_num_procs());
}

OR_API int or_get_threads(void) { return omp_get_max_threads(); }
