/*
 * sd_api.h -- C ABI of the MI355X (gfx950) quantized self-speculative
 * decoding engine.
 *
 * Method: "EfficientRollout: System-Aware Self-Speculative Decoding for RL
 * Rollouts".  A weight-quantized copy of the target (RTN int4, groups of 128
 * along K, fp16 scales; Sec. 4.1) drafts gamma tokens per sequence; the
 * target verifies all B*(gamma+1) positions in one forward pass; speculative
 * rejection sampling keeps the target distribution exactly; the KV entries of
 * rejected positions are discarded (App. D.1); a roofline cost model decides
 * when SD is on (Sec. 4.2, App. D.2) and how long drafts are (Sec. 4.3,
 * Algorithm 1).
 *
 * Conventions for every call below.
 *   Pointers.  Unless a comment says "host", a pointer argument is device
 *     memory on the engine's GPU, allocated and owned by the caller; the
 *     library never frees it and keeps bound pointers until sd_destroy.
 *   Streams.  `stream` is a hipStream_t passed as void*; NULL is the null
 *     stream.  GPU calls validate their arguments on the host, enqueue work
 *     and return without waiting.
 *   Errors.  Calls return sd_status; on anything but SD_OK, sd_last_error()
 *     gives a message (thread-local, valid until the next call on the same
 *     thread).  Device-side range errors (a slot index outside
 *     [0, max_slots), a token id outside [0, vocab), a position at or beyond
 *     max_ctx) never touch memory out of bounds: the offending row is
 *     skipped and a device flag is set; sd_sync reports it as SD_E_INVAL.
 *     No C++ exception crosses this interface.
 *   Types.  Tokens, lengths and slot indices are int32; logits and
 *     statistics are fp32.  The model dtype (fp32 or bf16) applies to the
 *     weights and the KV cache.
 *   KV semantics.  kv_len[slot] counts cached positions of a sequence; its
 *     last token (position kv_len) is not cached yet.  A step that starts
 *     with last token x at position kv_len caches x and predicts the tokens
 *     at kv_len + 1, kv_len + 2, ...
 *   Randomness.  Philox-4x64-10 with key (seed, step) and counter (block,
 *     position, slot, stream); streams: 0 token draws (draft, AR, bonus),
 *     1 accept tests, 2 residual draws.  A draw for the token at absolute
 *     position P of a slot uses counter position P.  A slot reused for a new
 *     sequence under the same (seed, step) repeats its uniforms: give each
 *     rollout its own `step`.
 */
#ifndef SD_API_H
#define SD_API_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sd_engine_s* sd_engine;   /* opaque; owned by the library */

typedef enum {
    SD_OK = 0,
    SD_E_INVAL = 1,        /* bad argument, or a device range error (sd_sync) */
    SD_E_NOMEM = 2,        /* workspace allocation failed */
    SD_E_HIP = 3,          /* a HIP runtime call or kernel launch failed */
    SD_E_STATE = 4,        /* weights / KV not bound, drafter not refreshed */
    SD_E_UNSUPPORTED = 5   /* shape outside what the kernels handle */
} sd_status;

typedef enum { SD_DTYPE_F32 = 0, SD_DTYPE_BF16 = 1 } sd_dtype;

/* Llama-style decoder (RMSNorm, RoPE rotate-half, GQA, SwiGLU, untied LM
 * head, no biases).  Requirements: hidden, ffn and n_q*head_dim multiples of
 * 128; (n_q + 2*n_kv)*head_dim and vocab multiples of 64; head_dim 64 or 128;
 * n_q a multiple of n_kv; group == 128. */
typedef struct {
    int32_t n_layers, hidden, n_q, n_kv, head_dim, ffn, vocab;
    int32_t dtype;      /* sd_dtype */
    int32_t group;      /* quantization group along K: 128 */
    float rms_eps;      /* RMSNorm epsilon */
    float rope_theta;   /* RoPE base */
} sd_model_cfg;

typedef struct { uint64_t seed, step; } sd_rng;

/* Message for the last non-OK status on this thread ("" if none). */
const char* sd_last_error(void);

/* ------------------------------------------------------------------ setup */

/* Creates an engine on the current HIP device.  max_slots: KV slots (and the
 * largest batch B); max_ctx: cached positions per slot; max_gamma: longest
 * draft.  The engine allocates its own workspace, sized for
 * max_slots*(max_gamma+1) rows. *out receives the handle. */
sd_status sd_create(const sd_model_cfg* cfg, int32_t max_slots, int32_t max_ctx, int32_t max_gamma,
                    sd_engine* out);
sd_status sd_destroy(sd_engine e);

/* Number of weight tensors sd_bind_weights expects: 3 + 6*n_layers. */
int32_t sd_num_weights(const sd_model_cfg* cfg);

/* Binds the target's weights (device pointers in the model dtype, row-major,
 * K contiguous).  tensors (host array of n pointers), in order:
 *   [0] embedding [vocab][hidden], [1] final norm gain [hidden],
 *   [2] LM head [vocab][hidden], then per layer l (base 3 + 6*l):
 *   attn-norm gain [hidden], Wqkv [(n_q+2*n_kv)*head_dim][hidden] (rows: Wq,
 *   then Wk, then Wv), Wo [hidden][n_q*head_dim], ffn-norm gain [hidden],
 *   Wgu [2*ffn][hidden] (rows: gate, then up), Wdown [hidden][ffn].
 * Every pointer must be 16-byte aligned (the kernels read weights in
 * 16-byte pieces); a NULL or misaligned pointer gives SD_E_INVAL. */
sd_status sd_bind_weights(sd_engine e, const void* const* tensors, int32_t n);

/* Bytes of EACH of the K and V caches: n_layers*max_slots*n_kv*max_ctx*
 * head_dim elements of the model dtype, laid out [L][slot][n_kv][pos][d]. */
size_t sd_kv_bytes(const sd_model_cfg* cfg, int32_t max_slots, int32_t max_ctx);

/* Binds the shared KV cache (App. D.1: the drafter writes provisional
 * entries into the target's cache) and the per-slot lengths kv_len
 * (device int32[max_slots]).  K holds post-RoPE keys.  k and v must be
 * 16-byte aligned (SD_E_INVAL otherwise). */
sd_status sd_bind_kv(sd_engine e, void* k, void* v, int32_t* kv_len);

/* Bytes of EACH of the K and V pages of a paged cache: n_layers*n_kv*
 * page_size*head_dim elements of the model dtype (0 for page_size < 1). */
size_t sd_kv_page_bytes(const sd_model_cfg* cfg, int32_t page_size);

/* Binds a paged KV cache instead (the page-granular memory of serving
 * engines the paper's rollouts run in, Sec. 4.1 and App. B.2): K and V pools
 * of n_pages pages, each laid out [L][n_kv][page_size][head_dim], and a
 * block table block_table (device int32 [max_slots][pages_per_seq]) whose
 * entry (slot, j) names the page holding that slot's positions
 * [j*page_size, (j+1)*page_size).  All three are caller-owned and read by
 * every later call; the caller may change table entries between calls (e.g.
 * hand pages of finished sequences to new ones) but not while a call it
 * enqueued is running.  Positions are still kv_len-relative: rollback only
 * moves kv_len, and pages past it stay the caller's to reuse.  Requires
 * page_size a multiple of 32, pages_per_seq*page_size >= max_ctx and
 * 16-byte aligned pools (SD_E_INVAL otherwise).  A table entry outside [0, n_pages) met on the
 * device is skipped and reported by sd_sync as SD_E_INVAL.  Replaces any
 * earlier binding. */
sd_status sd_bind_kv_paged(sd_engine e, void* k_pages, void* v_pages, int32_t n_pages, int32_t page_size,
                           const int32_t* block_table, int32_t pages_per_seq, int32_t* kv_len);

/* Drafter weight formats (RTN, groups of 128 weights along K, one fp16 scale
 * per (output column, group)): int4 symmetric (Sec. 4.1, the default), int4
 * asymmetric with a zero point per (column, group) (App. B.2), and int8
 * symmetric (the W8 drafter of App. B.3 / Table 4). */
typedef enum { SD_DRAFT_W4 = 0, SD_DRAFT_W4A = 1, SD_DRAFT_W8 = 2 } sd_draft_fmt;

/* Bytes of the quantized drafter for cfg in format fmt (0 for an unknown
 * format): for each layer, the projections qkv, o, gu, down in that order,
 * each as packed codes (N*K/2 bytes for int4, N*K for int8), then fp16
 * scales (N*K/64 bytes), then for SD_DRAFT_W4A one zero-point byte per
 * (column, group) (N*K/128 bytes), every block 256-byte aligned.  Packed
 * layout: see sd_refresh_drafter_fmt. */
size_t sd_drafter_bytes_fmt(const sd_model_cfg* cfg, int32_t fmt);

/* sd_drafter_bytes_fmt(cfg, SD_DRAFT_W4). */
size_t sd_drafter_bytes(const sd_model_cfg* cfg);

/* Drafter refresh (Sec. 4.1; Algorithm 1 does it at the start of every
 * training step): RTN quantization of Wqkv, Wo, Wgu, Wdown of every layer of
 * the bound target, in format fmt, into qbuf (device, 16-byte aligned,
 * >= sd_drafter_bytes_fmt(cfg, fmt) bytes, owned by the caller and read by
 * every later sd_draft).  Embedding, norms and LM head are shared with the
 * target, unquantized.  Per group of 128 weights of one row:
 *   SD_DRAFT_W4:  s = fp16(max|w|/7), q = clamp(rint(w/s), -8, 7);
 *   SD_DRAFT_W4A: s = fp16((max-min)/15), z = clamp(rint(-min/s), 0, 15),
 *                 q = clamp(rint(w/s) + z, 0, 15), weight s*(q - z);
 *   SD_DRAFT_W8:  s = fp16(max|w|/127), q = clamp(rint(w/s), -128, 127)
 * (q = z = 0 when s = 0; fp32 arithmetic, round half to even).
 * Packed layout per matrix [N][K] (N a multiple of 32, G = K/128), for
 * column block nb = n/32 and group g = k/128; lane l = n%32 + 32*h (h = 0, 1)
 * stands for the codes k = 128g + 16st + 8h + e, st = 0..7, e = 0..7:
 *   int4: code e of k-step st in the nibble at bit 4*(e/2) + 16*(e%2) of
 *         word (((nb*G + g)*2 + st/4)*64 + l)*4 + st%4, stored as q + 8
 *         (W4) or q (W4A);
 *   int8: code e of k-step st in byte e%4 of word j = 2*st + e/4 at index
 *         (((nb*G + g)*4 + j/4)*64 + l)*4 + j%4, stored as q + 128.
 * Scale and zero point of (n, g) at index (nb*G + g)*32 + n%32.  Errors:
 * SD_E_INVAL (NULL, misaligned or short qbuf, unknown fmt), SD_E_STATE
 * (weights not bound).  Must be called again after the weights change; a
 * failed refresh leaves the engine without a drafter. */
sd_status sd_refresh_drafter_fmt(sd_engine e, int32_t fmt, void* qbuf, size_t bytes, void* stream);

/* sd_refresh_drafter_fmt(e, SD_DRAFT_W4, qbuf, bytes, stream). */
sd_status sd_refresh_drafter(sd_engine e, void* qbuf, size_t bytes, void* stream);

/* --------------------------------------------------------- the SD step */

/* Target prefill: caches tokens[b*n + i] (device int32[B][n]) of sequence
 * slots[b] at positions kv_len + i, then kv_len += n. */
sd_status sd_prefill(sd_engine e, int32_t B, const int32_t* slots, const int32_t* tokens, int32_t n,
                     void* stream);

/* Target prefill of prompts of different lengths (the rollout's prompts,
 * Sec. 5.1; every decoding step then starts from each sequence's own
 * kv_len, App. D.1): caches tokens[b*ld + i] for i < len[b] (tokens: device
 * int32[B][ld], row b's entries past len[b] are never read) of sequence
 * slots[b] at positions kv_len + i, then kv_len += len[b].  len: device
 * int32[B] with 0 <= len[b] <= ld.  The batch runs in rounds of a common
 * number of positions; a sequence whose prompt has ended computes padding
 * rows that are neither cached nor counted.  Errors: SD_E_INVAL (NULL
 * pointers, ld outside [1, max_ctx]), SD_E_STATE; a length outside [0, ld]
 * is reported by sd_sync (and that sequence is left unchanged), as are bad
 * slots, token ids and positions past max_ctx. */
sd_status sd_prefill_ragged(sd_engine e, int32_t B, const int32_t* slots, const int32_t* tokens, int32_t ld,
                            const int32_t* len, void* stream);

/* Draft (Algorithm 1's SD branch, App. D.1): for j = 1..gamma the drafter
 * runs x_{j-1} (x_0 = last_tok[b]) at position kv_len + j - 1, writes
 * provisional KV there, and draws d_j ~ softmax(q_j / temperature) by
 * exponential race (stream 0, position kv_len + j).  Outputs (device):
 * draft_tok int32[B][gamma], q_logits fp32[B][gamma][vocab] (raw logits),
 * q_stats fp32[B][gamma][2] = (max, log-sum-exp) of q_logits/temperature.
 * kv_len is not changed. */
sd_status sd_draft(sd_engine e, int32_t B, const int32_t* slots, const int32_t* last_tok, int32_t gamma,
                   float temperature, sd_rng rng, int32_t* draft_tok, float* q_logits, float* q_stats,
                   void* stream);

/* Verify (App. D.1): the target runs [last_tok[b], d_1..d_gamma] at positions
 * kv_len..kv_len+gamma in one forward pass (causal inside the block),
 * overwriting the provisional KV with clean target KV.  p_logits:
 * fp32[B][gamma+1][vocab], row i predicting the token at kv_len + i + 1. */
sd_status sd_verify(sd_engine e, int32_t B, const int32_t* slots, const int32_t* last_tok,
                    const int32_t* draft_tok, int32_t gamma, float* p_logits, void* stream);

/* Speculative rejection sampling (Sec. 3.1, App. D.1): for j = 1..gamma,
 * accept d_j iff u_j <= p_j(d_j)/q_j(d_j) with u_j from stream 1 at position
 * kv_len + j; at the first rejection draw from norm(max(0, p_j - q_j))
 * (stream 2 at kv_len + j; from p_j if the residual vanishes); if all pass
 * draw a bonus token from p_{gamma+1} (stream 0 at kv_len + gamma + 1).
 * q_j uses q_stats (the distribution the drafts were drawn from).
 * Outputs: out_tok int32[B][gamma+1] (entries past n_emit set to -1),
 * n_emit int32[B] in [1, gamma+1], next_tok int32[B] = the last emitted
 * token (may be NULL).  kv_len is not changed. */
sd_status sd_accept(sd_engine e, int32_t B, const int32_t* slots, const int32_t* draft_tok,
                    const float* q_logits, const float* q_stats, const float* p_logits, int32_t gamma,
                    float temperature, sd_rng rng, int32_t* out_tok, int32_t* n_emit, int32_t* next_tok,
                    void* stream);

/* The rejection sampler of sd_accept for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): no engine, and no hipMalloc, hipFree or
 * allocating library call.  The same kernels as sd_accept, with the same
 * decisions and outputs; the engine's state becomes arguments: vocab, and
 * kv_len (device int32[max_slots]) holding each slot's cached length, which
 * places the Philox counters exactly as in sd_accept (slots[b] must lie in
 * [0, max_slots)).  All other arguments, layouts and outputs as sd_accept.
 * Scratch: the kernels' partial results live in a static device array of
 * 2^20 floats (4 MiB) per GPU, held until the process ends; a call needs
 * B*(gamma+1)*C*2 + B*C*4 + 6*B + 5 floats with C = ceil(vocab / 4096)
 * vocabulary chunks, and a larger one returns SD_E_INVAL before launching
 * anything.  Every call on a GPU shares that GPU's array: calls whose work
 * overlaps on one GPU (different streams, or threads) race and must not be
 * made.  A slot index outside [0, max_slots) yields n_emit = 0, out_tok
 * row -1 and next_tok -1 for that row (there is no engine to report it). */
sd_status sd_accept_noalloc(int32_t B, int32_t vocab, const int32_t* slots, const int32_t* kv_len,
                            int32_t max_slots, const int32_t* draft_tok, const float* q_logits,
                            const float* q_stats, const float* p_logits, int32_t gamma, float temperature,
                            sd_rng rng, int32_t* out_tok, int32_t* n_emit, int32_t* next_tok, void* stream);

/* KV rollback (App. D.1): kv_len[slots[b]] += n_emit[b]; positions at or
 * beyond the new length (the rejected drafts' KV) are discarded.  With the
 * debug poison switch on, the discarded span is overwritten with NaN. */
sd_status kv_rollback(sd_engine e, int32_t B, const int32_t* slots, const int32_t* n_emit, void* stream);

/* Plain autoregressive step (the baseline and the SD-off path): the target
 * runs last_tok at kv_len, out_tok[b] ~ softmax(p/temperature) (stream 0 at
 * kv_len + 1), p_logits fp32[B][vocab] receives the logits, kv_len += 1. */
sd_status sd_ar_step(sd_engine e, int32_t B, const int32_t* slots, const int32_t* last_tok, float temperature,
                     sd_rng rng, int32_t* out_tok, float* p_logits, void* stream);

/* Waits for `stream` and reports device-side range errors raised since the
 * last sd_sync (SD_E_INVAL) or HIP errors (SD_E_HIP); clears the flags. */
sd_status sd_sync(sd_engine e, void* stream);

/* Debug switches (flags, host): bit 0 = kv_rollback poisons discarded KV with
 * NaN; bit 1 = the gate/up projection and SwiGLU run as two kernels (by
 * default SwiGLU runs in the projection's epilogue where a fused kernel
 * exists); bit 2 = bf16 GEMMs with 320-row tiles stage their operands through
 * registers instead of loading them into LDS by DMA.  Each switch gives
 * identical results.  Other bits: SD_E_INVAL. */
sd_status sd_set_debug(sd_engine e, int32_t flags);

/* Kernel timing (diagnostics).  While on, the engine brackets each launch of
 * a kernel class with HIP events recorded on the launch stream.  Classes:
 * 0 attention over the cache for one query token per sequence (draft and AR
 * steps; the partial kernel only), 1 attention for the gamma+1 verify
 * queries (partial kernel), 2 int4 projections (drafter), 3 bf16/fp32
 * projections (target layers), 4 LM head, 5 token sampler, 6 accept,
 * 7 norms / RoPE / embedding / SwiGLU / attention combine / KV bookkeeping.
 * sd_timing(e, 1) also clears the accumulated records. */
sd_status sd_timing(sd_engine e, int32_t on);

/* Waits for the recorded events and returns, for class `cls`, the summed
 * kernel time in milliseconds and the number of launches (host pointers). */
sd_status sd_timing_read(sd_engine e, int32_t cls, double* total_ms, int32_t* launches);

/* Dense GEMM with the library's bf16 kernels, for the F_eff microbenchmark
 * of the cost-model calibration (App. D.2: effective compute throughput from
 * repeated dense matrix multiplications).  C[M][N] (fp32, row stride N) =
 * A[M][K] (bf16, row-major) x W[N][K]^T (bf16, row-major); device pointers,
 * caller-owned.  Needs N % 128 == 0 and K % 128 == 0; M >= 1.  No split-K
 * (no workspace).  Enqueued on `stream`. */
sd_status sd_dense_gemm_bf16(const void* A, const void* W, float* C, int32_t M, int32_t N, int32_t K, void* stream);

/* ------------------------------------------------ host policy (no GPU) */

/* Roofline cost model of Sec. 4.2 / App. D.2.  Architecture terms: W_T, W_D
 * bytes of target and drafter weights (embedding and LM head included),
 * kappa_th = layers*2*n_kv*head_dim*kv_bytes per cached token, C_dense =
 * 2*(QKVO + FFN + LM-head parameters) FLOP per token, C_attn =
 * 4*layers*n_q*head_dim FLOP per token per context entry.  Calibrated:
 * BW_eff (B/s), F_eff (FLOP/s), rho_kappa, eta_D, c_T, c_D, c_V (s per
 * sequence). */
typedef struct {
    double W_T, W_D, kappa_th, C_dense, C_attn;
    double BW_eff, F_eff, rho_kappa, eta_D, c_T, c_D, c_V;
} sd_cost_model;

/* Fills the architecture terms for cfg (weight_bytes per target weight,
 * drafter_bits per quantized weight, kv_bytes per cache element) and sets
 * the calibrated terms to neutral values (rho_kappa = eta_D = 1, overheads
 * 0, BW_eff = 8e12, F_eff = 2.5e15).  cfg and out are host pointers. */
sd_status sd_cost_init(const sd_model_cfg* cfg, double weight_bytes, double drafter_bits, double kv_bytes,
                       sd_cost_model* out);

/* T_p, T_q, T_V of Sec. 4.2 at batch B, mean live length S, draft length
 * gamma:  M_T = (W_T + kappa_eff*B*S)/BW_eff,
 * M_D = (eta_D*W_D + kappa_eff*B*S)/BW_eff, C = B*(C_dense + S*C_attn)/F_eff,
 * T_p = max(M_T, C) + c_T*B, T_q = max(M_D, C) + c_D*B,
 * T_V = max(M_T, (gamma+1)*C) + c_V*B.  Host pointers. */
sd_status sd_cost_times(const sd_cost_model* m, double B, double S, int32_t gamma, double* Tp, double* Tq,
                        double* Tv);

/* SD toggle pi_SD (eq:sd_speedup_toggle): on iff
 * tau*T_p/(gamma*T_q + T_V) >= 1 + eps.  *sd_on (host, in/out) is sticky:
 * once 1 it stays 1 (Algorithm 1).  Returns the new *sd_on, or -1 on a bad
 * argument. */
int32_t sd_toggle(const sd_cost_model* m, int32_t B, double S_mean, double tau, int32_t gamma, double eps,
                  int32_t* sd_on);

/* Adaptive draft length (Sec. 4.3, Algorithm 1).  State: the ordered set
 * Gamma (<= 16 entries), patience P, thresholds alpha_up, alpha_down, the
 * current gamma and the tau history.  Initial gamma = Gamma[0]. */
typedef struct {
    int32_t set[16];
    int32_t n_set, P, gamma, n_hist;
    double a_up, a_down;
    double hist[64];
} sd_gamma_ctl;

sd_status sd_gamma_init(sd_gamma_ctl* c, const int32_t* set, int32_t n_set, int32_t P, double a_up,
                        double a_down);

/* Records the step's measured block efficiency tau_t and moves gamma:
 * next(Gamma) if min of the last P taus >= 1 + gamma*a_up (gamma below the
 * top), prev(Gamma) if max of the last P taus <= 1 + gamma*a_down (gamma
 * above the bottom), else unchanged; fewer than P taus: unchanged.
 * *gamma_next (host) receives the new gamma. */
sd_status sd_gamma_next(sd_gamma_ctl* c, double tau_t, int32_t* gamma_next);

/* Block efficiency under i.i.d. acceptance (Sec. 3.1):
 * tau = (1 - alpha^(gamma+1))/(1 - alpha); and its inverse (App. E.2). */
double sd_tau_from_alpha(double alpha, int32_t gamma);
double sd_alpha_from_tau(double tau, int32_t gamma);

#ifdef __cplusplus
}
#endif

#endif /* SD_API_H */
