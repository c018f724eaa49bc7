// kernels.h -- launcher prototypes shared by the engine and the kernel files.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

// Activation element types fed to the GEMMs.
enum act_t : int { ACT_F32 = 0, ACT_BF16 = 1, ACT_F16 = 2 };

inline size_t act_bytes(act_t a) { return a == ACT_F32 ? 4 : 2; }

// Row geometry of one forward call: B sequences with n new tokens each; row
// r = b*n + i sits at absolute position kv_len[slots[b]] + off + i.
struct rows_t {
    int B, n, off;
    const int32_t* slots;   // device [B]
    const int32_t* kv_len;  // device [max_slots]
    int max_slots, max_ctx;
    uint32_t* err;          // device error words
    const int32_t* lim = nullptr;   // device [B] or NULL: rows (b, i >= lim[b]) are padding, skipped silently
};

// KV cache geometry.  The element offset of (slot, layer, KV head h,
// position p) is page * PS + layer * LS + h * HS + (p % P) * head_dim, with
//   dense cache [L][max_slots][n_kv][max_ctx][head_dim]: P = max_ctx and
//     page = slot;
//   paged cache, pages [n_pages][L][n_kv][P][head_dim]: page =
//     bt[slot * mpp + p / P] from the caller's block table (an entry outside
//     [0, n_pages) is reported as ERR_PAGE and its positions are skipped).
struct kv_geom {
    int P;                     // positions per page
    long long PS, LS, HS;      // element strides of a page, a layer and a KV head
    const int32_t* bt;         // device int32 [max_slots][mpp], or NULL for the dense cache
    int mpp, n_pages;
};

struct cache_t {
    void* k;
    void* v;
    int kv_f32;             // 1: fp32 cache, 0: bf16 cache
    int n_kv, head_dim;
    kv_geom g;
};

// ---- model kernels (kernels_model.hip)
// A kernel input produced by a split-K projection is given as partials P with
// S > 1 splits ([S][rows][cols], summed on read); S <= 1 means the producer
// wrote its output directly.
void launch_embed_rmsnorm(const rows_t& r, const int32_t* tokA, int sA, const int32_t* tokB, int sB,
                          const void* E, int w_f32, int H, int V, float* h, const void* gain, float eps,
                          void* out, act_t out_t, hipStream_t s);
void launch_add_rmsnorm(float* h, const float* P, int S, int R, int H, const void* gain, int g_f32,
                        float eps, void* out, act_t out_t, hipStream_t s);
void launch_rope_kv(const rows_t& r, const float* qkv, const float* P, int S, const float2* rope, int n_q,
                    const cache_t& c, int layer, float* q_out, hipStream_t s);
// Attention in two launches: per-chunk partial softmax-weighted sums into
// part, then the combine over chunks into out.
// chunks and chunk length of a split-context attention launch; done when
// each sequence was a single chunk and the kernel wrote the output itself
struct attn_split { int chunks, chunk; bool done; };
// The QKV projection's output as k_rope_kv reads it (qkv, or S > 1 split-K
// partials P) with the RoPE table.  The attention applies RoPE and writes the
// new rows: with a bf16 cache the attention kernel itself rotates its query
// rows and writes its KV head's new K (rotated) and V rows of its context
// range before reading them; with an fp32 cache k_rope_kv runs first, writing
// the rotated queries into q (scratch, [rows][n_q][head_dim] fp32).
struct qkv_src {
    const float* qkv;
    const float* P;
    int S;
    const float2* rope;
};
// ev0/ev1, when given, are bound to the attention kernel's own dispatch
// (hipExtLaunchKernelGGL): their elapsed time is the kernel's run time.
attn_split launch_attention(const rows_t& r, qkv_src qs, float* q, int n_q, const cache_t& c, int layer, float* part,
                            int max_chunks, void* out, act_t out_t, hipStream_t s, hipEvent_t ev0 = nullptr,
                            hipEvent_t ev1 = nullptr);
void launch_attention_combine(const rows_t& r, int n_q, int head_dim, const float* part, attn_split sp, void* out,
                              act_t out_t, hipStream_t s);
size_t attention_part_floats(int R, int n_q, int head_dim, int max_chunks);
int attention_chunk();
void launch_silu_mul(const float* gu, const float* P, int S, int R, int F, void* out, act_t out_t, hipStream_t s);
void launch_kv_advance(int B, const int32_t* slots, const int32_t* inc, int inc_const,
                       int32_t* kv_len, int max_slots, uint32_t* err, hipStream_t s);
// lim[b] = clamp(len[b] - t0, 0, nc) for one round of a ragged prefill; a
// length outside [0, ld] sets ERR_LEN and counts as 0
void launch_prefill_lim(int B, const int32_t* len, int t0, int nc, int ld, int32_t* lim, uint32_t* err, hipStream_t s);
void launch_kv_poison(int B, const int32_t* slots, const int32_t* kv_len, int span,
                      const cache_t& c, int n_layers, int max_slots, int max_ctx, hipStream_t s);

// ---- GEMMs (kernels_gemm.hip): C[M][N] (fp32, row stride ldc) = or += A[M][K] W^T
enum gemm_mode : int { GEMM_STORE = 0, GEMM_ADD = 1 };
// bf16 MFMA GEMM: weight-streaming kernel for M <= 64 per m-tile, LDS-tiled
// kernel for M > 64.  part is split-K scratch of part_cap floats (no split
// when too small).  Returns the number of K splits S used.  With
// defer_reduce and S > 1 the partials are left in part ([S][M][N]) for the
// consumer to sum; otherwise C holds the result.  lds_dma: 320-row tiles
// without split-K use the DMA-fed kernel (same sums as the register-staged
// one; false selects the latter).
int launch_gemm_bf16(const uint16_t* A, const uint16_t* W, float* C, float* part, size_t part_cap, int M, int N, int K,
                     int ldc, gemm_mode mode, bool defer_reduce, hipStream_t s, bool lds_dma = true);
// The gate/up projection with SwiGLU in its epilogue: out[M][F] (type out_t)
// = SiLU(g) * u, [g | u] = A W^T with W [2F][K] (gate rows, then up rows).
// Returns 1 when launched, 0 when the shape has no fused kernel (the caller
// then runs the plain GEMM and launch_silu_mul).  The int4 form takes the
// packed drafter layout of kernels_q4.hip.
int launch_gemm_bf16_swiglu(const uint16_t* A, const uint16_t* W, void* out, act_t out_t, int M, int F, int K,
                            hipStream_t s, bool lds_dma = true);
int launch_gemm_q4_swiglu(const uint16_t* A, const uint32_t* Wq, const uint16_t* Sc, const uint8_t* Z, int fmt,
                          void* out, act_t out_t, int M, int F, int K, hipStream_t s);
size_t gemm_part_floats(int M, int N, int K);
// ---- drafter weight formats: RTN over groups of 128 weights along K, one
// fp16 scale per (column, group); int4 symmetric (codes stored as q + 8),
// int4 asymmetric (codes q in 0..15 plus a zero point z per (column,
// group), w = s (q - z)) and int8 symmetric (codes stored as q + 128).
enum qfmt : int { QF_W4 = 0, QF_W4A = 1, QF_W8 = 2 };
// bytes of the packed codes of an [N][K] matrix
inline size_t qfmt_code_bytes(int fmt, int N, int K) { return (size_t)N * K / (fmt == QF_W8 ? 1 : 2); }

// ---- quantized drafter GEMM (kernels_q4.hip): C[M][N] (+)= A[M][K] Wq^T,
// A fp16, Wq in the packed 32-column tile layout of format fmt, Z the zero
// points (QF_W4A only), N % 32 == 0.  Returns the number of K splits S
// (partials left in part as [S][M][N] when S > 1, for the consumer to sum),
// or -1 for an unsupported shape or a too small part.
int launch_gemm_q4(const uint16_t* A, const uint32_t* Wq, const uint16_t* Sc, const uint8_t* Z, int fmt, float* C,
                   float* part, size_t part_cap, int M, int N, int K, int ldc, gemm_mode mode, hipStream_t s);
size_t gemm_q4_part_floats(int M, int N, int K);
// 1 if the quantized GEMM supports reduction length K.
int gemm_q4_k_ok(int K);
void launch_gemm_f32(const float* A, const float* W, float* C, int M, int N, int K, int ldc,
                     gemm_mode mode, hipStream_t s);
void launch_gemm_q4_f32(const float* A, const uint32_t* Wq, const uint16_t* Sc, const uint8_t* Z, int fmt, float* C,
                        int M, int N, int K, int ldc, gemm_mode mode, hipStream_t s);

// ---- RTN quantizer (kernels_quant.hip): W [N][K] (fp32 or bf16) into the
// packed layout of format fmt, scales Sc and (QF_W4A) zero points Z
void launch_quant(int fmt, const void* W, int w_f32, int N, int K, uint32_t* Wq, uint16_t* Sc, uint8_t* Z,
                  hipStream_t s);

// ---- sampling and acceptance (kernels_sample.hip)
struct rng_t { uint64_t seed, step; };
enum { STREAM_TOKEN = 0, STREAM_ACCEPT = 1, STREAM_RESIDUAL = 2 };
int sample_chunks(int V);
size_t sample_part_floats(int rows, int V);
// Draws one token per row b of logits (row stride ld) with the TOKEN stream at
// position kv_len[slots[b]] + pos_off.  Writes tok[b*tok_stride] and, if
// stats != null, stats[b*stats_stride + {0,1}] = (max, lse) of logits/T.
void launch_sample(const rows_t& r, const float* logits, long ld, int V, float T, rng_t rng,
                   int pos_off, int32_t* tok, int tok_stride, float* stats, int stats_stride,
                   float* part, hipStream_t s);
void launch_accept(const rows_t& r, int gamma, int V, float T, rng_t rng, const int32_t* draft,
                   const float* q_logits, const float* q_stats, const float* p_logits,
                   int32_t* out_tok, int32_t* n_emit, int32_t* next_tok, float* part,
                   float* work, hipStream_t s);
size_t accept_work_floats(int B, int gamma);
size_t accept_part_floats(int B, int gamma, int V);
