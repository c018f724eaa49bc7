// engine.hip -- the SD engine behind the C ABI (include/sd_api.h): bound
// weights and KV, the engine-owned workspace, and the sequencing of one
// forward pass / draft / verify / accept / rollback on a HIP stream.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <limits.h>

#include <mutex>
#include <string>
#include <vector>

#include "../../include/sd_api.h"
#include "common.h"
#include "kernels.h"

// ------------------------------------------------------------------ errors
static thread_local std::string g_err;

static sd_status fail(sd_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
static sd_status fail(sd_status st, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

extern "C" const char* sd_last_error(void) { return g_err.c_str(); }

#define HIP_TRY(call)                                                                        \
    do {                                                                                     \
        hipError_t e_ = (call);                                                              \
        if (e_ != hipSuccess) return fail(SD_E_HIP, "%s: %s", #call, hipGetErrorString(e_)); \
    } while (0)

static sd_status launched(const char* what)
{
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(SD_E_HIP, "%s: kernel launch failed: %s", what, hipGetErrorString(e));
    return SD_OK;
}

// ------------------------------------------------------------------ engine
enum { PRJ_QKV = 0, PRJ_O = 1, PRJ_GU = 2, PRJ_DOWN = 3 };
enum { T_ATTN_D = 0, T_ATTN_V = 1, T_Q4 = 2, T_PROJ = 3, T_LMHEAD = 4, T_SAMPLE = 5, T_ACCEPT = 6, T_MISC = 7, T_CLASSES = 8 };

struct sd_engine_s {
    sd_model_cfg c;
    int max_slots, max_ctx, max_gamma, rows_max, max_chunks;
    int dev;
    bool f32;
    int poison = 0;
    int no_fuse = 0;             // debug: SwiGLU as its own kernel after the gate/up GEMM
    int no_dma = 0;              // debug: register-staged 320-row GEMM tiles instead of the DMA-fed ones
    // bound (caller-owned)
    std::vector<const void*> w;
    bool weights_bound = false;
    void* k = nullptr;
    void* v = nullptr;
    int32_t* kv_len = nullptr;
    kv_geom geo = {};                  // dense or paged layout of k / v
    std::vector<const uint32_t*> qw;   // [L*4] packed codes
    std::vector<const uint16_t*> qs;   // [L*4] scales
    std::vector<const uint8_t*> qz;    // [L*4] zero points (asymmetric format), else NULL
    int qfmt = QF_W4;                  // format of the last refresh
    bool drafter_ready = false;
    // workspace (engine-owned)
    float* h = nullptr;
    void* a = nullptr;
    float* qkv = nullptr;
    float* qrot = nullptr;
    void* att = nullptr;
    float* gu = nullptr;
    void* act = nullptr;
    float* att_part = nullptr;
    float* samp_part = nullptr;
    float* acc_work = nullptr;
    float2* rope = nullptr;
    uint32_t* err = nullptr;
    int32_t* pf_lim = nullptr;   // [max_slots] rows of one ragged-prefill round
    float* gpart = nullptr;      // split-K partial sums
    size_t gpart_cap = 0;        // floats
    int launch_err = 0;          // a GEMM shape the kernels refused (reported by sd_sync)
    // kernel timing (diagnostics)
    bool timing = false;
    std::vector<hipEvent_t> ev_pool;
    size_t ev_used = 0;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> marks[T_CLASSES];
};

// Brackets the launches made during its lifetime with events of class cls.
struct tscope {
    sd_engine e;
    int cls;
    hipStream_t s;
    hipEvent_t stop = nullptr;
    tscope(sd_engine e_, int cls_, hipStream_t s_) : e(e_), cls(cls_), s(s_)
    {
        if (!e->timing) return;
        hipEvent_t start = next_event(e);
        stop = next_event(e);
        if (!start || !stop) { stop = nullptr; return; }
        (void)hipEventRecord(start, s);
        e->marks[cls].push_back({start, stop});
    }
    ~tscope()
    {
        if (stop) (void)hipEventRecord(stop, s);
    }
    static hipEvent_t next_event(sd_engine e)
    {
        if (e->ev_used == e->ev_pool.size()) {
            hipEvent_t ev;
            if (hipEventCreate(&ev) != hipSuccess) return nullptr;
            e->ev_pool.push_back(ev);
        }
        return e->ev_pool[e->ev_used++];
    }
};

// Times exactly one kernel: the events are handed to the launch, which binds
// them to the kernel's own dispatch, so their elapsed time is the kernel's
// run time with no launch gap (the figure rocprofv3's kernel trace reports).
struct kscope {
    hipEvent_t start = nullptr, stop = nullptr;
    kscope(sd_engine e, int cls)
    {
        if (!e->timing) return;
        start = tscope::next_event(e);
        stop = tscope::next_event(e);
        if (!start || !stop) { start = stop = nullptr; return; }
        e->marks[cls].push_back({start, stop});
    }
};

static void prj_shape(const sd_model_cfg& c, int which, int* N, int* K)
{
    int qkvN = (c.n_q + 2 * c.n_kv) * c.head_dim;
    switch (which) {
        case PRJ_QKV: *N = qkvN; *K = c.hidden; break;
        case PRJ_O: *N = c.hidden; *K = c.n_q * c.head_dim; break;
        case PRJ_GU: *N = 2 * c.ffn; *K = c.hidden; break;
        default: *N = c.hidden; *K = c.ffn; break;
    }
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// bytes of one quantized projection in format fmt: codes, fp16 scales and
// (asymmetric format) one zero-point byte per (column, group), each block
// 256-byte aligned
static size_t prj_bytes(const sd_model_cfg& c, int which, int fmt, size_t* codes, size_t* scales, size_t* zeros)
{
    int N, K;
    prj_shape(c, which, &N, &K);
    *codes = align256(qfmt_code_bytes(fmt, N, K));
    *scales = align256((size_t)N * (K / 128) * 2);
    *zeros = fmt == QF_W4A ? align256((size_t)N * (K / 128)) : 0;
    return *codes + *scales + *zeros;
}

static sd_status check_cfg(const sd_model_cfg* c)
{
    if (!c) return fail(SD_E_INVAL, "cfg is NULL");
    if (c->n_layers < 1 || c->hidden < 1 || c->n_q < 1 || c->n_kv < 1 || c->ffn < 1 || c->vocab < 1)
        return fail(SD_E_INVAL, "model dimensions must be positive");
    if (c->dtype != SD_DTYPE_F32 && c->dtype != SD_DTYPE_BF16) return fail(SD_E_INVAL, "dtype must be F32 or BF16");
    if (c->group != 128) return fail(SD_E_UNSUPPORTED, "group must be 128");
    if (c->head_dim != 64 && c->head_dim != 128) return fail(SD_E_UNSUPPORTED, "head_dim must be 64 or 128");
    if (c->n_q % c->n_kv) return fail(SD_E_INVAL, "n_q must be a multiple of n_kv");
    if (c->hidden % 128 || c->ffn % 128 || (c->n_q * c->head_dim) % 128)
        return fail(SD_E_UNSUPPORTED, "hidden, ffn and n_q*head_dim must be multiples of 128");
    if (((c->n_q + 2 * c->n_kv) * c->head_dim) % 64 || c->vocab % 64)
        return fail(SD_E_UNSUPPORTED, "(n_q+2*n_kv)*head_dim and vocab must be multiples of 64");
    if (!(c->rms_eps > 0.f) || !(c->rope_theta > 0.f)) return fail(SD_E_INVAL, "rms_eps and rope_theta must be > 0");
    if (!gemm_q4_k_ok(c->hidden) || !gemm_q4_k_ok(c->ffn) || !gemm_q4_k_ok(c->n_q * c->head_dim))
        return fail(SD_E_UNSUPPORTED, "hidden, ffn and n_q*head_dim must be 128*g*2^s with g <= 32, s <= 3");
    return SD_OK;
}

extern "C" int32_t sd_num_weights(const sd_model_cfg* c) { return c ? 3 + 6 * c->n_layers : -1; }

extern "C" size_t sd_kv_bytes(const sd_model_cfg* c, int32_t max_slots, int32_t max_ctx)
{
    if (!c) return 0;
    size_t el = c->dtype == SD_DTYPE_F32 ? 4 : 2;
    return (size_t)c->n_layers * max_slots * c->n_kv * (size_t)max_ctx * c->head_dim * el;
}

extern "C" size_t sd_drafter_bytes_fmt(const sd_model_cfg* c, int32_t fmt)
{
    if (!c || fmt < SD_DRAFT_W4 || fmt > SD_DRAFT_W8) return 0;
    size_t total = 0, a, b, z;
    for (int w = 0; w < 4; ++w) total += prj_bytes(*c, w, fmt, &a, &b, &z);
    return total * (size_t)c->n_layers;
}

extern "C" size_t sd_drafter_bytes(const sd_model_cfg* c) { return sd_drafter_bytes_fmt(c, SD_DRAFT_W4); }

// Largest split-K scratch any projection or the LM head needs for up to R rows.
static size_t gpart_bytes(const sd_model_cfg& c, int R)
{
    if (c.dtype == SD_DTYPE_F32) return 256;
    size_t mx = 0;
    for (int M = 1; M <= R; M = (M < 64 ? M + 1 : M + 64)) {
        int m = M > R ? R : M;
        for (int w = 0; w < 4; ++w) {
            int N, K;
            prj_shape(c, w, &N, &K);
            size_t f = gemm_part_floats(m, N, K);
            mx = f > mx ? f : mx;
            f = gemm_q4_part_floats(m, N, K);
            mx = f > mx ? f : mx;
        }
        size_t f = gemm_part_floats(m, c.vocab, c.hidden);
        mx = f > mx ? f : mx;
    }
    for (int w = 0; w < 4; ++w) {
        int N, K;
        prj_shape(c, w, &N, &K);
        size_t f = gemm_part_floats(R, N, K);
        mx = f > mx ? f : mx;
        f = gemm_q4_part_floats(R, N, K);
        mx = f > mx ? f : mx;
    }
    return (mx > 64 ? mx : 64) * 4;
}

static void free_ws(sd_engine e)
{
    void* ps[] = {e->h, e->a, e->qkv, e->qrot, e->att, e->gu, e->act, e->att_part, e->samp_part, e->acc_work, e->rope, e->err,
                  e->pf_lim, e->gpart};
    for (void* p : ps)
        if (p) (void)hipFree(p);
}

extern "C" sd_status sd_create(const sd_model_cfg* cfg, int32_t max_slots, int32_t max_ctx, int32_t max_gamma,
                               sd_engine* out)
{
    sd_status st = check_cfg(cfg);
    if (st != SD_OK) return st;
    if (!out) return fail(SD_E_INVAL, "out is NULL");
    if (max_slots < 1 || max_ctx < 2 || max_gamma < 1 || max_gamma > 64)
        return fail(SD_E_INVAL, "need max_slots >= 1, max_ctx >= 2, 1 <= max_gamma <= 64");
    sd_engine e = new sd_engine_s();
    e->c = *cfg;
    e->max_slots = max_slots;
    e->max_ctx = max_ctx;
    e->max_gamma = max_gamma;
    e->rows_max = max_slots * (max_gamma + 1);
    e->max_chunks = (max_ctx + attention_chunk() - 1) / attention_chunk();
    e->f32 = cfg->dtype == SD_DTYPE_F32;
    e->w.assign(sd_num_weights(cfg), nullptr);
    e->qw.assign(4 * cfg->n_layers, nullptr);
    e->qs.assign(4 * cfg->n_layers, nullptr);
    e->qz.assign(4 * cfg->n_layers, nullptr);
    if (hipGetDevice(&e->dev) != hipSuccess) { delete e; return fail(SD_E_HIP, "hipGetDevice failed"); }

    const sd_model_cfg& c = *cfg;
    size_t R = (size_t)e->rows_max;
    int qkvN = (c.n_q + 2 * c.n_kv) * c.head_dim, qd = c.n_q * c.head_dim;
    struct { void** p; size_t bytes; } allocs[] = {
        {(void**)&e->h, R * c.hidden * 4},
        {(void**)&e->a, R * c.hidden * 4},
        {(void**)&e->qkv, R * qkvN * 4},
        {(void**)&e->qrot, R * qd * 4},
        {(void**)&e->att, R * qd * 4},
        {(void**)&e->gu, R * 2 * (size_t)c.ffn * 4},
        {(void**)&e->act, R * c.ffn * 4},
        {(void**)&e->att_part, attention_part_floats((int)R, c.n_q, c.head_dim, e->max_chunks) * 4},
        {(void**)&e->samp_part, sample_part_floats((int)R, c.vocab) * 4},
        {(void**)&e->acc_work, accept_work_floats(max_slots, max_gamma) * 4},
        {(void**)&e->rope, (size_t)max_ctx * (c.head_dim / 2) * sizeof(float2)},
        {(void**)&e->err, ERR_COUNT * 4},
        {(void**)&e->pf_lim, (size_t)max_slots * 4},
        {(void**)&e->gpart, gpart_bytes(c, e->rows_max)},
    };
    e->gpart_cap = gpart_bytes(c, e->rows_max) / 4;
    for (auto& al : allocs) {
        if (hipMalloc(al.p, al.bytes) != hipSuccess) {
            free_ws(e);
            delete e;
            (void)hipGetLastError();
            return fail(SD_E_NOMEM, "workspace allocation of %zu bytes failed", al.bytes);
        }
    }
    // RoPE table: cos/sin(pos * theta^(-2i/d)) computed in double on the host
    int hd = c.head_dim / 2;
    std::vector<float2> tab((size_t)max_ctx * hd);
    for (int p = 0; p < max_ctx; ++p)
        for (int i = 0; i < hd; ++i) {
            double ang = p * pow((double)c.rope_theta, -2.0 * i / c.head_dim);
            tab[(size_t)p * hd + i] = make_float2((float)cos(ang), (float)sin(ang));
        }
    if (hipMemcpy(e->rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice) != hipSuccess ||
        hipMemset(e->err, 0, ERR_COUNT * 4) != hipSuccess) {
        free_ws(e);
        delete e;
        return fail(SD_E_HIP, "workspace initialisation failed");
    }
    *out = e;
    return SD_OK;
}

extern "C" sd_status sd_destroy(sd_engine e)
{
    if (!e) return fail(SD_E_INVAL, "engine is NULL");
    (void)hipDeviceSynchronize();
    free_ws(e);
    for (hipEvent_t ev : e->ev_pool) (void)hipEventDestroy(ev);
    delete e;
    return SD_OK;
}

extern "C" sd_status sd_bind_weights(sd_engine e, const void* const* t, int32_t n)
{
    if (!e || !t) return fail(SD_E_INVAL, "NULL argument");
    if (n != sd_num_weights(&e->c)) return fail(SD_E_INVAL, "expected %d tensors, got %d", sd_num_weights(&e->c), n);
    for (int i = 0; i < n; ++i) {
        if (!t[i]) return fail(SD_E_INVAL, "tensor %d is NULL", i);
        if ((uintptr_t)t[i] & 15) return fail(SD_E_INVAL, "tensor %d is not 16-byte aligned", i);
    }
    for (int i = 0; i < n; ++i) e->w[i] = t[i];
    e->weights_bound = true;
    e->drafter_ready = false;   // quantized copy is stale until refreshed
    return SD_OK;
}

extern "C" sd_status sd_bind_kv(sd_engine e, void* k, void* v, int32_t* kv_len)
{
    if (!e || !k || !v || !kv_len) return fail(SD_E_INVAL, "NULL argument");
    if (((uintptr_t)k | (uintptr_t)v) & 15) return fail(SD_E_INVAL, "k and v must be 16-byte aligned");
    e->k = k;
    e->v = v;
    e->kv_len = kv_len;
    const long long D = e->c.head_dim, H = e->c.n_kv, C = e->max_ctx;
    e->geo = kv_geom{e->max_ctx, H * C * D, (long long)e->max_slots * H * C * D, C * D, nullptr, 1, e->max_slots};
    return SD_OK;
}

extern "C" size_t sd_kv_page_bytes(const sd_model_cfg* c, int32_t page_size)
{
    if (!c || page_size < 1) return 0;
    size_t el = c->dtype == SD_DTYPE_F32 ? 4 : 2;
    return (size_t)c->n_layers * c->n_kv * (size_t)page_size * c->head_dim * el;
}

extern "C" sd_status sd_bind_kv_paged(sd_engine e, void* k_pages, void* v_pages, int32_t n_pages, int32_t page_size,
                                      const int32_t* block_table, int32_t pages_per_seq, int32_t* kv_len)
{
    if (!e || !k_pages || !v_pages || !block_table || !kv_len) return fail(SD_E_INVAL, "NULL argument");
    if (((uintptr_t)k_pages | (uintptr_t)v_pages) & 15)
        return fail(SD_E_INVAL, "k_pages and v_pages must be 16-byte aligned");
    if (n_pages < 1 || page_size < 32 || page_size % 32)
        return fail(SD_E_INVAL, "need n_pages >= 1 and page_size a positive multiple of 32 (got %d, %d)", n_pages,
                    page_size);
    if (pages_per_seq < 1 || (long long)pages_per_seq * page_size < e->max_ctx)
        return fail(SD_E_INVAL, "pages_per_seq * page_size = %lld must cover max_ctx = %d",
                    (long long)pages_per_seq * page_size, e->max_ctx);
    e->k = k_pages;
    e->v = v_pages;
    e->kv_len = kv_len;
    const long long D = e->c.head_dim, H = e->c.n_kv, L = e->c.n_layers, P = page_size;
    e->geo = kv_geom{page_size, L * H * P * D, H * P * D, P * D, block_table, pages_per_seq, n_pages};
    return SD_OK;
}

extern "C" sd_status sd_set_debug(sd_engine e, int32_t flags)
{
    if (!e) return fail(SD_E_INVAL, "engine is NULL");
    if (flags & ~7) return fail(SD_E_INVAL, "unknown debug flag");
    e->poison = (flags & 1) != 0;
    e->no_fuse = (flags & 2) != 0;
    e->no_dma = (flags & 4) != 0;
    return SD_OK;
}

static const void* W(sd_engine e, int layer, int idx) { return e->w[3 + 6 * layer + idx]; }

extern "C" sd_status sd_refresh_drafter_fmt(sd_engine e, int32_t fmt, void* qbuf, size_t bytes, void* stream)
{
    if (!e || !qbuf) return fail(SD_E_INVAL, "NULL argument");
    if (fmt < SD_DRAFT_W4 || fmt > SD_DRAFT_W8) return fail(SD_E_INVAL, "unknown drafter format %d", fmt);
    if (((uintptr_t)qbuf) & 15) return fail(SD_E_INVAL, "qbuf must be 16-byte aligned");
    if (!e->weights_bound) return fail(SD_E_STATE, "weights not bound");
    const size_t need = sd_drafter_bytes_fmt(&e->c, fmt);
    if (bytes < need) return fail(SD_E_INVAL, "qbuf holds %zu bytes, need %zu", bytes, need);
    e->drafter_ready = false;
    hipStream_t s = (hipStream_t)stream;
    char* p = (char*)qbuf;
    static const int widx[4] = {1, 2, 4, 5};   // Wqkv, Wo, Wgu, Wdown within a layer
    for (int l = 0; l < e->c.n_layers; ++l)
        for (int wh = 0; wh < 4; ++wh) {
            int N, K;
            size_t cb, sb, zb;
            prj_shape(e->c, wh, &N, &K);
            prj_bytes(e->c, wh, fmt, &cb, &sb, &zb);
            uint32_t* q = (uint32_t*)p;
            uint16_t* sc = (uint16_t*)(p + cb);
            uint8_t* z = zb ? (uint8_t*)(p + cb + sb) : nullptr;
            launch_quant(fmt, W(e, l, widx[wh]), e->f32, N, K, q, sc, z, s);
            e->qw[4 * l + wh] = q;
            e->qs[4 * l + wh] = sc;
            e->qz[4 * l + wh] = z;
            p += cb + sb + zb;
        }
    sd_status st = launched("sd_refresh_drafter");
    if (st == SD_OK) {
        e->qfmt = fmt;
        e->drafter_ready = true;
    }
    return st;
}

extern "C" sd_status sd_refresh_drafter(sd_engine e, void* qbuf, size_t bytes, void* stream)
{
    return sd_refresh_drafter_fmt(e, SD_DRAFT_W4, qbuf, bytes, stream);
}

// ------------------------------------------------------------------ forward
static act_t act_of(sd_engine e, bool draft) { return e->f32 ? ACT_F32 : (draft ? ACT_F16 : ACT_BF16); }

// Returns the K splits of a deferred split-K projection (partials in gpart),
// or 1 when C holds the result.
static int proj(sd_engine e, bool draft, int layer, int which, const void* A, float* C, int M, int ldc, gemm_mode mode,
                hipStream_t s)
{
    int N, K;
    prj_shape(e->c, which, &N, &K);
    static const int widx[4] = {1, 2, 4, 5};
    if (draft) {
        const uint32_t* q = e->qw[4 * layer + which];
        const uint16_t* sc = e->qs[4 * layer + which];
        const uint8_t* z = e->qz[4 * layer + which];
        if (e->f32) { launch_gemm_q4_f32((const float*)A, q, sc, z, e->qfmt, C, M, N, K, ldc, mode, s); return 1; }
        const int S = launch_gemm_q4((const uint16_t*)A, q, sc, z, e->qfmt, C, e->gpart, e->gpart_cap, M, N, K, ldc,
                                     mode, s);
        if (S < 1) e->launch_err = 1;   // cannot happen for a configuration check_cfg accepted
        return S < 1 ? 1 : S;
    }
    const void* w = W(e, layer, widx[which]);
    if (e->f32) { launch_gemm_f32((const float*)A, (const float*)w, C, M, N, K, ldc, mode, s); return 1; }
    return launch_gemm_bf16((const uint16_t*)A, (const uint16_t*)w, C, e->gpart, e->gpart_cap, M, N, K, ldc, mode, true, s,
                            !e->no_dma);
}

// The gate/up projection with SwiGLU in its epilogue, writing act directly;
// false when the shape has no fused kernel (or fusion is switched off).
static bool proj_swiglu(sd_engine e, bool draft, int layer, const void* A, void* act, act_t at, int M, hipStream_t s)
{
    if (e->f32 || e->no_fuse) return false;
    const sd_model_cfg& c = e->c;
    if (draft) {
        const int w = 4 * layer + PRJ_GU;
        return launch_gemm_q4_swiglu((const uint16_t*)A, e->qw[w], e->qs[w], e->qz[w], e->qfmt, act, at, M, c.ffn,
                                     c.hidden, s) != 0;
    }
    return launch_gemm_bf16_swiglu((const uint16_t*)A, (const uint16_t*)W(e, layer, 4), act, at, M, c.ffn, c.hidden,
                                   s, !e->no_dma) != 0;
}

// One forward pass over B sequences x n tokens (row r = b*n + i at position
// kv_len + off + i).  Token of row (b, i): i == 0 ? tokA[b*sA] :
// tokB[b*sB + i - 1].  If logits != NULL, row r's logits go to logits + r*ldl;
// otherwise the last layer's FFN (which only feeds the logits) is skipped.
static void forward(sd_engine e, bool draft, int B, const int32_t* slots, const int32_t* tokA, int sA,
                    const int32_t* tokB, int sB, int n, int off, float* logits, long ldl, hipStream_t s,
                    const int32_t* lim = nullptr)
{
    const sd_model_cfg& c = e->c;
    rows_t r = {B, n, off, slots, e->kv_len, e->max_slots, e->max_ctx, e->err};
    r.lim = lim;
    cache_t kv = {e->k, e->v, e->f32 ? 1 : 0, c.n_kv, c.head_dim, e->geo};
    const int R = B * n;
    const act_t at = act_of(e, draft);
    const int qkvN = (c.n_q + 2 * c.n_kv) * c.head_dim;
    const int pcls = draft ? T_Q4 : T_PROJ;
    int S;
    { tscope t(e, T_MISC, s);
      launch_embed_rmsnorm(r, tokA, sA, tokB, sB, e->w[0], e->f32, c.hidden, c.vocab, e->h, W(e, 0, 0), c.rms_eps, e->a, at, s); }
    for (int l = 0; l < c.n_layers; ++l) {
        { tscope t(e, pcls, s); S = proj(e, draft, l, PRJ_QKV, e->a, e->qkv, R, qkvN, GEMM_STORE, s); }
        if (!logits && l == c.n_layers - 1) {
            // the rest of the last layer only feeds the logits: the new K/V rows alone
            tscope t(e, T_MISC, s);
            launch_rope_kv(r, e->qkv, e->gpart, S, e->rope, c.n_q, kv, l, e->qrot, s);
            break;
        }
        attn_split sp;
        { kscope t(e, n == 1 ? T_ATTN_D : T_ATTN_V);      // RoPE and the new K/V rows are part of the attention
          sp = launch_attention(r, qkv_src{e->qkv, e->gpart, S, e->rope}, e->qrot, c.n_q, kv, l, e->att_part,
                                e->max_chunks, e->att, at, s, t.start, t.stop); }
        if (!sp.done) { tscope t(e, T_MISC, s); launch_attention_combine(r, c.n_q, c.head_dim, e->att_part, sp, e->att, at, s); }
        { tscope t(e, pcls, s); S = proj(e, draft, l, PRJ_O, e->att, e->h, R, c.hidden, GEMM_ADD, s); }
        { tscope t(e, T_MISC, s); launch_add_rmsnorm(e->h, e->gpart, S, R, c.hidden, W(e, l, 3), e->f32, c.rms_eps, e->a, at, s); }
        bool fused;
        { tscope t(e, pcls, s); fused = proj_swiglu(e, draft, l, e->a, e->act, at, R, s); }
        if (!fused) {
            { tscope t(e, pcls, s); S = proj(e, draft, l, PRJ_GU, e->a, e->gu, R, 2 * c.ffn, GEMM_STORE, s); }
            { tscope t(e, T_MISC, s); launch_silu_mul(e->gu, e->gpart, S, R, c.ffn, e->act, at, s); }
        }
        { tscope t(e, pcls, s); S = proj(e, draft, l, PRJ_DOWN, e->act, e->h, R, c.hidden, GEMM_ADD, s); }
        // next layer's attention norm, or the final norm (the LM head stays in the target precision)
        const bool last = l == c.n_layers - 1;
        const act_t nt = last ? (e->f32 ? ACT_F32 : ACT_BF16) : at;
        const void* g = last ? e->w[1] : W(e, l + 1, 0);
        { tscope t(e, T_MISC, s); launch_add_rmsnorm(e->h, e->gpart, S, R, c.hidden, g, e->f32, c.rms_eps, e->a, nt, s); }
    }
    if (logits) {
        tscope t(e, T_LMHEAD, s);
        if (e->f32) launch_gemm_f32((const float*)e->a, (const float*)e->w[2], logits, R, c.vocab, c.hidden, (int)ldl, GEMM_STORE, s);
        else launch_gemm_bf16((const uint16_t*)e->a, (const uint16_t*)e->w[2], logits, e->gpart, e->gpart_cap, R, c.vocab,
                                c.hidden, (int)ldl, GEMM_STORE, false, s, !e->no_dma);
    }
}

static sd_status check_step(sd_engine e, int B, const void* slots, bool need_drafter)
{
    if (!e) return fail(SD_E_INVAL, "engine is NULL");
    if (!slots) return fail(SD_E_INVAL, "slots is NULL");
    if (B < 1 || B > e->max_slots) return fail(SD_E_INVAL, "B=%d outside [1, %d]", B, e->max_slots);
    if (!e->weights_bound) return fail(SD_E_STATE, "weights not bound");
    if (!e->kv_len) return fail(SD_E_STATE, "KV cache not bound");
    if (need_drafter && !e->drafter_ready) return fail(SD_E_STATE, "drafter not refreshed");
    return SD_OK;
}

extern "C" sd_status sd_prefill(sd_engine e, int32_t B, const int32_t* slots, const int32_t* tokens, int32_t n,
                                void* stream)
{
    sd_status st = check_step(e, B, slots, false);
    if (st != SD_OK) return st;
    if (!tokens || n < 1) return fail(SD_E_INVAL, "need tokens and n >= 1");
    if (n > e->max_ctx) return fail(SD_E_INVAL, "n=%d exceeds max_ctx=%d", n, e->max_ctx);
    hipStream_t s = (hipStream_t)stream;
    int chunk = e->rows_max / B;
    for (int t0 = 0; t0 < n; t0 += chunk) {
        int nc = n - t0 < chunk ? n - t0 : chunk;
        forward(e, false, B, slots, tokens + t0, n, tokens + t0 + 1, n, nc, 0, nullptr, 0, s);
        launch_kv_advance(B, slots, nullptr, nc, e->kv_len, e->max_slots, e->err, s);
    }
    return launched("sd_prefill");
}

extern "C" sd_status sd_prefill_ragged(sd_engine e, int32_t B, const int32_t* slots, const int32_t* tokens, int32_t ld,
                                       const int32_t* len, void* stream)
{
    sd_status st = check_step(e, B, slots, false);
    if (st != SD_OK) return st;
    if (!tokens || !len) return fail(SD_E_INVAL, "NULL tokens or len");
    if (ld < 1 || ld > e->max_ctx) return fail(SD_E_INVAL, "ld=%d outside [1, max_ctx=%d]", ld, e->max_ctx);
    hipStream_t s = (hipStream_t)stream;
    // rounds of nc positions for the whole batch; row (b, i) of a round is
    // padding once sequence b has no token left (i >= lim[b])
    int chunk = e->rows_max / B;
    for (int t0 = 0; t0 < ld; t0 += chunk) {
        int nc = ld - t0 < chunk ? ld - t0 : chunk;
        launch_prefill_lim(B, len, t0, nc, ld, e->pf_lim, e->err, s);
        forward(e, false, B, slots, tokens + t0, ld, tokens + t0 + 1, ld, nc, 0, nullptr, 0, s, e->pf_lim);
        launch_kv_advance(B, slots, e->pf_lim, 0, e->kv_len, e->max_slots, e->err, s);
    }
    return launched("sd_prefill_ragged");
}

static sd_status check_gamma(sd_engine e, int gamma, float T)
{
    if (gamma < 1 || gamma > e->max_gamma) return fail(SD_E_INVAL, "gamma=%d outside [1, %d]", gamma, e->max_gamma);
    if (!(T > 0.f) || !isfinite(T)) return fail(SD_E_INVAL, "temperature must be finite and > 0");
    return SD_OK;
}

extern "C" sd_status sd_draft(sd_engine e, int32_t B, const int32_t* slots, const int32_t* last_tok, int32_t gamma,
                              float T, sd_rng rng, int32_t* draft_tok, float* q_logits, float* q_stats, void* stream)
{
    sd_status st = check_step(e, B, slots, true);
    if (st != SD_OK) return st;
    if ((st = check_gamma(e, gamma, T)) != SD_OK) return st;
    if (!last_tok || !draft_tok || !q_logits || !q_stats) return fail(SD_E_INVAL, "NULL buffer");
    hipStream_t s = (hipStream_t)stream;
    int V = e->c.vocab;
    rows_t r = {B, 1, 0, slots, e->kv_len, e->max_slots, e->max_ctx, e->err};
    rng_t rg = {rng.seed, rng.step};
    long ld = (long)gamma * V;
    for (int j = 1; j <= gamma; ++j) {
        const int32_t* tok = j == 1 ? last_tok : draft_tok + (j - 2);
        int stride = j == 1 ? 1 : gamma;
        float* lg = q_logits + (size_t)(j - 1) * V;
        forward(e, true, B, slots, tok, stride, tok, stride, 1, j - 1, lg, ld, s);
        tscope t(e, T_SAMPLE, s);
        launch_sample(r, lg, ld, V, T, rg, j, draft_tok + (j - 1), gamma, q_stats + 2 * (j - 1), 2 * gamma,
                      e->samp_part, s);
    }
    return launched("sd_draft");
}

extern "C" sd_status sd_verify(sd_engine e, int32_t B, const int32_t* slots, const int32_t* last_tok,
                               const int32_t* draft_tok, int32_t gamma, float* p_logits, void* stream)
{
    sd_status st = check_step(e, B, slots, false);
    if (st != SD_OK) return st;
    if ((st = check_gamma(e, gamma, 1.0f)) != SD_OK) return st;
    if (!last_tok || !draft_tok || !p_logits) return fail(SD_E_INVAL, "NULL buffer");
    forward(e, false, B, slots, last_tok, 1, draft_tok, gamma, gamma + 1, 0, p_logits, e->c.vocab,
            (hipStream_t)stream);
    return launched("sd_verify");
}

extern "C" sd_status sd_accept(sd_engine e, int32_t B, const int32_t* slots, const int32_t* draft_tok,
                               const float* q_logits, const float* q_stats, const float* p_logits, int32_t gamma,
                               float T, sd_rng rng, int32_t* out_tok, int32_t* n_emit, int32_t* next_tok,
                               void* stream)
{
    sd_status st = check_step(e, B, slots, false);
    if (st != SD_OK) return st;
    if ((st = check_gamma(e, gamma, T)) != SD_OK) return st;
    if (!draft_tok || !q_logits || !q_stats || !p_logits || !out_tok || !n_emit)
        return fail(SD_E_INVAL, "NULL buffer");
    rows_t r = {B, 1, 0, slots, e->kv_len, e->max_slots, e->max_ctx, e->err};
    rng_t rg = {rng.seed, rng.step};
    tscope t(e, T_ACCEPT, (hipStream_t)stream);
    launch_accept(r, gamma, e->c.vocab, T, rg, draft_tok, q_logits, q_stats, p_logits, out_tok, n_emit, next_tok,
                  e->samp_part, e->acc_work, (hipStream_t)stream);
    return launched("sd_accept");
}

// ------------------------------------------------------- accept without allocating
// sd_accept_noalloc's scratch: the rejection sampler's partial results
// (launch_accept's part and work) and its device error words.  One copy per
// GPU, held until the process ends; every call on a GPU shares it, and
// nothing in it has to start at zero (each call writes every partial it later
// reads).  In host code `scratch` names a host-side stand-in: kernels get the
// per-device address from hipGetSymbolAddress instead.
constexpr size_t NOALLOC_FLOATS = (size_t)1 << 20;      // 4 MiB
static __device__ __align__(256) float scratch[NOALLOC_FLOATS];

constexpr int NOALLOC_MAX_DEVICES = 64;
static float* g_scratch_dev[NOALLOC_MAX_DEVICES];
static std::once_flag g_scratch_once[NOALLOC_MAX_DEVICES];
static hipError_t g_scratch_status[NOALLOC_MAX_DEVICES];

// The current device's copy of `scratch`, looked up once per device with that
// device current.
static sd_status noalloc_scratch(float** out)
{
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= NOALLOC_MAX_DEVICES)
        return fail(SD_E_UNSUPPORTED, "device %d beyond the %d this library tracks", dev, NOALLOC_MAX_DEVICES);
    std::call_once(g_scratch_once[dev], [dev] {
        void* p = nullptr;
        g_scratch_status[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch_dev[dev] = (float*)p;
    });
    if (g_scratch_status[dev] != hipSuccess || !g_scratch_dev[dev])
        return fail(SD_E_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                    hipGetErrorString(g_scratch_status[dev]));
    *out = g_scratch_dev[dev];
    return SD_OK;
}

extern "C" sd_status sd_accept_noalloc(int32_t B, int32_t vocab, const int32_t* slots, const int32_t* kv_len,
                                       int32_t max_slots, const int32_t* draft_tok, const float* q_logits,
                                       const float* q_stats, const float* p_logits, int32_t gamma, float T,
                                       sd_rng rng, int32_t* out_tok, int32_t* n_emit, int32_t* next_tok,
                                       void* stream)
{
    if (!slots || !kv_len || !draft_tok || !q_logits || !q_stats || !p_logits || !out_tok || !n_emit)
        return fail(SD_E_INVAL, "NULL buffer");
    if (B < 1 || vocab < 1 || max_slots < 1) return fail(SD_E_INVAL, "need B, vocab, max_slots >= 1");
    if (gamma < 1 || gamma > 64) return fail(SD_E_INVAL, "gamma=%d outside [1, 64]", gamma);
    if (!(T > 0.f) || !isfinite(T)) return fail(SD_E_INVAL, "temperature must be finite and > 0");
    const size_t part = accept_part_floats(B, gamma, vocab), work = accept_work_floats(B, gamma);
    const size_t need = part + work + ERR_COUNT;
    if (need > NOALLOC_FLOATS)
        return fail(SD_E_INVAL, "B=%d, gamma=%d, vocab=%d need %zu scratch floats, the maximum is %zu", B, gamma,
                    vocab, need, NOALLOC_FLOATS);
    float* sc = nullptr;
    sd_status st = noalloc_scratch(&sc);
    if (st != SD_OK) return st;
    rows_t r = {B, 1, 0, slots, kv_len, max_slots, INT_MAX, (uint32_t*)(sc + part + work)};
    rng_t rg = {rng.seed, rng.step};
    launch_accept(r, gamma, vocab, T, rg, draft_tok, q_logits, q_stats, p_logits, out_tok, n_emit, next_tok, sc,
                  sc + part, (hipStream_t)stream);
    return launched("sd_accept_noalloc");
}

extern "C" sd_status kv_rollback(sd_engine e, int32_t B, const int32_t* slots, const int32_t* n_emit, void* stream)
{
    sd_status st = check_step(e, B, slots, false);
    if (st != SD_OK) return st;
    if (!n_emit) return fail(SD_E_INVAL, "n_emit is NULL");
    hipStream_t s = (hipStream_t)stream;
    tscope t(e, T_MISC, s);
    launch_kv_advance(B, slots, n_emit, 0, e->kv_len, e->max_slots, e->err, s);
    if (e->poison) {
        cache_t kv = {e->k, e->v, e->f32 ? 1 : 0, e->c.n_kv, e->c.head_dim, e->geo};
        launch_kv_poison(B, slots, e->kv_len, e->max_gamma + 1, kv, e->c.n_layers, e->max_slots, e->max_ctx, s);
    }
    return launched("kv_rollback");
}

extern "C" sd_status sd_ar_step(sd_engine e, int32_t B, const int32_t* slots, const int32_t* last_tok, float T,
                                sd_rng rng, int32_t* out_tok, float* p_logits, void* stream)
{
    sd_status st = check_step(e, B, slots, false);
    if (st != SD_OK) return st;
    if (!(T > 0.f) || !isfinite(T)) return fail(SD_E_INVAL, "temperature must be finite and > 0");
    if (!last_tok || !out_tok || !p_logits) return fail(SD_E_INVAL, "NULL buffer");
    hipStream_t s = (hipStream_t)stream;
    forward(e, false, B, slots, last_tok, 1, last_tok, 1, 1, 0, p_logits, e->c.vocab, s);
    rows_t r = {B, 1, 0, slots, e->kv_len, e->max_slots, e->max_ctx, e->err};
    rng_t rg = {rng.seed, rng.step};
    { tscope t(e, T_SAMPLE, s); launch_sample(r, p_logits, e->c.vocab, e->c.vocab, T, rg, 1, out_tok, 1, nullptr, 0, e->samp_part, s); }
    { tscope t(e, T_MISC, s); launch_kv_advance(B, slots, nullptr, 1, e->kv_len, e->max_slots, e->err, s); }
    return launched("sd_ar_step");
}

extern "C" sd_status sd_sync(sd_engine e, void* stream)
{
    if (!e) return fail(SD_E_INVAL, "engine is NULL");
    HIP_TRY(hipStreamSynchronize((hipStream_t)stream));
    uint32_t flags[ERR_COUNT];
    HIP_TRY(hipMemcpy(flags, e->err, sizeof flags, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemset(e->err, 0, sizeof flags));
    if (flags[ERR_SLOT]) return fail(SD_E_INVAL, "device: slot index outside [0, max_slots)");
    if (flags[ERR_TOKEN]) return fail(SD_E_INVAL, "device: token id outside [0, vocab)");
    if (flags[ERR_CTX]) return fail(SD_E_INVAL, "device: position at or beyond max_ctx");
    if (flags[ERR_LEN]) return fail(SD_E_INVAL, "device: prefill length outside [0, ld]");
    if (flags[ERR_PAGE]) return fail(SD_E_INVAL, "device: block-table entry outside [0, n_pages)");
    if (e->launch_err) { e->launch_err = 0; return fail(SD_E_UNSUPPORTED, "an int4 GEMM shape was refused"); }
    return SD_OK;
}

extern "C" sd_status sd_dense_gemm_bf16(const void* A, const void* W, float* C, int32_t M, int32_t N, int32_t K,
                                        void* stream)
{
    if (!A || !W || !C) return fail(SD_E_INVAL, "NULL argument");
    if (M < 1 || N < 128 || K < 128 || N % 128 || K % 128)
        return fail(SD_E_UNSUPPORTED, "need M >= 1 and N, K positive multiples of 128");
    launch_gemm_bf16((const uint16_t*)A, (const uint16_t*)W, C, nullptr, 0, M, N, K, N, GEMM_STORE, false,
                     (hipStream_t)stream);
    HIP_TRY(hipGetLastError());
    return SD_OK;
}

extern "C" sd_status sd_timing(sd_engine e, int32_t on)
{
    if (!e) return fail(SD_E_INVAL, "engine is NULL");
    if (on) {
        HIP_TRY(hipDeviceSynchronize());
        for (auto& m : e->marks) m.clear();
        e->ev_used = 0;
    }
    e->timing = on != 0;
    return SD_OK;
}

extern "C" sd_status sd_timing_read(sd_engine e, int32_t cls, double* total_ms, int32_t* launches)
{
    if (!e || !total_ms || !launches) return fail(SD_E_INVAL, "NULL argument");
    if (cls < 0 || cls >= T_CLASSES) return fail(SD_E_INVAL, "timing class %d outside [0, %d)", cls, (int)T_CLASSES);
    double tot = 0.0;
    for (auto& m : e->marks[cls]) {
        HIP_TRY(hipEventSynchronize(m.second));
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, m.first, m.second));
        tot += ms;
    }
    *total_ms = tot;
    *launches = (int32_t)e->marks[cls].size();
    return SD_OK;
}
