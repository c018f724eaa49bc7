// policy.cpp -- host-side SD policy: the roofline cost model (Sec. 3.2
// eq:roofline_basic, Sec. 4.2, App. D.2), the sticky SD toggle
// (eq:sd_speedup_toggle, Algorithm 1), the adaptive draft-length controller
// (Sec. 4.3, Algorithm 1) and the tau <-> alpha relation (Sec. 3.1, App. E.2).
#include <math.h>
#include <string.h>

#include "../../include/sd_api.h"

extern "C" sd_status sd_cost_init(const sd_model_cfg* c, double weight_bytes, double drafter_bits, double kv_bytes,
                                  sd_cost_model* m)
{
    if (!c || !m || weight_bytes <= 0 || drafter_bits <= 0 || kv_bytes <= 0) return SD_E_INVAL;
    double L = c->n_layers, H = c->hidden, d = c->head_dim;
    double attn_params = L * (H * (c->n_q + 2.0 * c->n_kv) * d + c->n_q * d * H);   // Wq,Wk,Wv,Wo
    double ffn_params = L * 3.0 * H * c->ffn;                                        // gate, up, down
    double vocab_params = (double)c->vocab * H;                                      // one of embed / LM head
    memset(m, 0, sizeof *m);
    m->W_T = weight_bytes * (attn_params + ffn_params + 2.0 * vocab_params);
    m->W_D = drafter_bits / 8.0 * (attn_params + ffn_params) + weight_bytes * 2.0 * vocab_params;
    m->kappa_th = L * 2.0 * c->n_kv * d * kv_bytes;
    m->C_dense = 2.0 * (attn_params + ffn_params + vocab_params);
    m->C_attn = 4.0 * L * c->n_q * d;
    m->BW_eff = 8.0e12;
    m->F_eff = 2.5e15;
    m->rho_kappa = 1.0;
    m->eta_D = 1.0;
    return SD_OK;
}

static inline double dmax(double a, double b) { return a > b ? a : b; }

extern "C" sd_status sd_cost_times(const sd_cost_model* m, double B, double S, int32_t gamma, double* Tp, double* Tq,
                                   double* Tv)
{
    if (!m || !Tp || !Tq || !Tv || B < 0 || S < 0 || gamma < 1 || m->BW_eff <= 0 || m->F_eff <= 0)
        return SD_E_INVAL;
    double kv_traffic = m->rho_kappa * m->kappa_th * B * S;
    double mem_target = (m->W_T + kv_traffic) / m->BW_eff;
    double mem_draft = (m->eta_D * m->W_D + kv_traffic) / m->BW_eff;
    double compute = B * (m->C_dense + S * m->C_attn) / m->F_eff;
    *Tp = dmax(mem_target, compute) + m->c_T * B;
    *Tq = dmax(mem_draft, compute) + m->c_D * B;
    *Tv = dmax(mem_target, (gamma + 1.0) * compute) + m->c_V * B;
    return SD_OK;
}

extern "C" int32_t sd_toggle(const sd_cost_model* m, int32_t B, double S_mean, double tau, int32_t gamma, double eps,
                             int32_t* sd_on)
{
    if (!sd_on) return -1;
    if (*sd_on) return 1;   // sticky for the rest of the rollout
    double Tp, Tq, Tv;
    if (sd_cost_times(m, B, S_mean, gamma, &Tp, &Tq, &Tv) != SD_OK || eps < 0) return -1;
    double predicted = tau * Tp / (gamma * Tq + Tv);
    if (predicted >= 1.0 + eps) *sd_on = 1;
    return *sd_on;
}

extern "C" sd_status sd_gamma_init(sd_gamma_ctl* c, const int32_t* set, int32_t n_set, int32_t P, double a_up,
                                   double a_down)
{
    if (!c || !set || n_set < 1 || n_set > 16 || P < 1 || P > 64) return SD_E_INVAL;
    for (int i = 0; i < n_set; ++i)
        if (set[i] < 1 || (i > 0 && set[i] <= set[i - 1])) return SD_E_INVAL;   // ordered, increasing
    memset(c, 0, sizeof *c);
    memcpy(c->set, set, sizeof(int32_t) * n_set);
    c->n_set = n_set;
    c->P = P;
    c->a_up = a_up;
    c->a_down = a_down;
    c->gamma = set[0];   // gamma_1 = gamma_low
    return SD_OK;
}

extern "C" sd_status sd_gamma_next(sd_gamma_ctl* c, double tau_t, int32_t* gamma_next)
{
    if (!c || !gamma_next) return SD_E_INVAL;
    // append to the (bounded) history
    if (c->n_hist == 64) {
        memmove(c->hist, c->hist + 1, sizeof(double) * 63);
        c->n_hist = 63;
    }
    c->hist[c->n_hist++] = tau_t;
    int pos = 0;
    while (pos < c->n_set && c->set[pos] != c->gamma) ++pos;
    if (c->n_hist >= c->P && pos < c->n_set) {
        double lo = INFINITY, hi = -INFINITY;
        for (int i = c->n_hist - c->P; i < c->n_hist; ++i) {
            lo = c->hist[i] < lo ? c->hist[i] : lo;
            hi = c->hist[i] > hi ? c->hist[i] : hi;
        }
        int g = c->gamma;
        if (pos + 1 < c->n_set && lo >= 1.0 + g * c->a_up) c->gamma = c->set[pos + 1];
        else if (pos > 0 && hi <= 1.0 + g * c->a_down) c->gamma = c->set[pos - 1];
    }
    *gamma_next = c->gamma;
    return SD_OK;
}

extern "C" double sd_tau_from_alpha(double alpha, int32_t gamma)
{
    // geometric series 1 + alpha + ... + alpha^gamma
    double t = 0.0, p = 1.0;
    for (int i = 0; i <= gamma; ++i) { t += p; p *= alpha; }
    return t;
}

extern "C" double sd_alpha_from_tau(double tau, int32_t gamma)
{
    if (gamma < 1) return NAN;
    if (tau <= 1.0) return 0.0;
    if (tau >= gamma + 1.0) return 1.0;
    // tau(alpha) is increasing on [0, 1]: Newton from alpha = 1, guarded by bisection
    double lo = 0.0, hi = 1.0, a = 0.5;
    for (int it = 0; it < 100; ++it) {
        double f = sd_tau_from_alpha(a, gamma) - tau;
        if (f > 0) hi = a; else lo = a;
        double df = 0.0, p = 1.0;
        for (int i = 1; i <= gamma; ++i) { df += i * p; p *= a; }
        double nx = df > 0 ? a - f / df : 0.5 * (lo + hi);
        if (!(nx > lo && nx < hi)) nx = 0.5 * (lo + hi);
        if (fabs(nx - a) < 1e-15) { a = nx; break; }
        a = nx;
    }
    return a;
}
