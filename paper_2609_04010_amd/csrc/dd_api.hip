// Host side of the C ABI declared in include/dd.h: validation, parameter and workspace layouts,
// kernel dispatch, the T-step loop driver and the launch profiler.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <vector>

#include "kernels.h"

namespace dd {

// ---------------------------------------------------------------- errors
static thread_local char g_err[512] = "";

void set_error(const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
}

dd_status launch_status(const char* what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        set_error("%s: launch failed: %s", what, hipGetErrorString(e));
        return DD_E_HIP;
    }
    return DD_OK;
}

#define DD_TRY(x)                            \
    do {                                     \
        const dd_status st_ = (x);           \
        if (st_ != DD_OK) return st_;        \
    } while (0)

#define DD_CHECK(cond, code, ...)            \
    do {                                     \
        if (!(cond)) {                       \
            set_error(__VA_ARGS__);          \
            return code;                     \
        }                                    \
    } while (0)

// ---------------------------------------------------------------- profiler
static const char* kClassNames[KC_COUNT] = {
    "time_embedding", "embed_layernorm", "layernorm", "gemm_qkv", "attention", "gemm_attn_out",
    "gemm_mlp_up", "gemm_mlp_down", "gemm_vocab", "posterior_sample", "gaussian_latent",
    "init_params", "copy", "compact_masked", "gemm_lora_down"};

// The recorder is the library's only process-wide mutable state: guarded by g_prof_mu, and skipped
// without taking the lock while it is off.
struct Profiler {
    std::atomic<bool> on{false};
    int cap = 0;
    uint32_t mask = 0xFFFFFFFFu;
    std::vector<hipEvent_t> ev;   // 2 per launch
    std::vector<int> cls;         // class per launch
    int open = -1;                // index of the open sample
    bool open_kernel = false;     // its events go with a kernel dispatch (else recorded around)
    int64_t dropped = 0;
};
static Profiler g_prof;
static std::mutex g_prof_mu;

// The event pair a kernel-launch scope opened and its launch has not taken yet (per host thread).
static thread_local hipEvent_t t_pend[2] = {nullptr, nullptr};

void prof_start(int c, hipStream_t s, bool kernel) {
    if (!g_prof.on.load(std::memory_order_relaxed)) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (!g_prof.on || !((g_prof.mask >> c) & 1u)) return;
    const int n = (int)g_prof.cls.size();
    if (n >= g_prof.cap) { g_prof.dropped++; g_prof.open = -1; return; }
    if (kernel) {
        t_pend[0] = g_prof.ev[2 * n];
        t_pend[1] = g_prof.ev[2 * n + 1];
    } else {
        (void)hipEventRecord(g_prof.ev[2 * n], s);
    }
    g_prof.cls.push_back(c);
    g_prof.open = n;
    g_prof.open_kernel = kernel;
}

bool prof_take(hipEvent_t* start, hipEvent_t* stop) {
    if (!t_pend[0]) return false;
    *start = t_pend[0];
    *stop = t_pend[1];
    t_pend[0] = t_pend[1] = nullptr;
    return true;
}

void prof_stop(int c, hipStream_t s) {
    (void)c;
    if (!g_prof.on.load(std::memory_order_relaxed)) {
        t_pend[0] = t_pend[1] = nullptr;
        return;
    }
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (!g_prof.on || g_prof.open < 0) {
        t_pend[0] = t_pend[1] = nullptr;
        return;
    }
    if (g_prof.open_kernel) {
        if (t_pend[0]) {        // the scope launched nothing (an early return): no sample
            t_pend[0] = t_pend[1] = nullptr;
            g_prof.cls.pop_back();
        }                       // else the dispatch recorded both events
    } else {
        (void)hipEventRecord(g_prof.ev[2 * g_prof.open + 1], s);
    }
    g_prof.open = -1;
}

// ---------------------------------------------------------------- layouts
struct Tensor {
    size_t off;
    int64_t rows, cols;
};

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
static size_t esize(int dtype) { return dtype == DD_BF16 ? 2 : 4; }

// The mask id a prior takes: V (the K-th category) under the masked prior, none (-1) under the
// uniform prior.
static dd_status check_mask_id(int prior, int V, int mask_id) {
    const int want = prior == DD_PRIOR_MASK ? V : -1;
    DD_CHECK(mask_id == want, DD_E_UNSUPPORTED, "mask_id %d unsupported for the %s prior (it must be %d)",
             mask_id, prior == DD_PRIOR_MASK ? "masked" : "uniform", want);
    return DD_OK;
}

// Validation of a configuration; sets the error message itself (callers return the status as is).
static dd_status cfg_check(const dd_config* c) {
    DD_CHECK(c, DD_E_ARG, "config is NULL");
    DD_CHECK(c->n_layers >= 0 && c->d_model > 0 && c->n_heads > 0 && c->d_mlp > 0 && c->vocab > 0 &&
                 c->max_len > 0, DD_E_ARG, "config sizes must be positive");
    DD_CHECK(c->d_model % c->n_heads == 0 && c->d_model % 2 == 0, DD_E_ARG,
             "d_model must be even and divisible by n_heads");
    DD_CHECK(c->prior == DD_PRIOR_MASK || c->prior == DD_PRIOR_UNIFORM, DD_E_ARG, "unknown prior");
    DD_CHECK(c->dtype == DD_BF16 || c->dtype == DD_FP32, DD_E_ARG, "unknown dtype");
    DD_CHECK(c->norm == DD_NORM_LAYER || c->norm == DD_NORM_RMS, DD_E_ARG, "unknown norm %d", c->norm);
    DD_CHECK(c->norm_eps >= 0.f, DD_E_ARG, "norm_eps must be >= 0");
    DD_CHECK(c->lora_rank >= 0 && c->lora_rank % 8 == 0, DD_E_ARG,
             "lora_rank must be a non-negative multiple of 8 (got %d)", c->lora_rank);
    DD_CHECK(c->lora_rank == 0 || (c->lora_alpha > 0.f && c->lora_alpha < INFINITY), DD_E_ARG,
             "lora_alpha must be positive and finite");
    return check_mask_id(c->prior, c->vocab, c->mask_id);
}
static bool cfg_ok(const dd_config* c) { return cfg_check(c) == DD_OK; }

static int n_tok(const dd_config* c) { return c->prior == DD_PRIOR_MASK ? c->vocab + 1 : c->vocab; }

// With adapters each projection row holds W[o][:] then B[o][:] (r more columns), so one GEMM over
// K = in + r, with the gated down-projection written beside its input, applies W + g (alpha/r) B A.
static std::vector<Tensor> tensor_list(const dd_config* c) {
    const int64_t d = c->d_model, F = c->d_mlp, V = c->vocab, r = c->lora_rank;
    std::vector<std::pair<int64_t, int64_t>> shapes;
    shapes.push_back({n_tok(c), d});
    shapes.push_back({c->max_len, d});
    for (int l = 0; l < c->n_layers; ++l) {
        shapes.push_back({1, d});          shapes.push_back({1, d});
        shapes.push_back({3 * d, d + r});  shapes.push_back({1, 3 * d});
        shapes.push_back({d, d + r});      shapes.push_back({1, d});
        shapes.push_back({1, d});          shapes.push_back({1, d});
        shapes.push_back({F, d + r});      shapes.push_back({1, F});
        shapes.push_back({d, F + r});      shapes.push_back({1, d});
    }
    shapes.push_back({1, d});
    shapes.push_back({1, d});
    shapes.push_back({V, d});
    if (r > 0)
        for (int l = 0; l < c->n_layers; ++l) {
            shapes.push_back({r, d});  shapes.push_back({r, d});
            shapes.push_back({r, d});  shapes.push_back({r, F});
        }
    std::vector<Tensor> t;
    size_t off = 0;
    const size_t es = esize(c->dtype);
    for (auto& s : shapes) {
        t.push_back({off, s.first, s.second});
        off = align256(off + (size_t)(s.first * s.second) * es);
    }
    return t;
}

static bool is_gain(const dd_config* c, int id) {
    const int nt = 2 + 12 * c->n_layers + 3;
    if (id == nt - 3) return true;                  // lnf_g
    if (id >= 2 && id < 2 + 12 * c->n_layers) {
        const int k = (id - 2) % 12;
        return k == 0 || k == 6;                      // ln1_g, ln2_g
    }
    return false;
}

struct WsLayout {
    size_t err, temb, h, xln, qkv, att, mlp, logits, rows, count, seq, glse, row_lse, total_fwd, total_loop;
    int64_t glse_ld;   // per-group log-sum-exps per logits row (a multiple of 4 floats)
};

// xln, att and mlp (the inputs of the projections) carry r more columns with adapters: the gated
// down-projection g (alpha/r) A a of each row is written there.
static WsLayout ws_layout(const dd_config* c, int64_t M) {
    const size_t es = esize(c->dtype);
    const int64_t d = c->d_model, F = c->d_mlp, r = c->lora_rank;
    WsLayout w;
    size_t off = 0;
    w.err = off; off = align256(off + 4);
    w.temb = off; off = align256(off + (size_t)d * 4);
    w.h = off; off = align256(off + (size_t)(M * d) * 4);
    w.xln = off; off = align256(off + (size_t)(M * (d + r)) * es);
    w.qkv = off; off = align256(off + (size_t)(M * 3 * d) * es);
    w.att = off; off = align256(off + (size_t)(M * (d + r)) * es);
    w.mlp = off; off = align256(off + (size_t)(M * (F + r)) * es);
    w.total_fwd = off;
    w.logits = off;
    const int64_t ld = (c->vocab + 63) / 64 * 64;
    off = align256(off + (size_t)(M * ld) * es);
    w.rows = off; off = align256(off + (size_t)M * 4);
    w.count = off; off = align256(off + 4);
    w.seq = off; off = align256(off + (size_t)(M + 1) * 4);   // per-sequence list starts (B + 1 <= M + 1)
    w.glse_ld = ((c->vocab + DD_GUMBEL_GROUP - 1) / DD_GUMBEL_GROUP + 3) / 4 * 4;
    w.glse = off; off = align256(off + (size_t)(M * w.glse_ld) * 4);
    w.row_lse = off; off = align256(off + (size_t)M * 4);
    w.total_loop = off;
    return w;
}

static dd_status forward_check(const dd_config* c) {
    const int dh = c->d_model / c->n_heads;
    DD_CHECK(ln_supported(c->d_model), DD_E_UNSUPPORTED,
             "d_model %d: LayerNorm kernels need d_model %% 64 == 0 and d_model <= 2048", c->d_model);
    DD_CHECK(attn_supported(c->dtype, dh), DD_E_UNSUPPORTED,
             "head dim %d unsupported for this dtype (bf16: 64; fp32: 16/32/64/128)", dh);
    DD_CHECK(c->d_mlp % 8 == 0, DD_E_UNSUPPORTED, "d_mlp must be a multiple of 8");
    return DD_OK;
}

// vocab_rows / vocab_count (device, nullable): restrict the vocabulary projection to the listed
// rows, written compacted (row j of `logits` belongs to token row vocab_rows[j]).
// attn_mask (device [3L], nullable): visibility pattern; lora_gate (device [L], nullable): adapter
// gate per position (all on when NULL).  vocab_lse (device, nullable; bf16 with d % 128 == 0): the
// vocabulary projection also writes each logits row's per-group log-sum-exps there, row stride
// lse_ld.
static dd_status run_forward(const dd_config* c, const void* params, const int32_t* z, int32_t B,
                             int32_t L, double alpha_t, void* logits, int64_t ld, char* ws,
                             hipStream_t s, const int32_t* vocab_rows = nullptr,
                             const int32_t* vocab_count = nullptr,
                             const int32_t* attn_mask = nullptr, const int32_t* lora_gate = nullptr,
                             float* vocab_lse = nullptr, int64_t lse_ld = 0,
                             int32_t* vocab_cand = nullptr, uint64_t cand_seed = 0,
                             uint32_t cand_step = 0, const int32_t* vocab_seq = nullptr) {
    const std::vector<Tensor> T = tensor_list(c);
    const WsLayout w = ws_layout(c, (int64_t)B * L);
    const char* P = (const char*)params;
    auto tp = [&](int id) -> const void* { return P + T[id].off; };
    const int d = c->d_model, F = c->d_mlp, H = c->n_heads, V = c->vocab, nl = c->n_layers;
    const int64_t M = (int64_t)B * L;
    const int dt = c->dtype;
    const size_t es = esize(dt);
    int32_t* err = (int32_t*)(ws + w.err);
    float* temb = (float*)(ws + w.temb);
    float* h = (float*)(ws + w.h);
    void* xln = ws + w.xln;
    void* qkv = ws + w.qkv;
    void* att = ws + w.att;
    void* mlp = ws + w.mlp;
    const int lnf = 2 + 12 * nl;
    const int r = c->lora_rank;
    const int dr = d + r, Fr = F + r;     // row strides of the projection inputs
    const float lscale = r > 0 ? c->lora_alpha / (float)r : 0.f;
    // adapter down-projection of `in` (row stride ldin, width kin) by A (id a_id), gated and scaled,
    // into the r columns after the input
    auto lora_down = [&](void* in, int64_t ldin, int kin, int a_id) -> dd_status {
        GemmArgs g = {in, ldin, tp(a_id), kin, nullptr, (char*)in + (size_t)kin * es, ldin, (int)M, r, kin,
                      nullptr, nullptr, lora_gate, L, lscale};
        return launch_gemm(dt, EPI_GATE, KC_GEMM_LORA, g, s);
    };

    // With vocab_rows only the listed rows get logits.  In the last layer only the attention's keys
    // and values mix rows, so from its queries on that layer runs on the listed rows alone,
    // compacted (row j is token row vocab_rows[j]; vocab_seq gives each sequence's first list
    // index): the attention takes the listed queries, and the attention-output projection adds the
    // listed residual rows and writes them into the q|k|v buffer, which the attention has finished
    // with (fp32 d per row fits in bf16 3d).
    const bool tail_rows = vocab_rows && vocab_count && vocab_seq && r == 0 && nl > 0 && dt == DD_BF16 &&
                           !attn_mask && gemm_gather_supported(dt, d) && gemm_gather_supported(dt, F);
    if (c->time_cond) DD_TRY(launch_temb(temb, d, 1000.0 * (1.0 - alpha_t), s));
    const int g0 = nl > 0 ? 2 : lnf;
    DD_TRY(launch_embed_ln(dt, c->norm, z, M, L, n_tok(c), d, tp(0), tp(1), c->time_cond ? temb : nullptr,
                           tp(g0), tp(g0 + 1), c->norm_eps, h, xln, dr, err, s));
    for (int l = 0; l < nl; ++l) {
        const int b = 2 + 12 * l;
        const int a0 = lnf + 3 + 4 * l;   // this layer's A matrices (adapters only)
        GemmArgs g;
        if (r > 0) DD_TRY(lora_down(xln, dr, d, a0));
        g = {xln, dr, tp(b + 2), dr, tp(b + 3), qkv, 3 * d, (int)M, 3 * d, dr, nullptr, nullptr};
        DD_TRY(launch_gemm(dt, EPI_BIAS, KC_GEMM_QKV, g, s));
        AttnArgs aa = {qkv, 3 * d, att, dr, B, L, H, d,
                       (float)(1.4426950408889634 / sqrt((double)(d / H))), attn_mask, err};
        const bool tail = tail_rows && l + 1 == nl;
        if (tail) {
            aa.qrows = vocab_rows;
            aa.qseq = vocab_seq;
        }
        DD_TRY(launch_attn(dt, aa, s));
        if (tail) {
            // The listed rows are few in most steps (about M / T from an all-mask start), where the
            // 256-row tiles leave most CUs idle through a whole K loop.  Each of these GEMMs is
            // launched twice, gated on the device-side count: the shape's usual tiles above
            // TAIL_ROWS rows, 64 x 32 tiles of one wavefront up to it (several workgroups per CU;
            // 4.172 -> 4.159 ms per reverse step against 64 x 128 tiles of four wavefronts).
            constexpr int TAIL_ROWS = 2048;
            auto gated = [&](GemmArgs ga, int epi, int cls) -> dd_status {
                ga.m_gate = TAIL_ROWS;
                ga.m_side = 0;
                DD_TRY(launch_gemm(dt, epi, cls, ga, s));
                ga.m_side = 1;
                ga.tile_hint = 10 + 1;
                return launch_gemm(dt, epi, cls, ga, s);
            };
            float* hc = (float*)qkv;
            g = {att, dr, tp(b + 4), dr, tp(b + 5), hc, d, (int)M, d, dr, nullptr, vocab_count};
            g.c_in = h;
            g.c_rows = vocab_rows;
            DD_TRY(gated(g, EPI_BIAS_RESID, KC_GEMM_O));
            DD_TRY(launch_ln(dt, c->norm, hc, M, d, tp(b + 6), tp(b + 7), c->norm_eps, xln, dr, s, vocab_count));
            g = {xln, dr, tp(b + 8), dr, tp(b + 9), mlp, Fr, (int)M, F, dr, nullptr, vocab_count};
            DD_TRY(gated(g, EPI_BIAS_GELU, KC_GEMM_MLP1));
            g = {mlp, Fr, tp(b + 10), Fr, tp(b + 11), hc, d, (int)M, d, Fr, nullptr, vocab_count};
            DD_TRY(gated(g, EPI_BIAS_RESID, KC_GEMM_MLP2));
            DD_TRY(launch_ln(dt, c->norm, hc, M, d, tp(lnf), tp(lnf + 1), c->norm_eps, xln, dr, s, vocab_count));
            break;
        }
        if (r > 0) DD_TRY(lora_down(att, dr, d, a0 + 1));
        g = {att, dr, tp(b + 4), dr, tp(b + 5), h, d, (int)M, d, dr, nullptr, nullptr};
        DD_TRY(launch_gemm(dt, EPI_BIAS_RESID, KC_GEMM_O, g, s));
        DD_TRY(launch_ln(dt, c->norm, h, M, d, tp(b + 6), tp(b + 7), c->norm_eps, xln, dr, s));
        if (r > 0) DD_TRY(lora_down(xln, dr, d, a0 + 2));
        g = {xln, dr, tp(b + 8), dr, tp(b + 9), mlp, Fr, (int)M, F, dr, nullptr, nullptr};
        DD_TRY(launch_gemm(dt, EPI_BIAS_GELU, KC_GEMM_MLP1, g, s));
        if (r > 0) DD_TRY(lora_down(mlp, Fr, F, a0 + 3));
        g = {mlp, Fr, tp(b + 10), Fr, tp(b + 11), h, d, (int)M, d, Fr, nullptr, nullptr};
        DD_TRY(launch_gemm(dt, EPI_BIAS_RESID, KC_GEMM_MLP2, g, s));
        const int gn = (l + 1 < nl) ? b + 12 : lnf;
        DD_TRY(launch_ln(dt, c->norm, h, M, d, tp(gn), tp(gn + 1), c->norm_eps, xln, dr, s));
    }
    // with vocab_rows only the listed rows (count on the device) get logits, compacted; after the
    // compacted last layer the normalised rows are already in list order
    GemmArgs g = {xln, dr, tp(lnf + 2), d, nullptr, logits, ld, (int)M, V, d,
                  tail_rows ? nullptr : vocab_rows, vocab_count};
    g.row_ids = tail_rows ? vocab_rows : nullptr;
    g.lse = vocab_lse;
    g.lse_ld = lse_ld;
    g.cand = vocab_cand;
    g.cand_ld = lse_ld;
    g.seed = cand_seed;
    g.step = cand_step;
    g.row0 = 0;
    DD_TRY(launch_gemm(dt, vocab_cand ? EPI_LSE_CDF : vocab_lse ? EPI_LSE : EPI_PLAIN, KC_GEMM_VOCAB, g, s));
    (void)es;
    return DD_OK;
}

static dd_status check_schedule(double at, double as) {
    DD_CHECK(at >= 0.0 && as <= 1.0 && at < as, DD_E_ARG,
             "schedule values must satisfy 0 <= alpha_t < alpha_s <= 1 (got %.17g, %.17g)", at, as);
    return DD_OK;
}

static int32_t ntop_of(int prior, int V) {
    return (V + DD_GUMBEL_GROUP - 1) / DD_GUMBEL_GROUP + (prior == DD_PRIOR_MASK ? 1 : 0);
}

// Coefficients of the Psi transition (App. A.4, eq. (psi-sampler) in the closed forms eqs.
// (psi-mdm), (psi-usdm)); kappa = 1 is the ancestral posterior (App. A.1 / A.2).  Each term is
// written as its kappa = 1 value plus a (1 - kappa) correction, so kappa = 1 reproduces the
// ancestral coefficients bit for bit.
static PostArgs make_post(int prior, const void* logits, int64_t ld, int32_t rows, int32_t V,
                          const int32_t* z_t, double at, double as, double kappa,
                          const uint32_t* noise, uint64_t seed, uint32_t step, uint32_t row0,
                          int32_t* z_s, float* row_lse, float* probs, int32_t* err) {
    PostArgs a;
    memset(&a, 0, sizeof(a));
    a.logits = logits; a.ld = ld; a.rows = rows; a.V = V; a.prior = prior;
    a.z_t = z_t; a.z_s = z_s;
    const double omk = 1.0 - kappa;
    if (prior == DD_PRIOR_MASK) {
        // masked rows: (a_s - k a_t (1 - a_s)/(1 - a_t)) x + (1 - a_s + k a_t (1 - a_s)/(1 - a_t)) m
        const double corr = omk * at * (1.0 - as) / (1.0 - at);
        a.wx = (as - at) / (1.0 - at) + corr;
        a.wm = (1.0 - as) / (1.0 - at) - corr;
        a.log_wx = log(a.wx);
        // unmasked rows (x_theta = one-hot of the token): keep a_s + k (1 - a_s), remask the rest
        a.rmask = omk * (1.0 - as);
        a.keep = 1.0 - a.rmask;
        a.remask = a.rmask > 0.0;
    } else {
        const double K = (double)V, ats = at / as;
        const double cu1 = (1.0 - ats) * (1.0 - as) / K;
        a.c_x = (as - at) + omk * at * (1.0 - as);
        a.c_u = cu1 - omk * cu1;
        a.u1 = omk * (1.0 - as) / K;
        a.c_z = (ats - at) - omk * (1.0 - as) * ats;
        a.Ka_t = K * at;
        a.Ka_r = K * at * (1.0 - omk * (1.0 - as));
        a.one_m_at = 1.0 - at;
    }
    a.noise = noise;
    a.ntop = ntop_of(prior, V);
    a.nu = a.ntop + V;
    a.seed = seed; a.step = step; a.row0 = row0;
    a.probs = probs; a.err = err;
    a.row_lse = row_lse;
    return a;
}

__global__ void fill_i32_kernel(int32_t* p, int32_t v, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

}  // namespace dd

using namespace dd;

extern "C" {

const char* dd_status_str(dd_status s) {
    switch (s) {
        case DD_OK: return "ok";
        case DD_E_ARG: return "invalid argument";
        case DD_E_SHAPE: return "inconsistent shape";
        case DD_E_DTYPE: return "unknown dtype";
        case DD_E_WORKSPACE: return "buffer too small";
        case DD_E_HIP: return "HIP runtime error";
        case DD_E_UNSUPPORTED: return "unsupported configuration";
        case DD_E_DEVICE: return "device error word set";
    }
    return "unknown status";
}

const char* dd_last_error(void) { return g_err; }

int32_t dd_param_count(const dd_config* cfg) {
    if (!cfg_ok(cfg)) return 0;
    return 2 + 12 * cfg->n_layers + 3 + (cfg->lora_rank > 0 ? 4 * cfg->n_layers : 0);
}

dd_status dd_param_tensor(const dd_config* cfg, int32_t id, size_t* offset_bytes, int64_t* rows,
                          int64_t* cols) {
    DD_TRY(cfg_check(cfg));
    DD_CHECK(offset_bytes && rows && cols, DD_E_ARG, "output pointers must not be NULL");
    const std::vector<Tensor> t = tensor_list(cfg);
    DD_CHECK(id >= 0 && id < (int32_t)t.size(), DD_E_ARG, "tensor id %d out of range", id);
    *offset_bytes = t[id].off;
    *rows = t[id].rows;
    *cols = t[id].cols;
    return DD_OK;
}

size_t dd_param_bytes(const dd_config* cfg) {
    if (!cfg_ok(cfg)) return 0;
    const std::vector<Tensor> t = tensor_list(cfg);
    const Tensor& l = t.back();
    return align256(l.off + (size_t)(l.rows * l.cols) * esize(cfg->dtype));
}

size_t dd_workspace_bytes(const dd_config* cfg, int32_t B, int32_t L) {
    if (!cfg_ok(cfg) || B <= 0 || L <= 0) return 0;
    return ws_layout(cfg, (int64_t)B * L).total_fwd;
}

size_t dd_loop_workspace_bytes(const dd_config* cfg, int32_t B, int32_t L) {
    if (!cfg_ok(cfg) || B <= 0 || L <= 0) return 0;
    return ws_layout(cfg, (int64_t)B * L).total_loop;
}

int64_t dd_logits_ld(int32_t V) { return V <= 0 ? 0 : ((int64_t)V + 63) / 64 * 64; }

int32_t dd_noise_width(int32_t prior, int32_t V) {
    if (V <= 0 || (prior != DD_PRIOR_MASK && prior != DD_PRIOR_UNIFORM)) return 0;
    return ntop_of(prior, V) + V;
}

dd_status dd_workspace_reset(void* ws, void* stream) {
    DD_CHECK(ws, DD_E_ARG, "workspace is NULL");
    launch_k(fill_i32_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream, (int32_t*)ws, 0,
                       (int64_t)1);
    return launch_status("workspace_reset");
}

dd_status dd_read_device_error(const int32_t* err_word, int32_t* code_out, void* stream) {
    DD_CHECK(err_word && code_out, DD_E_ARG, "NULL pointer");
    hipError_t e = hipStreamSynchronize((hipStream_t)stream);
    if (e == hipSuccess) e = hipMemcpy(code_out, err_word, sizeof(int32_t), hipMemcpyDeviceToHost);
    DD_CHECK(e == hipSuccess, DD_E_HIP, "read_device_error: %s", hipGetErrorString(e));
    return *code_out ? DD_E_DEVICE : DD_OK;
}

dd_status dd_init_params(const dd_config* cfg, void* params, size_t params_bytes, uint64_t seed,
                         const void* host_src, void* stream) {
    DD_TRY(cfg_check(cfg));
    DD_CHECK(params, DD_E_ARG, "params is NULL");
    const size_t need = dd_param_bytes(cfg);
    DD_CHECK(params_bytes >= need, DD_E_WORKSPACE, "parameter buffer has %zu bytes, needs %zu",
             params_bytes, need);
    hipStream_t s = (hipStream_t)stream;
    if (host_src) {
        const hipError_t e = hipMemcpyAsync(params, host_src, need, hipMemcpyHostToDevice, s);
        DD_CHECK(e == hipSuccess, DD_E_HIP, "init_params copy: %s", hipGetErrorString(e));
        return DD_OK;
    }
    const std::vector<Tensor> t = tensor_list(cfg);
    for (int id = 0; id < (int)t.size(); ++id) {
        DD_TRY(launch_init((char*)params + t[id].off, t[id].rows * t[id].cols, (uint32_t)id,
                           is_gain(cfg, id) ? 1.0 : 0.0, cfg->dtype == DD_BF16, seed, s));
    }
    return DD_OK;
}

dd_status dd_attn_mask_build(int32_t pattern, int32_t L, int32_t block, int32_t* out) {
    DD_CHECK(out, DD_E_ARG, "out is NULL");
    DD_CHECK(L > 0, DD_E_ARG, "L must be positive");
    DD_CHECK(pattern >= DD_ATTN_BIDIRECTIONAL && pattern <= DD_ATTN_DRAFT_TRAIN, DD_E_ARG,
             "unknown attention pattern %d", pattern);
    if (pattern == DD_ATTN_BLOCK_CAUSAL || pattern == DD_ATTN_DRAFT_TRAIN)
        DD_CHECK(block >= 1, DD_E_ARG, "block must be >= 1");
    if (pattern == DD_ATTN_DRAFT_TRAIN)
        DD_CHECK(L % 2 == 0 && (L / 2) % block == 0, DD_E_SHAPE,
                 "the [x, z_1] pattern needs L even and L/2 a multiple of block (L = %d, block = %d)", L, block);
    int32_t* pre = out;
    int32_t* lo = out + L;
    int32_t* hi = out + 2 * (int64_t)L;
    const int32_t n = L / 2;
    for (int32_t i = 0; i < L; ++i) {
        lo[i] = hi[i] = 0;
        switch (pattern) {
            case DD_ATTN_BIDIRECTIONAL: pre[i] = L; break;
            case DD_ATTN_CAUSAL: pre[i] = i + 1; break;
            case DD_ATTN_BLOCK_CAUSAL: pre[i] = (int32_t)std::min<int64_t>(L, ((int64_t)i / block + 1) * block); break;
            default:
                if (i < n) {             // clean token: causal within x
                    pre[i] = i + 1;
                } else {                 // token l of noisy block b: x^(<b), then its block up to itself
                    const int32_t b = (i - n) / block;
                    pre[i] = b * block;
                    lo[i] = n + b * block;
                    hi[i] = i + 1;
                }
        }
    }
    return DD_OK;
}

dd_status dd_denoise_forward_ex(const dd_config* cfg, const void* params, const int32_t* z_t,
                                int32_t B, int32_t L, double alpha_t, const int32_t* attn_mask,
                                const int32_t* lora_gate, void* logits, int64_t ld, void* ws,
                                size_t ws_bytes, void* stream) {
    DD_TRY(cfg_check(cfg));
    DD_CHECK(!lora_gate || cfg->lora_rank > 0, DD_E_ARG, "lora_gate given for a model without adapters");
    DD_CHECK(params && z_t && logits && ws, DD_E_ARG, "NULL pointer argument");
    DD_CHECK(B > 0 && L > 0, DD_E_ARG, "B and L must be positive");
    DD_CHECK(L <= cfg->max_len, DD_E_SHAPE, "L = %d exceeds max_len = %d", L, cfg->max_len);
    DD_CHECK(alpha_t >= 0.0 && alpha_t <= 1.0, DD_E_ARG, "alpha_t must lie in [0, 1]");
    DD_CHECK(ld >= cfg->vocab && ld % 8 == 0, DD_E_SHAPE, "ld must be >= V and a multiple of 8");
    DD_CHECK(((uintptr_t)logits & 15) == 0 && ((uintptr_t)ws & 255) == 0 && ((uintptr_t)params & 255) == 0,
             DD_E_ARG, "logits must be 16-byte aligned, params and ws 256-byte aligned");
    DD_TRY(forward_check(cfg));
    const size_t need = dd_workspace_bytes(cfg, B, L);
    DD_CHECK(ws_bytes >= need, DD_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
    return run_forward(cfg, params, z_t, B, L, alpha_t, logits, ld, (char*)ws, (hipStream_t)stream,
                       nullptr, nullptr, attn_mask, lora_gate);
}

dd_status dd_denoise_forward(const dd_config* cfg, const void* params, const int32_t* z_t,
                             int32_t B, int32_t L, double alpha_t, void* logits, int64_t ld,
                             void* ws, size_t ws_bytes, void* stream) {
    DD_TRY(cfg_check(cfg));
    DD_CHECK(params && z_t && logits && ws, DD_E_ARG, "NULL pointer argument");
    DD_CHECK(B > 0 && L > 0, DD_E_ARG, "B and L must be positive");
    DD_CHECK(L <= cfg->max_len, DD_E_SHAPE, "L = %d exceeds max_len = %d", L, cfg->max_len);
    DD_CHECK(alpha_t >= 0.0 && alpha_t <= 1.0, DD_E_ARG, "alpha_t must lie in [0, 1]");
    DD_CHECK(ld >= cfg->vocab && ld % 8 == 0, DD_E_SHAPE, "ld must be >= V and a multiple of 8");
    DD_CHECK(((uintptr_t)logits & 15) == 0 && ((uintptr_t)ws & 255) == 0 && ((uintptr_t)params & 255) == 0,
             DD_E_ARG, "logits must be 16-byte aligned, params and ws 256-byte aligned");
    DD_TRY(forward_check(cfg));
    const size_t need = dd_workspace_bytes(cfg, B, L);
    DD_CHECK(ws_bytes >= need, DD_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
    return run_forward(cfg, params, z_t, B, L, alpha_t, logits, ld, (char*)ws, (hipStream_t)stream);
}

dd_status dd_psi_posterior_sample(int32_t prior, const void* logits, int32_t logits_dtype, int64_t ld,
                                  int32_t rows, int32_t V, int32_t mask_id, const int32_t* z_t,
                                  double alpha_t, double alpha_s, double kappa,
                                  const uint32_t* noise_words, uint64_t seed, uint32_t step,
                                  uint32_t row0, int32_t* z_s, float* row_lse, float* probs,
                                  int32_t* dev_err, void* stream) {
    DD_CHECK(prior == DD_PRIOR_MASK || prior == DD_PRIOR_UNIFORM, DD_E_ARG, "unknown prior %d", prior);
    DD_CHECK(logits_dtype == DD_BF16 || logits_dtype == DD_FP32, DD_E_DTYPE, "unknown logits dtype");
    DD_CHECK(rows >= 0 && V > 0, DD_E_ARG, "rows must be >= 0 and V > 0");
    DD_CHECK(V <= (1 << 24), DD_E_UNSUPPORTED, "V > 2^24 unsupported");
    DD_TRY(check_mask_id(prior, V, mask_id));
    DD_CHECK(ld >= V && ld % 8 == 0, DD_E_SHAPE, "ld must be >= V and a multiple of 8");
    DD_TRY(check_schedule(alpha_t, alpha_s));
    DD_CHECK(kappa >= 0.0 && kappa <= 1.0, DD_E_ARG, "kappa must lie in [0, 1] (got %.17g)", kappa);
    if (rows == 0) return DD_OK;
    DD_CHECK(logits && z_t && z_s, DD_E_ARG, "NULL pointer argument");
    const PostArgs a = make_post(prior, logits, ld, rows, V, z_t, alpha_t, alpha_s, kappa, noise_words,
                                 seed, step, row0, z_s, row_lse, probs, dev_err);
    return launch_posterior(a, logits_dtype, (hipStream_t)stream);
}

dd_status dd_posterior_sample(int32_t prior, const void* logits, int32_t logits_dtype, int64_t ld,
                              int32_t rows, int32_t V, int32_t mask_id, const int32_t* z_t,
                              double alpha_t, double alpha_s, const uint32_t* noise_words,
                              uint64_t seed, uint32_t step, uint32_t row0, int32_t* z_s,
                              float* row_lse, float* probs, int32_t* dev_err, void* stream) {
    return dd_psi_posterior_sample(prior, logits, logits_dtype, ld, rows, V, mask_id, z_t, alpha_t, alpha_s,
                                   1.0, noise_words, seed, step, row0, z_s, row_lse, probs, dev_err, stream);
}

dd_status dd_loop_workspace_layout(const dd_config* cfg, int32_t B, int32_t L, dd_loop_ws_layout* out) {
    DD_TRY(cfg_check(cfg));
    DD_CHECK(B > 0 && L > 0 && out, DD_E_ARG, "B and L must be positive and out non-NULL");
    const WsLayout w = ws_layout(cfg, (int64_t)B * L);
    out->err = w.err;
    out->logits = w.logits;
    out->rows = w.rows;
    out->count = w.count;
    out->glse = w.glse;
    out->cand = w.logits;
    out->row_lse = w.row_lse;
    out->logits_ld = dd_logits_ld(cfg->vocab);
    out->glse_ld = w.glse_ld;
    return DD_OK;
}

dd_status dd_psi_sample_loop(const dd_config* cfg, const void* params, int32_t B, int32_t L,
                             int32_t T, const double* alphas, const double* kappas, uint32_t flags,
                             int32_t* z, const uint32_t* noise_words, uint64_t noise_seed,
                             int32_t* z_trace, void* ws, size_t ws_bytes, void* stream) {
    DD_TRY(cfg_check(cfg));
    DD_CHECK((flags & ~(DD_LOOP_POSTERIOR_PASS | DD_LOOP_STORE_FREE)) == 0, DD_E_ARG, "unknown loop flags 0x%x",
             flags);
    const bool store_free = (flags & DD_LOOP_STORE_FREE) != 0;
    DD_CHECK(!store_free || !(flags & DD_LOOP_POSTERIOR_PASS), DD_E_ARG,
             "DD_LOOP_STORE_FREE and DD_LOOP_POSTERIOR_PASS exclude each other");
    DD_CHECK(!store_free || (cfg->prior == DD_PRIOR_MASK && gemm_lse_supported(cfg->dtype, cfg->d_model) &&
                             gemm_gather_supported(cfg->dtype, cfg->d_model)),
             DD_E_UNSUPPORTED, "DD_LOOP_STORE_FREE needs the masked prior, bf16 and d_model %% 128 == 0");
    DD_CHECK(!store_free || !noise_words, DD_E_UNSUPPORTED, "DD_LOOP_STORE_FREE draws Philox noise only");
    DD_CHECK(params && z && ws && alphas, DD_E_ARG, "NULL pointer argument");
    DD_CHECK(B > 0 && L > 0 && T > 0, DD_E_ARG, "B, L and T must be positive");
    DD_CHECK(L <= cfg->max_len, DD_E_SHAPE, "L = %d exceeds max_len = %d", L, cfg->max_len);
    DD_TRY(forward_check(cfg));
    DD_CHECK(((uintptr_t)ws & 255) == 0 && ((uintptr_t)params & 255) == 0, DD_E_ARG,
             "params and ws must be 256-byte aligned");
    for (int k = 1; k <= T; ++k) DD_TRY(check_schedule(alphas[k], alphas[k - 1]));
    if (kappas)
        for (int k = 1; k <= T; ++k)
            DD_CHECK(kappas[k] >= 0.0 && kappas[k] <= 1.0, DD_E_ARG, "kappas[%d] = %.17g is outside [0, 1]",
                     k, kappas[k]);
    const size_t need = dd_loop_workspace_bytes(cfg, B, L);
    DD_CHECK(ws_bytes >= need, DD_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
    hipStream_t s = (hipStream_t)stream;
    const int64_t M = (int64_t)B * L;
    const WsLayout w = ws_layout(cfg, M);
    char* wsc = (char*)ws;
    void* logits = wsc + w.logits;
    const int64_t ld = dd_logits_ld(cfg->vocab);
    const int32_t nu = dd_noise_width(cfg->prior, cfg->vocab);
    auto trace_copy = [&](int slot) -> dd_status {
        if (!z_trace) return DD_OK;
        ProfScope ps(KC_COPY, s, false);
        const hipError_t e = hipMemcpyAsync(z_trace + (int64_t)slot * M, z, M * sizeof(int32_t),
                                            hipMemcpyDeviceToDevice, s);
        DD_CHECK(e == hipSuccess, DD_E_HIP, "trace copy: %s", hipGetErrorString(e));
        return DD_OK;
    };
    // Masked prior: rows already unmasked are carried over and need no logits, so the vocabulary
    // projection and the draw run on the compacted list of still-masked rows (same per-row
    // arithmetic and noise counters as the full path, so the result is identical).
    const bool compact = cfg->prior == DD_PRIOR_MASK && gemm_gather_supported(cfg->dtype, cfg->d_model);
    int32_t* rows = (int32_t*)(wsc + w.rows);
    int32_t* count = (int32_t*)(wsc + w.count);
    int32_t* seq = (int32_t*)(wsc + w.seq);
    float* row_lse = (float*)(wsc + w.row_lse);
    // bf16 path: the vocabulary projection also emits each row's per-group log-sum-exps, so the
    // draw reads one group of logits per row instead of the whole row.  DD_LOOP_POSTERIOR_PASS keeps
    // the posterior's own pass over the rows instead.
    const bool fused = gemm_lse_supported(cfg->dtype, cfg->d_model) && !(flags & DD_LOOP_POSTERIOR_PASS);
    float* glse = fused ? (float*)(wsc + w.glse) : nullptr;
    // store-free: the logits region holds the group candidates [rows][glse_ld] int32 instead
    int32_t* cand = store_free ? (int32_t*)logits : nullptr;
    if (!compact) {   // the layout query reports count = -1 for a loop that does not compact
        launch_k(fill_i32_kernel, dim3(1), dim3(64), 0, s, count, -1, (int64_t)1);
        DD_TRY(launch_status("loop count"));
    }
    DD_TRY(trace_copy(0));
    for (int k = T; k >= 1; --k) {
        const uint32_t* nw = noise_words ? noise_words + (int64_t)(k - 1) * M * nu : nullptr;
        PostArgs a = make_post(cfg->prior, logits, ld, (int32_t)M, cfg->vocab, z, alphas[k],
                               alphas[k - 1], kappas ? kappas[k] : 1.0, nw, noise_seed, (uint32_t)k,
                               0u, z, row_lse, nullptr, (int32_t*)(wsc + w.err));
        // the list holds the masked rows that stage 0 of the draw unmasks: the others stay masked
        // whatever their logits
        if (compact) DD_TRY(launch_compact(z, M, cfg->mask_id, rows, count, s, L, seq, &a));
        DD_TRY(run_forward(cfg, params, z, B, L, alphas[k], logits, ld, wsc, s,
                           compact ? rows : nullptr, compact ? count : nullptr, nullptr, nullptr,
                           glse, w.glse_ld, cand, noise_seed, (uint32_t)k, compact ? seq : nullptr));
        if (compact) {
            // kappa < 1: the rows unmasked before this step keep or remask first (they read no
            // logits and are not in the compacted list, which was taken before the step)
            if (a.remask) DD_TRY(launch_remask(a, s));
            a.rows_idx = rows;
            a.count = count;
        }
        a.glse = glse;
        a.glse_ld = w.glse_ld;
        a.cand = cand;
        a.cand_ld = w.glse_ld;
        DD_TRY(launch_posterior(a, cfg->dtype, s));
        DD_TRY(trace_copy(T - k + 1));
    }
    return DD_OK;
}

dd_status dd_sample_loop(const dd_config* cfg, const void* params, int32_t B, int32_t L,
                         int32_t T, const double* alphas, int32_t* z, const uint32_t* noise_words,
                         uint64_t noise_seed, int32_t* z_trace, void* ws, size_t ws_bytes,
                         void* stream) {
    return dd_psi_sample_loop(cfg, params, B, L, T, alphas, nullptr, 0u, z, noise_words, noise_seed,
                              z_trace, ws, ws_bytes, stream);
}

size_t dd_spec_verify_workspace_bytes(int32_t S, int32_t B) {
    if (S <= 0 || B <= 0) return 0;
    return ((size_t)S * (2 * (size_t)B - 1) * sizeof(float) + 255) & ~(size_t)255;
}

int32_t dd_spec_verify_noise_width(int32_t B, int32_t V) {
    return (B - 1) + ntop_of(DD_PRIOR_UNIFORM, V) + V;
}

// Validation shared by dd_spec_verify and dd_spec_verify_noalloc (everything but the workspace).
static dd_status verify_check(const void* p_logits, const void* q_logits, int32_t logits_dtype, int64_t ld,
                              int32_t S, int32_t B, int32_t V, const int32_t* draft, int32_t* n_out,
                              int32_t* z_out) {
    DD_CHECK(logits_dtype == DD_BF16 || logits_dtype == DD_FP32, DD_E_DTYPE, "unknown logits dtype");
    DD_CHECK(S >= 0 && B >= 1 && V > 0, DD_E_ARG, "need S >= 0, B >= 1 and V > 0");
    DD_CHECK(V <= (1 << 24), DD_E_UNSUPPORTED, "V > 2^24 unsupported");
    DD_CHECK((int64_t)S * (2 * (int64_t)B - 1) <= INT32_MAX, DD_E_UNSUPPORTED, "too many rows");
    DD_CHECK(ld >= V && ld % 8 == 0, DD_E_SHAPE, "ld must be >= V and a multiple of 8");
    if (S == 0) return DD_OK;
    DD_CHECK(p_logits && n_out && z_out, DD_E_ARG, "NULL pointer argument");
    DD_CHECK(B == 1 || (q_logits && draft), DD_E_ARG, "B > 1 needs draft logits and tokens");
    return DD_OK;
}

static VerifyArgs make_verify(const void* p_logits, const void* q_logits, int64_t ld, int32_t S, int32_t B,
                              int32_t V, const int32_t* draft, const uint32_t* noise_words, uint64_t seed,
                              uint32_t step, uint32_t row0, int32_t* n_out, int32_t* z_out, int32_t* dev_err) {
    VerifyArgs a;
    memset(&a, 0, sizeof(a));
    a.p = p_logits; a.q = q_logits; a.ld = ld;
    a.S = S; a.B = B; a.V = V;
    a.draft = draft;
    a.noise = noise_words;
    a.nu = dd_spec_verify_noise_width(B, V);
    a.seed = seed; a.step = step; a.row0 = row0;
    a.n_out = n_out; a.z_out = z_out; a.err = dev_err;
    return a;
}

dd_status dd_spec_verify(const void* p_logits, const void* q_logits, int32_t logits_dtype, int64_t ld,
                         int32_t S, int32_t B, int32_t V, const int32_t* draft,
                         const uint32_t* noise_words, uint64_t seed, uint32_t step, uint32_t row0,
                         int32_t* n_out, int32_t* z_out, void* ws, size_t ws_bytes, int32_t* dev_err,
                         void* stream) {
    DD_TRY(verify_check(p_logits, q_logits, logits_dtype, ld, S, B, V, draft, n_out, z_out));
    if (S == 0) return DD_OK;
    DD_CHECK(ws, DD_E_ARG, "NULL pointer argument");
    const size_t need = dd_spec_verify_workspace_bytes(S, B);
    DD_CHECK(ws_bytes >= need, DD_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
    const VerifyArgs a = make_verify(p_logits, q_logits, ld, S, B, V, draft, noise_words, seed, step, row0,
                                     n_out, z_out, dev_err);
    return launch_verify(a, logits_dtype, (float*)ws, (hipStream_t)stream);
}

dd_status dd_spec_verify_noalloc(const void* p_logits, const void* q_logits, int32_t logits_dtype,
                                 int64_t ld, int32_t S, int32_t B, int32_t V, const int32_t* draft,
                                 const uint32_t* noise_words, uint64_t seed, uint32_t step,
                                 uint32_t row0, int32_t* n_out, int32_t* z_out, int32_t* dev_err,
                                 void* stream) {
    DD_TRY(verify_check(p_logits, q_logits, logits_dtype, ld, S, B, V, draft, n_out, z_out));
    if (S == 0) return DD_OK;
    const int64_t rows = (int64_t)S * (2 * (int64_t)B - 1);
    DD_CHECK(rows <= DD_SPEC_VERIFY_NOALLOC_ROWS, DD_E_WORKSPACE,
             "S (2B - 1) = %lld logit rows exceed the %d row log-sum-exps the library holds per device",
             (long long)rows, DD_SPEC_VERIFY_NOALLOC_ROWS);
    float* lse = nullptr;
    DD_TRY(verify_noalloc_scratch(&lse));
    const VerifyArgs a = make_verify(p_logits, q_logits, ld, S, B, V, draft, noise_words, seed, step, row0,
                                     n_out, z_out, dev_err);
    return launch_verify(a, logits_dtype, lse, (hipStream_t)stream);
}

dd_status dd_gaussian_latent_argmax(const int32_t* x, int32_t rows, int32_t V, double alpha_tilde,
                                    double sigma, uint64_t seed, uint32_t step, uint32_t row0,
                                    int32_t* z_out, int32_t* dev_err, void* stream) {
    DD_CHECK(rows >= 0 && V > 0, DD_E_ARG, "rows must be >= 0 and V > 0");
    DD_CHECK(alpha_tilde >= 0.0 && sigma > 0.0 && isfinite(alpha_tilde) && isfinite(sigma), DD_E_ARG,
             "need alpha_tilde >= 0 and sigma > 0");
    if (rows == 0) return DD_OK;
    DD_CHECK(x && z_out, DD_E_ARG, "NULL pointer argument");
    return launch_latent(x, rows, V, alpha_tilde, sigma, seed, step, row0, z_out, dev_err,
                         (hipStream_t)stream);
}

dd_status dd_profile_begin(int32_t max_launches, uint32_t class_mask) {
    DD_CHECK(max_launches > 0, DD_E_ARG, "max_launches must be positive");
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if ((int)g_prof.ev.size() < 2 * max_launches) {
        for (auto e : g_prof.ev) (void)hipEventDestroy(e);
        g_prof.ev.assign(2 * max_launches, nullptr);
        for (auto& e : g_prof.ev) {
            const hipError_t r = hipEventCreate(&e);
            DD_CHECK(r == hipSuccess, DD_E_HIP, "hipEventCreate: %s", hipGetErrorString(r));
        }
    }
    g_prof.cap = max_launches;
    g_prof.mask = class_mask ? class_mask : 0xFFFFFFFFu;
    g_prof.cls.clear();
    g_prof.dropped = 0;
    g_prof.open = -1;
    g_prof.on = true;
    return DD_OK;
}

dd_status dd_profile_end(void) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof.on = false;
    return DD_OK;
}

int32_t dd_profile_num_classes(void) { return KC_COUNT; }

dd_status dd_profile_read(int32_t cls, const char** name, int64_t* launches, double* total_ms) {
    DD_CHECK(cls >= 0 && cls < KC_COUNT, DD_E_ARG, "class %d out of range", cls);
    DD_CHECK(name && launches && total_ms, DD_E_ARG, "NULL pointer argument");
    std::lock_guard<std::mutex> lk(g_prof_mu);
    *name = kClassNames[cls];
    int64_t n = 0;
    double tot = 0.0;
    for (size_t i = 0; i < g_prof.cls.size(); ++i) {
        if (g_prof.cls[i] != cls) continue;
        hipError_t e = hipEventSynchronize(g_prof.ev[2 * i + 1]);
        float ms = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, g_prof.ev[2 * i], g_prof.ev[2 * i + 1]);
        DD_CHECK(e == hipSuccess, DD_E_HIP, "event timing: %s", hipGetErrorString(e));
        tot += ms;
        ++n;
    }
    *launches = n;
    *total_ms = tot;
    return DD_OK;
}

}  // extern "C"
