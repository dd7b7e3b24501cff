// C ABI of the MOD-DiT hot path: argument validation, the predictor state
// machine (Algorithm 1), the host-side factorisation of the structured
// normal equations (Appendix B.4), and the kernel launches.
#include "../../include/moddit.h"
#include "moddit_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <thread>
#include <vector>

namespace {

thread_local std::string g_last_error;

mod_status fail(mod_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

mod_status hip_fail(hipError_t e, const char* what) {
    return fail(MOD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Shape checks shared by every entry point.  `need_frames`: the predictor
// needs L to be a whole number (>= 2) of frames.
mod_status check_shape(const mod_shape* s, bool need_frames) {
    if (!s) return fail(MOD_ERR_INVALID_ARG, "shape is NULL");
    if (s->B <= 0 || s->H <= 0 || s->L <= 0 || s->d <= 0 || s->block <= 0)
        return fail(MOD_ERR_INVALID_ARG, "shape sizes must be positive (B=%d H=%d L=%d d=%d block=%d)",
                    s->B, s->H, s->L, s->d, s->block);
    if (s->d != 64 && s->d != 128) return fail(MOD_ERR_UNSUPPORTED, "d=%d (supported: 64, 128)", s->d);
    if (s->block != 64 && s->block != 128)
        return fail(MOD_ERR_UNSUPPORTED, "block=%d (supported: 64, 128)", s->block);
    const long n = (s->L + (long)s->block - 1) / s->block;
    if (n > moddit::kMaxBlocks)
        return fail(MOD_ERR_UNSUPPORTED, "n=%ld blocks exceeds %d", n, moddit::kMaxBlocks);
    if ((long)s->B * s->H * n > (1L << 30))
        return fail(MOD_ERR_UNSUPPORTED, "B*H*n too large");
    if (need_frames) {
        if (s->frame_tokens <= 0) return fail(MOD_ERR_INVALID_ARG, "frame_tokens must be positive");
        if (s->text_tokens < 0 || s->text_tokens >= s->L)
            return fail(MOD_ERR_INVALID_ARG, "text_tokens=%d must be in [0, L)", s->text_tokens);
        const int Lv = s->L - s->text_tokens;
        if (Lv % s->frame_tokens != 0)
            return fail(MOD_ERR_UNSUPPORTED, "%d video tokens are not a whole number of frames of %d tokens",
                        Lv, s->frame_tokens);
        if (Lv / s->frame_tokens < 2)
            return fail(MOD_ERR_UNSUPPORTED, "need at least 2 frames (F=%d)", Lv / s->frame_tokens);
    }
    return MOD_OK;
}

// ---------------------------------------------------------------------------
// Host factorisation.  With the last vertical coefficient fixed to zero the
// normal matrix of Eq. 4 is SPD and its C^T C block is diagonal, so the
// system reduces to the Schur complement on u = [d_0..d_{n-2}, e_0..e_{F-1}]:
//   S = Y - W^T Dc^{-1} W      (q x q, q = n - 1 + F)
// with Dc = diag(n - |delta|) (C^T C), W = [C^T D (0/1), C^T E] and
// Y = [[n I, D^T E], [E^T D, E^T E]]; C^T E[delta, f] = max(0, |R_f| - |delta|),
// D^T E[j, f] = |R_f| [j in R_f], E^T E[f, g] = |R_f cap R_g|^2.
// S is formed in O(q^2 + n F |R|), factored (Cholesky) and inverted once.
// ---------------------------------------------------------------------------
template <class F>
void parallel_rows(int rows, F&& body) {
    unsigned nt = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
    if (rows < 256) nt = 1;
    if (nt == 1) {
        for (int r = 0; r < rows; ++r) body(r);
        return;
    }
    std::vector<std::thread> th;
    for (unsigned t = 0; t < nt; ++t)
        th.emplace_back([&, t] {
            for (int r = (int)t; r < rows; r += (int)nt) body(r);
        });
    for (auto& x : th) x.join();
}

bool build_schur_inverse(int n, const std::vector<int>& lo, const std::vector<int>& hi,
                         std::vector<double>& Sinv, std::string& why) {
    const int F = (int)lo.size();
    const int q = n - 1 + F;
    std::vector<double> S((size_t)q * q, 0.0);
    auto Dc = [n](int a) { return (double)(n - std::abs(a - (n - 1))); };
    std::vector<double> pref(2 * n, 0.0);
    for (int a = 0; a < 2 * n - 1; ++a) pref[a + 1] = pref[a] + 1.0 / Dc(a);
    // vertical x vertical
    for (int j = 0; j < n - 1; ++j)
        for (int jp = 0; jp < n - 1; ++jp) {
            const int mn = std::min(j, jp), mx = std::max(j, jp);
            double v = pref[mn + n] - pref[mx];
            S[(size_t)j * q + jp] = (j == jp ? (double)n : 0.0) - v;
        }
    // vertical x frame
    for (int f = 0; f < F; ++f) {
        const int sz = hi[f] - lo[f] + 1;
        for (int j = 0; j < n - 1; ++j) {
            const int a0 = std::max(j, n - sz), a1 = std::min(j + n - 1, n - 2 + sz);
            double v = 0.0;
            for (int a = a0; a <= a1; ++a) v += (double)(sz - std::abs(a - (n - 1))) / Dc(a);
            const double y = (j >= lo[f] && j <= hi[f]) ? (double)sz : 0.0;
            S[(size_t)j * q + (n - 1 + f)] = S[(size_t)(n - 1 + f) * q + j] = y - v;
        }
    }
    // frame x frame
    for (int f = 0; f < F; ++f)
        for (int g = 0; g < F; ++g) {
            const int sf = hi[f] - lo[f] + 1, sg = hi[g] - lo[g] + 1;
            const int ov = std::max(0, std::min(hi[f], hi[g]) - std::max(lo[f], lo[g]) + 1);
            double v = 0.0;
            for (int dl = -(std::min(sf, sg) - 1); dl <= std::min(sf, sg) - 1; ++dl)
                v += (double)(sf - std::abs(dl)) * (double)(sg - std::abs(dl)) /
                     (double)(n - std::abs(dl));
            S[(size_t)(n - 1 + f) * q + (n - 1 + g)] = (double)ov * ov - v;
        }
    // Cholesky S = L L^T (lower, row-major, in a separate array)
    std::vector<double> Lm((size_t)q * q, 0.0);
    for (int j = 0; j < q; ++j) {
        const double* Lj = &Lm[(size_t)j * q];
        double s = S[(size_t)j * q + j];
        for (int k = 0; k < j; ++k) s -= Lj[k] * Lj[k];
        if (!(s > 1e-12 * std::fabs(S[(size_t)j * q + j]))) {
            char b[160];
            std::snprintf(b, sizeof(b), "normal matrix not positive definite at pivot %d (%g)", j, s);
            why = b;
            return false;
        }
        const double djj = std::sqrt(s);
        Lm[(size_t)j * q + j] = djj;
        parallel_rows(q - j - 1, [&](int r) {
            const int i = j + 1 + r;
            double* Li = &Lm[(size_t)i * q];
            double t = S[(size_t)i * q + j];
            for (int k = 0; k < j; ++k) t -= Li[k] * Lj[k];
            Li[j] = t / djj;
        });
    }
    // XT = (L^{-1})^T row by row: XT[c][i] = (L^{-1})[i][c]
    std::vector<double> XT((size_t)q * q, 0.0);
    parallel_rows(q, [&](int c) {
        double* x = &XT[(size_t)c * q];
        x[c] = 1.0 / Lm[(size_t)c * q + c];
        for (int i = c + 1; i < q; ++i) {
            const double* Li = &Lm[(size_t)i * q];
            double t = 0.0;
            for (int k = c; k < i; ++k) t += Li[k] * x[k];
            x[i] = -t / Li[i];
        }
    });
    // S^{-1} = L^{-T} L^{-1}: S^{-1}[a][b] = sum_{k >= max(a,b)} XT[a][k] XT[b][k]
    Sinv.assign((size_t)q * q, 0.0);
    parallel_rows(q, [&](int a) {
        const double* xa = &XT[(size_t)a * q];
        for (int b = a; b < q; ++b) {
            const double* xb = &XT[(size_t)b * q];
            double t = 0.0;
            for (int k = b; k < q; ++k) t += xa[k] * xb[k];
            Sinv[(size_t)a * q + b] = t;
        }
    });
    for (int a = 0; a < q; ++a)
        for (int b = 0; b < a; ++b) Sinv[(size_t)a * q + b] = Sinv[(size_t)b * q + a];
    return true;
}

}  // namespace

struct mod_stats {
    mod_shape shape{};
    mod_params params{};
    int n = 0, F = 0, p = 0, q = 0, BH = 0;   // n: video blocks (the MOD model's)
    int Lv = 0;                // video tokens
    int nt = 0;                // blocks of the whole sequence (the masks')
    int tb0 = 0;               // first text block (nt without text)
    double scale = 0.0;
    int device = 0;
    // device buffers
    double* qbar = nullptr;
    double* kbar = nullptr;
    double* G = nullptr;
    double* r = nullptr;
    double* bU = nullptr;
    double* u = nullptr;
    double* X[2] = {nullptr, nullptr};
    double* pred = nullptr;
    double* Sinv = nullptr;
    int* reg = nullptr;
    int* row_lo = nullptr;
    int* row_hi = nullptr;
    int32_t* gate = nullptr;
    uint8_t* chosen = nullptr;   // pattern mode: chosen patterns [BH, 3n-1]
    // host state
    int n_anchors = 0;
    int newest = 1;            // slot of the newest anchor
    int anchor_step[2] = {0, 0};
    bool has_step = false;
    int last_step = 0;
    bool last_predicted = false;   // the last call was the predict of last_step
    bool gate_frozen = false;
    bool fitted = false;
    bool predicted = false;
};

namespace {

void free_stats(mod_stats* s) {
    if (!s) return;
    void* ptrs[] = {s->qbar, s->kbar, s->G,   s->r,      s->bU,     s->u,   s->X[0], s->X[1],
                    s->pred, s->Sinv, s->reg, s->row_lo, s->row_hi, s->gate, s->chosen};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
    delete s;
}

bool is_anchor_step(const mod_stats* s, int t) {
    const int dt = s->params.delta_t, m = s->params.warmup_m;
    if (dt <= 0) return false;
    if (s->params.anchor_rule == 0) return t > m && (t - m) % dt == 0;
    return t % dt == 0;
}

// rhs -> solve of the statistic in G into the next anchor slot
mod_status fit_stat_into_next_slot(mod_stats* s, int step, hipStream_t st) {
    const int slot = 1 - s->newest;
    // the solve's partial-product array u ([kSolveSplit, BH, q], q = n - 1 + F)
    // is free until the solve and holds the rhs row ranges' sums
    static_assert(moddit::kRhsChunks * 3 <= moddit::kSolveSplit, "rhs ranges must fit the solve's scratch");
    hipError_t e = moddit::launch_rhs(s->G, s->reg, s->r, s->u, s->BH, s->n, s->F, st);
    if (e != hipSuccess) return hip_fail(e, "rhs launch");
    e = moddit::launch_solve(s->r, s->reg, s->Sinv, s->bU, s->u, s->X[slot], s->BH, s->n, s->F, st);
    if (e != hipSuccess) return hip_fail(e, "solve launch");
    s->newest = slot;
    s->anchor_step[slot] = step;
    s->n_anchors = std::min(2, s->n_anchors + 1);
    s->fitted = true;
    return MOD_OK;
}

// pool -> block mass -> rhs -> solve into the next anchor slot (statistic 0)
mod_status fit_into_next_slot(mod_stats* s, const void* q, const void* k, int step,
                              hipStream_t st) {
    const mod_shape& sh = s->shape;
    hipError_t e = moddit::launch_pool(static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                                       s->qbar, s->kbar, s->BH, s->Lv, sh.L, sh.d, sh.block, s->n, st);
    if (e != hipSuccess) return hip_fail(e, "pool launch");
    e = moddit::launch_block_mass(s->qbar, s->kbar, s->G, s->BH, s->Lv, sh.d, sh.block, s->n, s->scale, st);
    if (e != hipSuccess) return hip_fail(e, "block-mass launch");
    return fit_stat_into_next_slot(s, step, st);
}

mod_status check_step(const mod_stats* s, int step) {
    if (s->has_step && step <= s->last_step)
        return fail(MOD_ERR_BAD_STATE, "step %d does not follow step %d", step, s->last_step);
    return MOD_OK;
}

// an update may also follow the predict of the same step (its attention)
mod_status check_update_step(const mod_stats* s, int step) {
    if (s->has_step && (step < s->last_step || (step == s->last_step && !s->last_predicted)))
        return fail(MOD_ERR_BAD_STATE, "step %d does not follow step %d", step, s->last_step);
    return MOD_OK;
}

}  // namespace

extern "C" {

int mod_num_blocks(const mod_shape* shape) {
    if (!shape || shape->L <= 0 || shape->block <= 0) return 0;
    return ceil_div(shape->L, shape->block);
}

int mod_num_coeffs(const mod_shape* shape) {
    if (mod_num_blocks(shape) == 0 || shape->frame_tokens <= 0 || shape->text_tokens < 0 ||
        shape->text_tokens >= shape->L)
        return 0;
    const int Lv = shape->L - shape->text_tokens;
    if (Lv % shape->frame_tokens) return 0;
    return 3 * ceil_div(Lv, shape->block) - 1 + Lv / shape->frame_tokens;
}

mod_status mod_stats_create(const mod_shape* shape, const mod_params* params, mod_stats** out) {
    if (!out) return fail(MOD_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (!params) return fail(MOD_ERR_INVALID_ARG, "params is NULL");
    mod_status st = check_shape(shape, true);
    if (st != MOD_OK) return st;
    if (params->warmup_m < 0) return fail(MOD_ERR_INVALID_ARG, "warmup_m must be >= 0");
    if (params->anchor_rule != 0 && params->anchor_rule != 1)
        return fail(MOD_ERR_INVALID_ARG, "anchor_rule must be 0 or 1");
    if (!std::isfinite(params->tau_e)) return fail(MOD_ERR_INVALID_ARG, "tau_e must be finite");
    if (params->statistic != 0 && params->statistic != 1)
        return fail(MOD_ERR_INVALID_ARG, "statistic must be 0 or 1");
    if (params->statistic == 1 && !(params->eta > 0.0f && std::isfinite(params->eta)))
        return fail(MOD_ERR_INVALID_ARG, "eta must be positive and finite");

    mod_stats* s = new (std::nothrow) mod_stats();
    if (!s) return fail(MOD_ERR_NOMEM, "host allocation failed");
    s->shape = *shape;
    s->params = *params;
    s->Lv = shape->L - shape->text_tokens;
    s->n = ceil_div(s->Lv, shape->block);
    s->nt = ceil_div(shape->L, shape->block);
    s->tb0 = shape->text_tokens > 0 ? s->Lv / shape->block : s->nt;
    s->F = s->Lv / shape->frame_tokens;
    s->p = 3 * s->n - 1 + s->F;
    s->q = s->n - 1 + s->F;
    s->BH = shape->B * shape->H;
    s->scale = 1.0 / std::sqrt((double)shape->d);
    (void)hipGetDevice(&s->device);

    const int n = s->n, F = s->F;
    std::vector<int> lo(F), hi(F), reg(2 * F), row_lo(n, n), row_hi(n, -1);
    for (int f = 0; f < F; ++f) {
        lo[f] = (int)(((long)f * shape->frame_tokens) / shape->block);
        hi[f] = (int)((((long)f + 1) * shape->frame_tokens - 1) / shape->block);
        reg[2 * f] = lo[f];
        reg[2 * f + 1] = hi[f];
        for (int i = lo[f]; i <= hi[f]; ++i) {
            row_lo[i] = std::min(row_lo[i], lo[f]);
            row_hi[i] = std::max(row_hi[i], hi[f]);
        }
    }
    std::vector<double> Sinv;
    std::string why;
    if (!build_schur_inverse(n, lo, hi, Sinv, why)) {
        free_stats(s);
        return fail(MOD_ERR_UNSUPPORTED, "%s", why.c_str());
    }

    const size_t BH = (size_t)s->BH;
    struct Alloc { void** p; size_t bytes; } allocs[] = {
        {(void**)&s->qbar, BH * n * shape->d * sizeof(double)},
        {(void**)&s->kbar, BH * n * shape->d * sizeof(double)},
        {(void**)&s->G, BH * n * n * sizeof(double)},
        {(void**)&s->r, BH * s->p * sizeof(double)},
        {(void**)&s->bU, BH * s->q * sizeof(double)},
        {(void**)&s->u, (size_t)moddit::kSolveSplit * BH * s->q * sizeof(double)},   // per-chunk partial products
        {(void**)&s->X[0], BH * s->p * sizeof(double)},
        {(void**)&s->X[1], BH * s->p * sizeof(double)},
        {(void**)&s->pred, BH * (3 * n - 1) * sizeof(double)},
        {(void**)&s->Sinv, (size_t)s->q * s->q * sizeof(double)},
        {(void**)&s->reg, 2 * (size_t)F * sizeof(int)},
        {(void**)&s->row_lo, (size_t)n * sizeof(int)},
        {(void**)&s->row_hi, (size_t)n * sizeof(int)},
        {(void**)&s->gate, BH * sizeof(int32_t)},
        {(void**)&s->chosen, BH * (3 * n - 1) * sizeof(uint8_t)},
    };
    for (auto& a : allocs) {
        hipError_t e = hipMalloc(a.p, a.bytes);
        if (e != hipSuccess) {
            free_stats(s);
            return fail(MOD_ERR_NOMEM, "hipMalloc(%zu): %s", a.bytes, hipGetErrorString(e));
        }
    }
    hipError_t e = hipMemcpy(s->Sinv, Sinv.data(), Sinv.size() * sizeof(double), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(s->reg, reg.data(), reg.size() * sizeof(int), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(s->row_lo, row_lo.data(), n * sizeof(int), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(s->row_hi, row_hi.data(), n * sizeof(int), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(s->gate, 0, BH * sizeof(int32_t));
    if (e == hipSuccess) e = hipMemset(s->G, 0, BH * n * n * sizeof(double));
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        free_stats(s);
        return hip_fail(e, "upload of the predictor tables");
    }
    *out = s;
    return MOD_OK;
}

mod_status mod_stats_destroy(mod_stats* stats) {
    if (!stats) return MOD_OK;
    hipError_t e = hipDeviceSynchronize();
    free_stats(stats);
    if (e != hipSuccess) return hip_fail(e, "synchronise before destroy");
    return MOD_OK;
}

mod_status mod_collect_stats(mod_stats* s, const void* q, const void* k, int step, void* stream) {
    if (!s) return fail(MOD_ERR_INVALID_ARG, "stats is NULL");
    if (!q || !k) return fail(MOD_ERR_INVALID_ARG, "q and k must not be NULL");
    if (s->params.statistic != 0)
        return fail(MOD_ERR_BAD_STATE, "statistic 1 records anchors with mod_update_stats");
    mod_status st = check_step(s, step);
    if (st != MOD_OK) return st;
    st = fit_into_next_slot(s, q, k, step, static_cast<hipStream_t>(stream));
    if (st != MOD_OK) return st;
    s->has_step = true;
    s->last_step = step;
    s->last_predicted = false;
    return MOD_OK;
}

mod_status mod_update_stats(mod_stats* s, const void* q, const void* k, const float* lse,
                            const int32_t* kv_idx, const int32_t* kv_cnt, int step, void* stream) {
    if (!s) return fail(MOD_ERR_INVALID_ARG, "stats is NULL");
    if (!q || !k || !lse || !kv_idx || !kv_cnt)
        return fail(MOD_ERR_INVALID_ARG, "q, k, lse, kv_idx and kv_cnt must not be NULL");
    if (s->params.statistic != 1)
        return fail(MOD_ERR_BAD_STATE, "mod_update_stats needs statistic 1");
    mod_status st = check_update_step(s, step);
    if (st != MOD_OK) return st;
    const mod_shape& sh = s->shape;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    hipError_t e = moddit::launch_stat_count(static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                                             kv_idx, kv_cnt, lse, (float)s->scale,
                                             (float)std::log((double)s->params.eta), s->G, s->BH, sh.L, sh.d,
                                             sh.block, s->nt, s->n, hs);
    if (e != hipSuccess) return hip_fail(e, "statistic launch");
    st = fit_stat_into_next_slot(s, step, hs);
    if (st != MOD_OK) return st;
    s->has_step = true;
    s->last_step = step;
    s->last_predicted = false;
    return MOD_OK;
}

mod_status mod_predict_block_mask(mod_stats* s, const void* q, const void* k, int step,
                                  const mod_budget* budget, int32_t* kv_idx, int32_t* kv_cnt,
                                  void* stream) {
    if (!s) return fail(MOD_ERR_INVALID_ARG, "stats is NULL");
    if (!budget) return fail(MOD_ERR_INVALID_ARG, "budget is NULL");
    if (!kv_idx || !kv_cnt) return fail(MOD_ERR_INVALID_ARG, "kv_idx and kv_cnt must not be NULL");
    const int n = s->n;
    int topk = 0;
    double tau = 0.0;
    if (budget->mode == MOD_BUDGET_TOPK) {
        if (!(budget->density > 0.0f && budget->density <= 1.0f))
            return fail(MOD_ERR_INVALID_ARG, "TOPK density must be in (0, 1]");
        const double kk = std::ceil((double)budget->density * n - 1e-6);
        topk = (int)std::min<double>(n, std::max<double>(1.0, kk));
    } else if (budget->mode == MOD_BUDGET_MASS) {
        if (!(budget->mass > 0.0f && budget->mass <= 1.0f))
            return fail(MOD_ERR_INVALID_ARG, "MASS mass must be in (0, 1]");
        tau = (double)budget->mass;
    } else if (budget->mode == MOD_BUDGET_PATTERN) {
        if (budget->patterns < 1 || budget->patterns > 3 * n - 1)
            return fail(MOD_ERR_INVALID_ARG, "PATTERN patterns must be in [1, 3n-1] = [1, %d]", 3 * n - 1);
    } else {
        return fail(MOD_ERR_INVALID_ARG, "unknown budget mode %d", budget->mode);
    }
    if (s->n_anchors == 0) return fail(MOD_ERR_BAD_STATE, "predict before any collected step");
    mod_status st = check_step(s, step);
    if (st != MOD_OK) return st;
    const bool anchor = s->params.statistic == 0 && is_anchor_step(s, step);
    if (anchor && (!q || !k))
        return fail(MOD_ERR_INVALID_ARG, "step %d re-anchors: q and k must not be NULL", step);
    hipStream_t hs = static_cast<hipStream_t>(stream);

    if (!s->gate_frozen) {
        const double* Xa = s->X[s->newest];
        const double* Xb = s->n_anchors > 1 ? s->X[1 - s->newest] : Xa;
        hipError_t e = moddit::launch_gate(Xa, Xb, s->gate, s->BH, n, s->F, (double)s->params.tau_e, hs);
        if (e != hipSuccess) return hip_fail(e, "gate launch");
        s->gate_frozen = true;
    }
    if (anchor) {
        st = fit_into_next_slot(s, q, k, step, hs);
        if (st != MOD_OK) return st;
    }
    const double* X2 = s->X[s->newest];
    const double* X1 = X2;
    double w = 0.0;
    if (s->n_anchors > 1) {
        X1 = s->X[1 - s->newest];
        const int t2 = s->anchor_step[s->newest], t1 = s->anchor_step[1 - s->newest];
        w = (double)(step - t2) / (double)(t2 - t1);
    }
    hipError_t e = moddit::launch_extrapolate(X1, X2, w, s->pred, s->BH, n, s->F, hs);
    if (e != hipSuccess) return hip_fail(e, "extrapolate launch");
    if (budget->mode == MOD_BUDGET_PATTERN)
        e = moddit::launch_select_patterns(s->pred, s->gate, s->row_lo, s->row_hi, budget->patterns,
                                           s->chosen, kv_idx, kv_cnt, s->BH, n, s->nt, s->tb0, hs);
    else
        e = moddit::launch_select(s->pred, s->gate, s->row_lo, s->row_hi, budget->mode, topk, tau,
                                  kv_idx, kv_cnt, s->BH, n, s->nt, s->tb0, hs);
    if (e != hipSuccess) return hip_fail(e, "select launch");
    s->has_step = true;
    s->last_step = step;
    s->last_predicted = true;
    s->predicted = true;
    return MOD_OK;
}

size_t mod_attn_workspace_bytes(const mod_shape* shape) {
    if (check_shape(shape, false) != MOD_OK) return 0;
    return moddit::attn_workspace_bytes(shape->B * shape->H, ceil_div(shape->L, shape->block), shape->d,
                                        shape->block);
}

size_t mod_attn_plan_bytes(const mod_shape* shape) {
    if (check_shape(shape, false) != MOD_OK) return 0;
    return moddit::attn_plan_bytes(shape->B * shape->H, ceil_div(shape->L, shape->block), 0);
}

mod_status mod_block_sparse_attn_fwd(const mod_shape* shape, const void* q, const void* k,
                                     const void* v, const int32_t* kv_idx, const int32_t* kv_cnt,
                                     float scale, void* o, float* lse, void* workspace,
                                     size_t ws_bytes, void* stream) {
    mod_status st = check_shape(shape, false);
    if (st != MOD_OK) return st;
    if (!q || !k || !v || !o || !kv_idx || !kv_cnt)
        return fail(MOD_ERR_INVALID_ARG, "q, k, v, o, kv_idx and kv_cnt must not be NULL");
    const size_t need = moddit::attn_plan_bytes(shape->B * shape->H, ceil_div(shape->L, shape->block), 0);
    if (!workspace || ws_bytes < need)
        return fail(MOD_ERR_INVALID_ARG, "workspace of at least %zu bytes needed (got %zu%s)", need, ws_bytes,
                    workspace ? "" : ", NULL");
    if (reinterpret_cast<uintptr_t>(workspace) % 16 != 0)
        return fail(MOD_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    if (!(scale >= 0.0f) || !std::isfinite(scale))
        return fail(MOD_ERR_INVALID_ARG, "scale must be finite and >= 0");
    const float sc = scale == 0.0f ? (float)(1.0 / std::sqrt((double)shape->d)) : scale;
    const int n = ceil_div(shape->L, shape->block);
    hipError_t e = moddit::launch_attn_fwd(
        static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v),
        kv_idx, kv_cnt, sc, static_cast<uint16_t*>(o), lse, shape->B * shape->H, shape->L, shape->d,
        shape->block, n, workspace, ws_bytes, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "attention launch");
    return MOD_OK;
}

mod_status mod_block_sparse_attn_fwd_noalloc(const mod_shape* shape, const void* q, const void* k,
                                             const void* v, const int32_t* kv_idx,
                                             const int32_t* kv_cnt, float scale, void* o, float* lse,
                                             void* stream) {
    mod_status st = check_shape(shape, false);
    if (st != MOD_OK) return st;
    // the work plan only: the no-allocation path does not split walks
    const size_t need = moddit::attn_plan_bytes(shape->B * shape->H, ceil_div(shape->L, shape->block), 0);
    if (need > (size_t)MOD_ATTN_NOALLOC_MAX_BYTES)
        return fail(MOD_ERR_UNSUPPORTED,
                    "work plan of %zu bytes exceeds the %zu-byte library array of the no-allocation "
                    "entry point (B*H*(ceil(n/2) + 16) too large); use mod_block_sparse_attn_fwd",
                    need, (size_t)MOD_ATTN_NOALLOC_MAX_BYTES);
    static_assert(moddit::kNoAllocScratchBytes == (size_t)MOD_ATTN_NOALLOC_MAX_BYTES,
                  "header and library disagree on the scratch size");
    void* ws = nullptr;
    const hipError_t e = moddit::noalloc_scratch(&ws);
    if (e != hipSuccess) return hip_fail(e, "device address of the library work-plan array");
    return mod_block_sparse_attn_fwd(shape, q, k, v, kv_idx, kv_cnt, scale, o, lse, ws, need, stream);
}

mod_status mod_stats_get_anchor(const mod_stats* s, int slot, double* host_coeffs, int* step) {
    if (!s || !host_coeffs) return fail(MOD_ERR_INVALID_ARG, "NULL argument");
    if (slot < 0 || slot > 1) return fail(MOD_ERR_INVALID_ARG, "slot must be 0 or 1");
    if (slot >= s->n_anchors) return fail(MOD_ERR_BAD_STATE, "anchor %d not recorded", slot);
    const int idx = slot == 0 ? s->newest : 1 - s->newest;
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess)
        e = hipMemcpy(host_coeffs, s->X[idx], (size_t)s->BH * s->p * sizeof(double), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "anchor copy");
    if (step) *step = s->anchor_step[idx];
    return MOD_OK;
}

mod_status mod_stats_get_pooled(const mod_stats* s, double* host_qbar, double* host_kbar) {
    if (!s || !host_qbar || !host_kbar) return fail(MOD_ERR_INVALID_ARG, "NULL argument");
    if (!s->fitted) return fail(MOD_ERR_BAD_STATE, "no fit yet");
    const size_t bytes = (size_t)s->BH * s->n * s->shape.d * sizeof(double);
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpy(host_qbar, s->qbar, bytes, hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = hipMemcpy(host_kbar, s->kbar, bytes, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "pooled copy");
    return MOD_OK;
}

mod_status mod_stats_get_block_mass(const mod_stats* s, double* host_G) {
    if (!s || !host_G) return fail(MOD_ERR_INVALID_ARG, "NULL argument");
    if (!s->fitted) return fail(MOD_ERR_BAD_STATE, "no fit yet");
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess)
        e = hipMemcpy(host_G, s->G, (size_t)s->BH * s->n * s->n * sizeof(double), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "block-mass copy");
    return MOD_OK;
}

mod_status mod_stats_get_prediction(const mod_stats* s, double* host_pred) {
    if (!s || !host_pred) return fail(MOD_ERR_INVALID_ARG, "NULL argument");
    if (!s->predicted) return fail(MOD_ERR_BAD_STATE, "no prediction yet");
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess)
        e = hipMemcpy(host_pred, s->pred, (size_t)s->BH * (3 * s->n - 1) * sizeof(double),
                      hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "prediction copy");
    return MOD_OK;
}

mod_status mod_stats_get_gate(const mod_stats* s, int32_t* host_gate) {
    if (!s || !host_gate) return fail(MOD_ERR_INVALID_ARG, "NULL argument");
    if (!s->gate_frozen) return fail(MOD_ERR_BAD_STATE, "gate not fixed before the first predict");
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess)
        e = hipMemcpy(host_gate, s->gate, (size_t)s->BH * sizeof(int32_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "gate copy");
    return MOD_OK;
}

const char* mod_status_string(mod_status status) {
    switch (status) {
        case MOD_OK: return "MOD_OK";
        case MOD_ERR_INVALID_ARG: return "MOD_ERR_INVALID_ARG";
        case MOD_ERR_UNSUPPORTED: return "MOD_ERR_UNSUPPORTED";
        case MOD_ERR_BAD_STATE: return "MOD_ERR_BAD_STATE";
        case MOD_ERR_HIP: return "MOD_ERR_HIP";
        case MOD_ERR_NOMEM: return "MOD_ERR_NOMEM";
    }
    return "MOD_ERR_UNKNOWN";
}

const char* mod_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
