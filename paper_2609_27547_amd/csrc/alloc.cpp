// Elastic resource allocation (Section 4.3.2): Algorithm 1 over the stage
// lookup tables, the objective of Eq. (2), the runtime trigger and table
// refinement.  Host-only C++; the readings of what the paper leaves open are
// listed in ebrl_alloc.h.
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <new>
#include <vector>

#include "ebrl.h"
#include "ebrl_alloc.h"

namespace {

bool ascending_quotas(const int32_t* g, int32_t n, int32_t lo) {
    if (!g || n < 1) return false;
    for (int32_t i = 0; i < n; ++i) {
        if (g[i] < lo || g[i] > 100) return false;
        if (i && g[i] <= g[i - 1]) return false;
    }
    return true;
}

bool rates_ok(const double* r, size_t n) {
    if (!r) return false;
    for (size_t i = 0; i < n; ++i)
        if (!(r[i] >= 0.0) || !std::isfinite(r[i])) return false;
    return true;
}

bool profiles_ok(const ebrl_alloc_profiles& p) {
    if (!p.cenv || p.n_cenv < 1 || !ascending_quotas(p.ssim, p.n_ssim, 0)) return false;
    for (int32_t c = 0; c < p.n_cenv; ++c)
        if (p.cenv[c] < 1) return false;
    if (!ascending_quotas(p.sgen, p.n_sgen, 1) || !ascending_quotas(p.strain, p.n_strain, 1)) return false;
    if (!p.bgen || p.n_bgen < 1 || !p.btrain || p.n_btrain < 1) return false;
    return rates_ok(p.sim_rate, (size_t)p.n_cenv * p.n_ssim) &&
           rates_ok(p.gen_rate, (size_t)p.n_sgen * p.n_bgen) && rates_ok(p.gen_mem, p.n_bgen) &&
           rates_ok(p.train_rate, (size_t)p.n_strain * p.n_btrain) && rates_ok(p.train_mem, p.n_btrain);
}

// Rate of batch column `col` at quota s (percent): piecewise linear over the
// profiled quotas, through (0, 0) below the first, flat past the last.
double quota_rate(const int32_t* grid, int32_t n, const double* table, int32_t ncol, int32_t col, int32_t s) {
    auto at = [&](int32_t i) { return table[(size_t)i * ncol + col]; };
    if (s <= 0) return 0.0;
    if (s >= grid[n - 1]) return at(n - 1);
    int32_t hi = 0;
    while (grid[hi] < s) ++hi;                  // first profiled quota >= s
    if (grid[hi] == s) return at(hi);
    const double s0 = hi ? grid[hi - 1] : 0.0, r0 = hi ? at(hi - 1) : 0.0;
    const double s1 = grid[hi], r1 = at(hi);
    return r0 + (r1 - r0) * ((double)s - s0) / (s1 - s0);
}

struct Choice {
    int32_t jg = -1, jt = -1;                   // batch indices
    double t_gen = 0, t_train = 0, t_roll = 0, theta = -1;
};

// The batch pair maximising Eq. (2) at quotas (sg, st) within the memory
// budget; the first pair in grid order wins ties.
Choice best_pair(const ebrl_alloc_profiles& p, double mem, double t_sim, int32_t sg, int32_t st) {
    Choice best;
    for (int32_t jg = 0; jg < p.n_bgen; ++jg) {
        const double tg = quota_rate(p.sgen, p.n_sgen, p.gen_rate, p.n_bgen, jg, sg);
        const double tr = std::min(t_sim, tg);
        for (int32_t jt = 0; jt < p.n_btrain; ++jt) {
            if (p.gen_mem[jg] + p.train_mem[jt] > mem) continue;
            const double tt = quota_rate(p.strain, p.n_strain, p.train_rate, p.n_btrain, jt, st);
            const double th = std::min(tr, tt);
            if (th > best.theta) {
                best.jg = jg; best.jt = jt;
                best.t_gen = tg; best.t_train = tt; best.t_roll = tr; best.theta = th;
            }
        }
    }
    return best;
}

int32_t index_of(const int32_t* g, int32_t n, int32_t v) {
    for (int32_t i = 0; i < n; ++i)
        if (g[i] == v) return i;
    return -1;
}

}  // namespace

struct ebrl_alloc_monitor {
    int32_t window, patience;
    double gap;
    std::vector<double> roll, train;            // ring buffers of the last `window` observations
    int32_t count = 0, head = 0, streak = 0;
};

extern "C" {

int ebrl_alloc_solve(const ebrl_alloc_profiles* prof, const ebrl_alloc_limits* lim, ebrl_alloc_result* out) {
    if (!prof || !lim || !out || !profiles_ok(*prof)) return EBRL_E_INVALID;
    const ebrl_alloc_profiles& p = *prof;
    if (lim->cores < 1 || !(lim->mem_bytes >= 0) || lim->sgen_min < 0 || lim->strain_min < 0 ||
        !(lim->knee_tol >= 0 && lim->knee_tol < 1))
        return EBRL_E_INVALID;

    // cores per environment and concurrency
    int32_t c_best = -1;
    for (int32_t c = 0; c < p.n_cenv; ++c) {
        if (lim->cores / p.cenv[c] < 1) continue;
        const double r = p.sim_rate[(size_t)c * p.n_ssim + p.n_ssim - 1];
        if (c_best < 0 || r > p.sim_rate[(size_t)c_best * p.n_ssim + p.n_ssim - 1]) c_best = c;
    }
    if (c_best < 0) return EBRL_E_INVALID;
    const double* row = p.sim_rate + (size_t)c_best * p.n_ssim;
    // simulator knee and capacity
    const double top = *std::max_element(row, row + p.n_ssim);
    int32_t knee = p.n_ssim - 1;
    for (int32_t j = 0; j < p.n_ssim; ++j)
        if (row[j] >= (1.0 - lim->knee_tol) * top) { knee = j; break; }
    const int32_t s_sim = p.ssim[knee];
    const double t_sim = row[knee];

    int32_t lo = lim->sgen_min, hi = 100 - s_sim - lim->strain_min;
    if (lo > hi) return EBRL_E_INVALID;
    bool any = false;
    for (int32_t jg = 0; jg < p.n_bgen && !any; ++jg)
        for (int32_t jt = 0; jt < p.n_btrain && !any; ++jt)
            any = p.gen_mem[jg] + p.train_mem[jt] <= lim->mem_bytes;
    if (!any) return EBRL_E_OOM;

    // bisection on the generation quota
    int32_t steps = 0;
    while (hi - lo > 1) {
        const int32_t sg = (lo + hi) / 2;
        const Choice ch = best_pair(p, lim->mem_bytes, t_sim, sg, 100 - s_sim - sg);
        if (ch.t_roll > ch.t_train) hi = sg;
        else lo = sg;
        ++steps;
    }
    const Choice a = best_pair(p, lim->mem_bytes, t_sim, lo, 100 - s_sim - lo);
    const Choice b = best_pair(p, lim->mem_bytes, t_sim, hi, 100 - s_sim - hi);
    const bool take_hi = b.theta > a.theta;
    const Choice& ch = take_hi ? b : a;
    const int32_t sg = take_hi ? hi : lo;

    out->cenv = p.cenv[c_best];
    out->envs = lim->cores / p.cenv[c_best];
    out->ssim = s_sim;
    out->sgen = sg;
    out->strain = 100 - s_sim - sg;
    out->bgen = p.bgen[ch.jg];
    out->btrain = p.btrain[ch.jt];
    out->iterations = steps;
    out->t_sim = t_sim;
    out->t_gen = ch.t_gen;
    out->t_train = ch.t_train;
    out->t_rollout = ch.t_roll;
    out->theta = ch.theta;
    return EBRL_OK;
}

int ebrl_alloc_objective(const ebrl_alloc_profiles* prof, ebrl_alloc_result* out) {
    if (!prof || !out || !profiles_ok(*prof)) return EBRL_E_INVALID;
    const ebrl_alloc_profiles& p = *prof;
    const int32_t jg = index_of(p.bgen, p.n_bgen, out->bgen), jt = index_of(p.btrain, p.n_btrain, out->btrain);
    if (jg < 0 || jt < 0 || out->sgen < 0 || out->sgen > 100 || out->strain < 0 || out->strain > 100 ||
        !(out->t_sim >= 0))
        return EBRL_E_INVALID;
    out->t_gen = quota_rate(p.sgen, p.n_sgen, p.gen_rate, p.n_bgen, jg, out->sgen);
    out->t_train = quota_rate(p.strain, p.n_strain, p.train_rate, p.n_btrain, jt, out->strain);
    out->t_rollout = std::min(out->t_sim, out->t_gen);
    out->theta = std::min(out->t_rollout, out->t_train);
    return EBRL_OK;
}

int ebrl_alloc_monitor_create(int32_t window, double gap, int32_t patience, ebrl_alloc_monitor** out) {
    if (!out || window < 1 || patience < 1 || !(gap >= 0) || !std::isfinite(gap)) return EBRL_E_INVALID;
    ebrl_alloc_monitor* m = new (std::nothrow) ebrl_alloc_monitor;
    if (!m) return EBRL_E_OOM;
    m->window = window;
    m->patience = patience;
    m->gap = gap;
    m->roll.assign(window, 0.0);
    m->train.assign(window, 0.0);
    *out = m;
    return EBRL_OK;
}

int ebrl_alloc_monitor_observe(ebrl_alloc_monitor* m, double rollout_rate, double train_rate, int32_t* trigger) {
    if (!m || !trigger || !(rollout_rate >= 0) || !(train_rate >= 0) || !std::isfinite(rollout_rate) ||
        !std::isfinite(train_rate))
        return EBRL_E_INVALID;
    m->roll[m->head] = rollout_rate;
    m->train[m->head] = train_rate;
    m->head = (m->head + 1) % m->window;
    m->count = std::min(m->count + 1, m->window);
    // averages over the observations held, oldest first
    double sr = 0, st = 0;
    for (int32_t k = 0; k < m->count; ++k) {
        const int32_t i = (m->head - m->count + k + m->window) % m->window;
        sr += m->roll[i];
        st += m->train[i];
    }
    const double ar = sr / m->count, at = st / m->count;
    m->streak = fabs(ar - at) > m->gap * std::max(ar, at) ? m->streak + 1 : 0;
    *trigger = 0;
    if (m->streak >= m->patience) {
        *trigger = 1;
        m->streak = 0;
        m->count = 0;
        m->head = 0;
    }
    return EBRL_OK;
}

void ebrl_alloc_monitor_destroy(ebrl_alloc_monitor* m) { delete m; }

int ebrl_alloc_refine(const ebrl_alloc_profiles* prof, const ebrl_alloc_result* cur, double observed_gen,
                      double observed_train, double* gen_rate_out, double* train_rate_out) {
    if (!prof || !cur || !gen_rate_out || !train_rate_out || !profiles_ok(*prof)) return EBRL_E_INVALID;
    if (!(observed_gen >= 0) || !(observed_train >= 0) || !std::isfinite(observed_gen) ||
        !std::isfinite(observed_train))
        return EBRL_E_INVALID;
    const ebrl_alloc_profiles& p = *prof;
    const int32_t jg = index_of(p.bgen, p.n_bgen, cur->bgen), jt = index_of(p.btrain, p.n_btrain, cur->btrain);
    if (jg < 0 || jt < 0) return EBRL_E_INVALID;
    const double fg = observed_gen > 0 && cur->t_gen > 0 ? observed_gen / cur->t_gen : 1.0;
    const double ft = observed_train > 0 && cur->t_train > 0 ? observed_train / cur->t_train : 1.0;
    for (int32_t i = 0; i < p.n_sgen; ++i)
        for (int32_t j = 0; j < p.n_bgen; ++j) {
            const size_t k = (size_t)i * p.n_bgen + j;
            gen_rate_out[k] = j == jg ? p.gen_rate[k] * fg : p.gen_rate[k];
        }
    for (int32_t i = 0; i < p.n_strain; ++i)
        for (int32_t j = 0; j < p.n_btrain; ++j) {
            const size_t k = (size_t)i * p.n_btrain + j;
            train_rate_out[k] = j == jt ? p.train_rate[k] * ft : p.train_rate[k];
        }
    return EBRL_OK;
}

}  // extern "C"
