// beLLMan's output-length controllers (arXiv 2510.15330): the paper's linear
// controller (Sec. 3) and readings of the controllers its future-work
// section names (Sec. 5, "Toward novel LLM congestion control"), with
// per-class policies ("Nuanced fairness issues").  Host code only.
//
// Linear (Sec. 3): the scheduler reports the average time between tokens
// (TBT) once per second; the controller smooths it with a moving average over
// the last `window` reports ("beLLMan in action": 5 seconds), triggers when
// that average exceeds T1 (the median TBT of an unbounded run, "Default
// unbounded run") with a word-reduction rate r = 5%, raises r linearly up to
// 20% at T2 (the 75th percentile), and resets r to 0 once the average is back
// at or below T1 ("Placeholder for congestion control").  A request whose
// predicted unbounded length is L is asked for N = L (1 - r) ("Our key
// proposal"), rounded half up, at least 1.
//
// The variants (MPC, BBR-style, PCC) observe one tick at a time: whether TBT
// samples arrived, their mean, the tokens they decoded and the tick length.
// Their rules are stated with the entry points in bellman.h.  Every
// expression is evaluated in binary64 in the order written, with no fused
// multiply-adds, so that results are reproducible operation for operation.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <vector>

#include "../../include/bellman.h"

#pragma clang fp contract(off)

struct bellman_controller {
    bellman_ctl_params_t p;
    double r = 0.0;
    // linear: ring of the last `window` samples
    std::vector<double> ring;
    int32_t count = 0;         // samples pushed so far (saturates at window)
    int32_t head = 0;          // next write position
    // MPC, BBR: recent TBT samples and delivery rates (oldest first)
    std::vector<double> ys, xs;
    int64_t ticks = 0;
    double r_base = 0.0;
    // PCC
    double center = 0.0;
    int64_t round = 0;
    bool second = false;
    double acc = 0.0;
    int64_t n_acc = 0, mi_ticks = 0;
    double first_r = 0.0, first_u = 0.0;
};

namespace {

double moving_average(const bellman_controller* c) {
    // Sum from the oldest to the newest sample kept.
    const int32_t n = c->count;
    const int32_t w = c->p.window;
    const int32_t start = (c->head - n + w) % w;
    double sum = 0.0;
    for (int32_t i = 0; i < n; ++i) sum += c->ring[(size_t)((start + i) % w)];
    return sum / (double)n;
}

void push_linear(bellman_controller* c, double tbt) {
    const bellman_ctl_params_t& p = c->p;
    c->ring[(size_t)c->head] = tbt;
    c->head = (c->head + 1) % p.window;
    if (c->count < p.window) ++c->count;
    const double ma = moving_average(c);
    if (!(ma > p.t1)) {
        c->r = 0.0;
    } else if (p.t2 <= p.t1) {
        c->r = p.r_max;
    } else {
        const double r = p.r_min + (p.r_max - p.r_min) * (ma - p.t1) / (p.t2 - p.t1);
        c->r = std::min(std::max(r, p.r_min), p.r_max);
    }
}

// keep at most `keep` newest values
void push_bounded(std::vector<double>& v, double x, size_t keep) {
    v.push_back(x);
    if (v.size() > keep) v.erase(v.begin(), v.begin() + (ptrdiff_t)(v.size() - keep));
}

double min_last(const std::vector<double>& v, size_t k) {
    const size_t n = std::min(k, v.size());
    double m = v[v.size() - n];
    for (size_t i = v.size() - n + 1; i < v.size(); ++i) m = std::min(m, v[i]);
    return m;
}

double max_last(const std::vector<double>& v, size_t k) {
    const size_t n = std::min(k, v.size());
    double m = v[v.size() - n];
    for (size_t i = v.size() - n + 1; i < v.size(); ++i) m = std::max(m, v[i]);
    return m;
}

double clamp(double x, double lo, double hi) { return std::min(std::max(x, lo), hi); }

// MPC: least-squares trend over the last `window` samples (slope per tick,
// value at the newest sample); before the window fills, no trend.
void mpc_trend(const bellman_controller* c, double* s, double* v) {
    const int32_t m = c->p.window;
    if ((int64_t)c->ys.size() < m || m < 2) {
        *s = 0.0;
        *v = c->ys.back();
        return;
    }
    const size_t off = c->ys.size() - (size_t)m;
    const double tm = (double)(m - 1) / 2.0;
    double total = 0.0;
    for (int32_t t = 0; t < m; ++t) total += c->ys[off + (size_t)t];
    const double ym = total / (double)m;
    double sxy = 0.0, sxx = 0.0;
    for (int32_t t = 0; t < m; ++t) {
        sxy += ((double)t - tm) * (c->ys[off + (size_t)t] - ym);
        sxx += ((double)t - tm) * ((double)t - tm);
    }
    *s = sxy / sxx;
    *v = ym + *s * ((double)(m - 1) - tm);
}

double mpc_cost(const bellman_controller* c, double rc, double s, double v, double b) {
    const bellman_ctl_params_t& p = c->p;
    double J = 0.0;
    for (int32_t h = 1; h <= p.horizon; ++h) {
        const double u = std::max(v + s * (double)h, b);
        const double f = 1.0 - exp(-(double)h / p.tau);
        const double y = b + (u - b) * ((1.0 - f) + f * (1.0 - rc) / (1.0 - c->r));
        const double e = std::max(0.0, y - p.t1) / (p.t2 - p.t1);
        J += p.w_lat * e * e;
    }
    const double d = (rc - c->r) / p.r_max;
    return J + (double)p.horizon * (p.w_quality - p.w_energy) * rc + p.w_delta * d * d;
}

void observe_mpc(bellman_controller* c, const bellman_ctl_obs_t* o) {
    const bellman_ctl_params_t& p = c->p;
    if (!o->has_sample) return;
    push_bounded(c->ys, o->tbt_avg, (size_t)std::max(p.window, p.floor_window));
    double s, v;
    mpc_trend(c, &s, &v);
    const double b = min_last(c->ys, (size_t)p.floor_window);
    double best = 0.0, best_j = INFINITY;
    auto consider = [&](double rc) {
        const double J = mpc_cost(c, rc, s, v, b);
        if (J < best_j) {
            best = rc;
            best_j = J;
        }
    };
    consider(0.0);
    for (int64_t i = 0;; ++i) {
        const double rc = p.r_min + (double)i * p.step;
        if (!(rc < p.r_max)) break;
        consider(rc);
    }
    consider(p.r_max);
    c->r = best;
}

void observe_bbr(bellman_controller* c, const bellman_ctl_obs_t* o) {
    const bellman_ctl_params_t& p = c->p;
    const double x = o->tokens / o->tick_s;
    push_bounded(c->xs, x, (size_t)p.bw_window);
    c->ticks += 1;
    if (o->has_sample) {
        push_bounded(c->ys, o->tbt_avg, (size_t)p.rt_window);
        const double btlbw = max_last(c->xs, (size_t)p.bw_window);
        const double rtprop = min_last(c->ys, (size_t)p.rt_window);
        if (o->tbt_avg > rtprop * (1.0 + p.margin) && x >= (1.0 - p.margin) * btlbw)
            c->r_base = std::min(c->r_base + p.bbr_step, p.r_max);
        else if (o->tbt_avg <= rtprop * (1.0 + p.margin / 2.0))
            c->r_base = std::max(c->r_base - p.bbr_step, 0.0);
    }
    const int64_t phase = (c->ticks - 1) % p.cycle;
    const double off = phase == 0 ? -p.probe : (phase == 1 ? p.probe : 0.0);
    c->r = clamp(c->r_base + off, 0.0, p.r_max);
}

double pcc_rate(const bellman_controller* c) {
    const bool up = (c->round % 2 == 0) != c->second;
    const double d = up ? c->p.epsilon : -c->p.epsilon;
    return clamp(c->center + d, 0.0, c->p.r_max);
}

void observe_pcc(bellman_controller* c, const bellman_ctl_obs_t* o) {
    const bellman_ctl_params_t& p = c->p;
    if (o->has_sample) {
        c->acc += o->tbt_avg;
        c->n_acc += 1;
    }
    c->mi_ticks += 1;
    if (c->mi_ticks < p.interval) return;
    double lat = 0.0;
    if (c->n_acc) lat = std::max(0.0, c->acc / (double)c->n_acc - p.t1) / (p.t2 - p.t1);
    const double U = -p.pcc_w_lat * lat - p.pcc_w_quality * c->r / p.r_max;
    if (!c->second) {
        c->first_r = c->r;
        c->first_u = U;
        c->second = true;
    } else {
        const double g = c->first_r == c->r ? 0.0 : (c->first_u - U) / (c->first_r - c->r);
        c->center = clamp(c->center + p.gain * g, 0.0, p.r_max);
        c->second = false;
        c->round += 1;
    }
    c->acc = 0.0;
    c->n_acc = 0;
    c->mi_ticks = 0;
    c->r = pcc_rate(c);
}

int32_t cap(double r, int32_t L) {
    if (r == 0.0 || L == 0) return L;
    const double n = floor((double)L * (1.0 - r) + 0.5);
    return n < 1.0 ? 1 : (int32_t)n;
}

bool finite_nonneg(double x) { return isfinite(x) && x >= 0.0; }

// p-th percentile of sorted xs by linear interpolation between neighbours.
double interp_percentile(const std::vector<double>& xs, double p) {
    const double pos = p / 100.0 * (double)(xs.size() - 1);
    const size_t lo = (size_t)floor(pos);
    const size_t hi = std::min(lo + 1, xs.size() - 1);
    return xs[lo] + (xs[hi] - xs[lo]) * (pos - (double)lo);
}

}  // namespace

extern "C" {

int bellman_ctl_params_default(int32_t kind, double t1, double t2, bellman_ctl_params_t* p) {
    if (!p || kind < BELLMAN_CTL_LINEAR || kind > BELLMAN_CTL_PCC) return BELLMAN_ERR_INVALID_ARG;
    memset(p, 0, sizeof(*p));
    p->kind = kind;
    p->window = 5;
    p->t1 = t1;
    p->t2 = t2;
    p->r_min = 0.05;
    p->r_max = 0.20;
    p->horizon = 10;
    p->floor_window = 60;
    p->tau = 20.0;
    p->w_lat = 1.0;
    p->w_quality = 0.25;
    p->w_energy = 0.1;
    p->w_delta = 0.2;
    p->step = 0.01;
    p->bw_window = 10;
    p->rt_window = 30;
    p->cycle = 8;
    p->margin = 0.25;
    p->bbr_step = 0.02;
    p->probe = 0.02;
    p->interval = 10;
    p->epsilon = 0.02;
    p->gain = 0.02;
    p->pcc_w_lat = 1.0;
    p->pcc_w_quality = 0.5;
    return BELLMAN_OK;
}

bellman_controller_t* bellman_controller_create_ex(const bellman_ctl_params_t* p) {
    if (!p || p->kind < BELLMAN_CTL_LINEAR || p->kind > BELLMAN_CTL_PCC) return nullptr;
    if (!isfinite(p->t1) || !isfinite(p->t2)) return nullptr;
    if (!(p->r_min >= 0.0) || !(p->r_max >= p->r_min) || !(p->r_max < 1.0)) return nullptr;
    switch (p->kind) {
        case BELLMAN_CTL_LINEAR:
            if (p->window < 1 || p->window > (1 << 20)) return nullptr;
            break;
        case BELLMAN_CTL_MPC:
            if (!(p->t2 > p->t1) || !(p->r_max > 0.0) || p->window < 1 || p->window > (1 << 20) || p->horizon < 1 ||
                p->horizon > 100000 || p->floor_window < 1 || p->floor_window > (1 << 20) || !(p->tau > 0.0) ||
                !isfinite(p->tau) || !finite_nonneg(p->w_lat) || !finite_nonneg(p->w_quality) ||
                !finite_nonneg(p->w_energy) || !finite_nonneg(p->w_delta) || !(p->step > 0.0) || !isfinite(p->step))
                return nullptr;
            break;
        case BELLMAN_CTL_BBR:
            if (p->bw_window < 1 || p->bw_window > (1 << 20) || p->rt_window < 1 || p->rt_window > (1 << 20) ||
                p->cycle < 1 || !finite_nonneg(p->margin) || !(p->margin < 1.0) || !finite_nonneg(p->bbr_step) ||
                !finite_nonneg(p->probe))
                return nullptr;
            break;
        case BELLMAN_CTL_PCC:
            if (!(p->t2 > p->t1) || !(p->r_max > 0.0) || p->interval < 1 || !finite_nonneg(p->epsilon) ||
                !finite_nonneg(p->gain) || !finite_nonneg(p->pcc_w_lat) || !finite_nonneg(p->pcc_w_quality))
                return nullptr;
            break;
    }
    bellman_controller* c = new (std::nothrow) bellman_controller;
    if (!c) return nullptr;
    c->p = *p;
    if (p->kind == BELLMAN_CTL_LINEAR) c->ring.assign((size_t)p->window, 0.0);
    if (p->kind == BELLMAN_CTL_PCC) c->r = pcc_rate(c);
    return c;
}

bellman_controller_t* bellman_controller_create(double t1, double t2, int32_t window, double r_min, double r_max) {
    bellman_ctl_params_t p;
    bellman_ctl_params_default(BELLMAN_CTL_LINEAR, t1, t2, &p);
    p.window = window;
    p.r_min = r_min;
    p.r_max = r_max;
    return bellman_controller_create_ex(&p);
}

void bellman_controller_destroy(bellman_controller_t* ctl) { delete ctl; }

double bellman_controller_rate(const bellman_controller_t* ctl) {
    return ctl ? ctl->r : (double)BELLMAN_ERR_INVALID_ARG;
}

double bellman_controller_observe(bellman_controller_t* ctl, const bellman_ctl_obs_t* obs) {
    if (!ctl || !obs) return (double)BELLMAN_ERR_INVALID_ARG;
    if (obs->has_sample && !isfinite(obs->tbt_avg)) return (double)BELLMAN_ERR_INVALID_ARG;
    if (!finite_nonneg(obs->tokens) || !(obs->tick_s > 0.0) || !isfinite(obs->tick_s))
        return (double)BELLMAN_ERR_INVALID_ARG;
    switch (ctl->p.kind) {
        case BELLMAN_CTL_LINEAR:
            if (obs->has_sample) push_linear(ctl, obs->tbt_avg);
            break;
        case BELLMAN_CTL_MPC: observe_mpc(ctl, obs); break;
        case BELLMAN_CTL_BBR: observe_bbr(ctl, obs); break;
        case BELLMAN_CTL_PCC: observe_pcc(ctl, obs); break;
    }
    return ctl->r;
}

int32_t bellman_length_cap(const bellman_load_signal_t* s) {
    if (!s || !s->controller) return BELLMAN_ERR_INVALID_ARG;
    if (s->predicted_len < 0) return BELLMAN_ERR_INVALID_ARG;
    if (s->has_sample) {
        const bellman_ctl_obs_t o{1, 0, s->tbt_avg, 0.0, 1.0};
        if (bellman_controller_observe(s->controller, &o) < 0.0) return BELLMAN_ERR_INVALID_ARG;
    }
    return cap(s->controller->r, s->predicted_len);
}

int32_t bellman_length_cap_class(const bellman_controller_t* ctl, int32_t predicted_len,
                                 const bellman_class_policy_t* policy) {
    if (!ctl || !policy || predicted_len < 0 || !finite_nonneg(policy->weight)) return BELLMAN_ERR_INVALID_ARG;
    if (predicted_len <= policy->bypass_len) return predicted_len;
    const double rc = std::min(policy->weight * ctl->r, ctl->p.r_max);
    return cap(rc, predicted_len);
}

int bellman_calibrate_thresholds(const double* tbt, int64_t n, double* t1, double* t2) {
    if (!tbt || n < 1 || !t1 || !t2) return BELLMAN_ERR_INVALID_ARG;
    std::vector<double> xs(tbt, tbt + n);
    for (double v : xs)
        if (!isfinite(v)) return BELLMAN_ERR_INVALID_ARG;
    std::sort(xs.begin(), xs.end());
    *t1 = interp_percentile(xs, 50.0);
    *t2 = interp_percentile(xs, 75.0);
    return BELLMAN_OK;
}

}  // extern "C"
