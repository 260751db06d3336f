// beLLMan's output-length controller (arXiv 2510.15330, Sec. 3).
//
// The scheduler reports the average time between tokens (TBT) once per
// second.  The controller smooths it with a moving average over the last
// `window` reports ("beLLMan in action": 5 seconds), triggers when that
// average exceeds T1 (the median TBT of an unbounded run, "Default unbounded
// run") with a word-reduction rate r = 5%, raises r linearly up to 20% at T2
// (the 75th percentile), and resets r to 0 once the average is back at or
// below T1 ("Placeholder for congestion control").  A request whose predicted
// unbounded length is L is asked for N = L (1 - r) ("Our key proposal"),
// rounded half up, at least 1.  Host code only.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <vector>

#include "../../include/bellman.h"

struct bellman_controller {
    double t1, t2, r_min, r_max;
    int32_t window;
    std::vector<double> ring;  // last `window` samples, oldest first after unrolling
    int32_t count = 0;         // samples pushed so far (saturates at window)
    int32_t head = 0;          // next write position
    double r = 0.0;
};

namespace {

double moving_average(const bellman_controller* c) {
    // Sum from the oldest to the newest sample kept.
    const int32_t n = c->count;
    const int32_t start = (c->head - n + c->window) % c->window;
    double sum = 0.0;
    for (int32_t i = 0; i < n; ++i) sum += c->ring[(size_t)((start + i) % c->window)];
    return sum / (double)n;
}

void push_sample(bellman_controller* c, double tbt) {
    c->ring[(size_t)c->head] = tbt;
    c->head = (c->head + 1) % c->window;
    if (c->count < c->window) ++c->count;
    const double ma = moving_average(c);
    if (!(ma > c->t1)) {
        c->r = 0.0;
    } else if (c->t2 <= c->t1) {
        c->r = c->r_max;
    } else {
        const double r = c->r_min + (c->r_max - c->r_min) * (ma - c->t1) / (c->t2 - c->t1);
        c->r = std::min(std::max(r, c->r_min), c->r_max);
    }
}

// p-th percentile of sorted xs by linear interpolation between neighbours.
double interp_percentile(const std::vector<double>& xs, double p) {
    const double pos = p / 100.0 * (double)(xs.size() - 1);
    const size_t lo = (size_t)floor(pos);
    const size_t hi = std::min(lo + 1, xs.size() - 1);
    return xs[lo] + (xs[hi] - xs[lo]) * (pos - (double)lo);
}

}  // namespace

extern "C" {

bellman_controller_t* bellman_controller_create(double t1, double t2, int32_t window, double r_min, double r_max) {
    if (!isfinite(t1) || !isfinite(t2) || window < 1 || window > (1 << 20)) return nullptr;
    if (!(r_min >= 0.0) || !(r_max >= r_min) || !(r_max < 1.0)) return nullptr;
    bellman_controller* c = new (std::nothrow) bellman_controller;
    if (!c) return nullptr;
    c->t1 = t1;
    c->t2 = t2;
    c->r_min = r_min;
    c->r_max = r_max;
    c->window = window;
    c->ring.assign((size_t)window, 0.0);
    return c;
}

void bellman_controller_destroy(bellman_controller_t* ctl) { delete ctl; }

double bellman_controller_rate(const bellman_controller_t* ctl) {
    return ctl ? ctl->r : (double)BELLMAN_ERR_INVALID_ARG;
}

int32_t bellman_length_cap(const bellman_load_signal_t* s) {
    if (!s || !s->controller) return BELLMAN_ERR_INVALID_ARG;
    if (s->predicted_len < 0) return BELLMAN_ERR_INVALID_ARG;
    if (s->has_sample) {
        if (!isfinite(s->tbt_avg)) return BELLMAN_ERR_INVALID_ARG;
        push_sample(s->controller, s->tbt_avg);
    }
    const double r = s->controller->r;
    const int32_t L = s->predicted_len;
    if (r == 0.0 || L == 0) return L;
    const double n = floor((double)L * (1.0 - r) + 0.5);
    return n < 1.0 ? 1 : (int32_t)n;
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
