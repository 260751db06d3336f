// Host build of the decode-attention work split (the same header the
// kernels compile), exported for tests/test_work_split.py.
#include "../../paper_2510_15330_amd/csrc/work_split.h"

namespace {
bellman::XcdWeights weights(const int* w) {
    bellman::XcdWeights x;
    for (int i = 0; i < bellman::kNumXcds; ++i) x.w[i] = w[i];
    return x;
}
}  // namespace

extern "C" {

// out[0..7]: the weights in force for P units over W waves.
void ws_in_force(const int* w, int P, int W, int* out) {
    const bellman::XcdWeights x = bellman::weights_in_force(weights(w), P, W);
    for (int i = 0; i < bellman::kNumXcds; ++i) out[i] = x.w[i];
}

// out[0..7]: the even/odd weights of skew k.
void ws_skew_weights(int k, int* out) {
    const bellman::XcdWeights x = bellman::skew_weights(k);
    for (int i = 0; i < bellman::kNumXcds; ++i) out[i] = x.w[i];
}

// out[0..W]: first unit of each wave, and P.
void ws_bounds(int P, int W, const int* w, int* out) {
    const bellman::XcdWeights x = weights(w);
    for (int v = 0; v <= W; ++v) out[v] = bellman::share_bound(v, P, W, x);
}

// out[i] = the wave that holds unit xs[i].
void ws_waves(int P, int W, const int* w, const int* xs, long n, int* out) {
    const bellman::XcdWeights x = weights(w);
    for (long i = 0; i < n; ++i) out[i] = bellman::wave_of(xs[i], P, W, x);
}

int ws_all_units(int P, int W, const int* w) { return bellman::every_wave_holds_units(P, W, weights(w)) ? 1 : 0; }

}
