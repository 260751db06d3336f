// Host build of the decode-attention work split (the same header the
// kernels compile), exported for tests/test_work_split.py.
#include "../../paper_2510_15330_amd/csrc/work_split.h"

extern "C" {

int ws_skew(int skew, int P, int W, int PP) { return bellman::share_skew(skew, P, W, PP); }

// out[0..W]: first unit of each wave, and P.
void ws_bounds(int P, int W, int skew, int* out) {
    for (int w = 0; w <= W; ++w) out[w] = bellman::share_bound(w, P, W, skew);
}

// out[i] = the wave that holds unit xs[i].
void ws_waves(int P, int W, int skew, const int* xs, long n, int* out) {
    for (long i = 0; i < n; ++i) out[i] = bellman::wave_of(xs[i], P, W, skew);
}

}
