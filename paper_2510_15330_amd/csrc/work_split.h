// The decode-attention work split: which contiguous range of the flattened
// step stream each wave takes, and its inverse (which wave took a given
// step).  The attention kernel finds its own range with share_bound; the
// merge kernel finds the waves that covered a cut (request, KV head) with
// wave_of.  The two must agree exactly, so both are written once here and
// compiled for the host as well, where a test checks that wave_of inverts
// share_bound.
//
// The work of a call is the flattened sequence of P units (request b, KV
// head g, step j), request-major, then head, then step, where step j of a
// (request, head) covers its pages [j*PP, min((j+1)*PP, pages)).  Wave w of
// W takes units [share_bound(w), share_bound(w + 1)).
//
// Shares by weight.  Workgroup i runs on XCD i mod 8 (four waves a
// workgroup), and the XCDs stream at measurably different rates.  Wave w
// weighs the weight of its XCD, x(w) = (w / 4) mod 8, and its range starts at
// unit floor(C(w) P / C(W)), C the cumulative weight (equal weights:
// [floor(w P / W), floor((w + 1) P / W))).  Weights apply only to long shares
// (at least kSkewMinSteps steps a wave), where the rate difference, not the
// ramp, sets the finish.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bellman {

constexpr int kSkewMinSteps = 256;   // steps a wave from which the weights apply
constexpr int kMaxSkew = 255;        // even/odd weights 256 +- k stay positive
constexpr int kNumXcds = 8;
constexpr int kMaxXcdWeight = 1023;  // weights 1 .. 1023: C(W) P stays below 2^63

// The share weight of each XCD's waves.
struct XcdWeights {
    int w[kNumXcds];
};

// Even-numbered XCDs 256 + k, odd-numbered 256 - k (k = 0: equal shares).
__host__ __device__ inline XcdWeights skew_weights(int k) {
    XcdWeights x;
    for (int i = 0; i < kNumXcds; ++i) x.w[i] = (i & 1) ? 256 - k : 256 + k;
    return x;
}

// The weights in force for P units over W waves: `x` on long shares, equal
// ones otherwise.
__host__ __device__ inline XcdWeights weights_in_force(const XcdWeights& x, int P, int W) {
    return (int64_t)P >= (int64_t)kSkewMinSteps * W ? x : skew_weights(0);
}

// Sum of the weights of XCDs 0 .. n-1 (constant indices only, so that device
// code keeps the weights in scalar registers).
__host__ __device__ inline int64_t weight_prefix(const XcdWeights& x, int n) {
    int64_t s = 0;
#pragma unroll
    for (int i = 0; i < kNumXcds; ++i) s += i < n ? x.w[i] : 0;
    return s;
}
__host__ __device__ inline int weight_of(const XcdWeights& x, int i) {
    int v = x.w[0];
#pragma unroll
    for (int j = 1; j < kNumXcds; ++j) v = i == j ? x.w[j] : v;
    return v;
}

// C(w): summed weight of waves 0 .. w-1.  A period of 32 waves (eight
// workgroups of four) weighs 4 S, S the sum of the weights.
__host__ __device__ inline int64_t share_weight(int w, const XcdWeights& x) {
    const int q = w >> 5, r = w & 31, i = r >> 2, j = r & 3;
    return (int64_t)q * 4 * weight_prefix(x, kNumXcds) + 4 * weight_prefix(x, i) + (int64_t)j * weight_of(x, i);
}

// First unit of wave w (w = W gives P).  C(W) <= 1023 W and P < 2^31, so the
// product stays below 2^63 for any W < 2^22.
__host__ __device__ inline int share_bound(int w, int P, int W, const XcdWeights& x) {
    return (int)(share_weight(w, x) * P / share_weight(W, x));
}

// The wave v with share_bound(v) <= u < share_bound(v + 1), for 0 <= u < P:
// the largest v whose start is at most u, i.e. the largest v with
// C(v) P < (u + 1) C(W), i.e. C(v) <= c = floor(((u + 1) C(W) - 1) / P).
__host__ __device__ inline int wave_of(int u, int P, int W, const XcdWeights& x) {
    const int64_t c = ((int64_t)(u + 1) * share_weight(W, x) - 1) / P;   // largest admissible C(v)
    const int64_t period = 4 * weight_prefix(x, kNumXcds);
    const int64_t q = c / period;
    int64_t rem = c - q * period;
    int64_t v = 32 * q + 31;
    bool found = false;
#pragma unroll
    for (int i = 0; i < kNumXcds; ++i) {
        const int64_t seg = 4 * (int64_t)x.w[i];
        if (!found && rem < seg) {
            v = 32 * q + 4 * i + rem / x.w[i];
            found = true;
        }
        if (!found) rem -= seg;
    }
    return (int)(v < (int64_t)W - 1 ? v : (int64_t)W - 1);
}

// Whether every wave holds at least one unit: the lightest wave's share
// exceeds one unit, since C(W) <= (heaviest weight) W.
__host__ __device__ inline bool every_wave_holds_units(int P, int W, const XcdWeights& x) {
    int lo = x.w[0], hi = x.w[0];
#pragma unroll
    for (int i = 1; i < kNumXcds; ++i) {
        lo = x.w[i] < lo ? x.w[i] : lo;
        hi = x.w[i] > hi ? x.w[i] : hi;
    }
    return (int64_t)lo * P > (int64_t)hi * W;
}

}  // namespace bellman
