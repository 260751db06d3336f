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
// Shares by weight.  Workgroup i runs on XCD i mod 8, and waves on the
// odd-numbered XCDs were measured to stream 4-5% slower than those on the
// even ones; with skew k the waves of even-XCD workgroups (w / 4 even) weigh
// 256 + k and the others 256 - k, and wave w's range starts at unit
// floor(C(w) P / C(W)), C the cumulative weight (k = 0: equal shares
// [floor(w P / W), floor((w + 1) P / W))).  The skew applies only to long
// shares (at least kSkewMinPages pages a wave: P steps of PP pages each),
// where the rate difference, not the ramp, sets the finish.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bellman {

constexpr int kSkewMinPages = 384;   // pages a wave from which the skew applies
constexpr int kMaxSkew = 255;        // weights stay positive

// The skew in force for P units of PP pages over W waves.
__host__ __device__ inline int share_skew(int skew, int P, int W, int PP) {
    return (int64_t)P * PP >= (int64_t)kSkewMinPages * W ? skew : 0;
}

// C(w): summed weight of waves 0 .. w-1 (period of 8 waves: 4 of an
// even-XCD workgroup, then 4 of an odd one).
__host__ __device__ inline int64_t share_weight(int w, int skew) {
    const int64_t a = 256 + skew, b = 256 - skew;
    const int r = w & 7;
    return (int64_t)(w >> 3) * 4 * (a + b) + (r <= 4 ? r * a : 4 * a + (r - 4) * b);
}

// First unit of wave w (w = W gives P).  C(W) <= 2^9 W and P < 2^31, so the
// product stays below 2^63 for any W < 2^22.
__host__ __device__ inline int share_bound(int w, int P, int W, int skew) {
    return (int)(share_weight(w, skew) * P / share_weight(W, skew));
}

// The wave v with share_bound(v) <= x < share_bound(v + 1), for 0 <= x < P:
// the largest v whose start is at most x, i.e. the largest v with
// C(v) P < (x + 1) C(W).
__host__ __device__ inline int wave_of(int x, int P, int W, int skew) {
    const int64_t a = 256 + skew, b = 256 - skew;
    const int64_t c = ((int64_t)(x + 1) * share_weight(W, skew) - 1) / P;   // largest admissible C(v)
    const int64_t q = c / (4 * (a + b)), rem = c - q * 4 * (a + b);
    const int64_t v = 8 * q + (rem <= 4 * a ? rem / a : 4 + (rem - 4 * a) / b);
    return (int)(v < (int64_t)W - 1 ? v : (int64_t)W - 1);
}

}  // namespace bellman
