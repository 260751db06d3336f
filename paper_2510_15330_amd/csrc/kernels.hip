// HIP kernels for gfx950: KV append, split planning, split-K partial decode
// attention on the matrix cores, and the log-sum-exp merge of the partials.
//
// The computation is one decode step of the serving loop that beLLMan
// (arXiv 2510.15330, Sec. 3) controls: every request attends its one new
// query token over its own KV cache (prompt plus tokens generated so far).
#include "internal.h"
#include "work_split.h"

#include <math.h>

#include <type_traits>

namespace bellman {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Two e4m3fn codes (the low or high 16 bits of w) -> two bf16, exactly (every
// e4m3fn value is representable in bf16; the scale operand is 1).
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t w, bool high) {
    bf16x2 r = high ? __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true)
                    : __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false);
    return __builtin_bit_cast(uint32_t, r);
}

// ------------------------------------------------------------- KV append ---
// x / scale rounded to OCP e4m3fn: nearest, ties to the even mantissa,
// saturating at +-448, NaN kept.  The quotient is one correctly rounded
// binary32 division.
__device__ __forceinline__ uint32_t quantize_e4m3fn(float x, float scale) {
    const float v = __fdiv_rn(x, scale);
    const uint32_t u = __float_as_uint(v);
    const uint32_t sign = (u >> 24) & 0x80u;
    const uint32_t a = u & 0x7fffffffu;
    if (a > 0x7f800000u) return sign | 0x7fu;          // NaN
    if (a >= 0x43e00000u) return sign | 0x7eu;         // |v| >= 448 (and inf)
    if (a < 0x3c800000u)                                // |v| < 2^-6: multiples of 2^-9
        return sign | (uint32_t)__builtin_rintf(__uint_as_float(a) * 512.0f);
    uint32_t e = (a >> 23) - 120u;                      // e4m3 biased exponent, 1..15
    uint32_t q = (a >> 20) & 7u;                        // top three mantissa bits
    const uint32_t rem = a & 0xfffffu;
    if (rem > 0x80000u || (rem == 0x80000u && (q & 1u))) ++q;
    if (q == 8u) {
        q = 0u;
        ++e;
    }
    return sign | (e << 3) | q;                         // below 448 nothing rounds past 448
}

// One workgroup per request: write the new K row into its 16-byte chunks and
// the new V row into its slot column (copying codes, or quantising bf16 rows
// into fp8 pools), then advance the request's length.  Every 32-byte sector
// the row touches is written whole: the neighbouring slot's K chunk and the
// rest of the V dim rows are read back and stored unchanged.  The attention
// kernel reads these lines right after, and lines left holding partial
// writes read back more slowly (measured: 8.6 us of a 1.5 ms attention call
// over 256 requests).  Work items are K chunks and V sectors (one bf16 dim
// row, or two fp8 dim rows); each thread issues the source loads of up to
// kAppendPer items before the length and block-table reads return, then the
// sector reads, then the stores.
constexpr int kAppendPer = 4;

// Element at byte `pos` (NB bytes) of a 32-byte sector held as two 16-byte
// words set to e; each word is selected by its own comparison, so the sector
// stays in registers.
template <int NB>
__device__ __forceinline__ void put_elem(u32x4& q0, u32x4& q1, int pos, uint32_t e) {
    const int wi = pos >> 2, sh = 8 * (pos & 3);
    const uint32_t keep = ~((NB == 2 ? 0xffffu : 0xffu) << sh), add = e << sh;
    q0.x = wi == 0 ? (q0.x & keep) | add : q0.x;
    q0.y = wi == 1 ? (q0.y & keep) | add : q0.y;
    q0.z = wi == 2 ? (q0.z & keep) | add : q0.z;
    q0.w = wi == 3 ? (q0.w & keep) | add : q0.w;
    q1.x = wi == 4 ? (q1.x & keep) | add : q1.x;
    q1.y = wi == 5 ? (q1.y & keep) | add : q1.y;
    q1.z = wi == 6 ? (q1.z & keep) | add : q1.z;
    q1.w = wi == 7 ? (q1.w & keep) | add : q1.w;
}

template <int EB, bool QUANT>
__device__ __forceinline__ void append_rows(const AppendArgs& a, int b, int pg, int slot, bool ok) {
    constexpr int X = 16 / EB;                  // pool elements per 16-byte K chunk
    constexpr int DV = 32 / (kPage * EB);       // V dims per 32-byte sector: 1 (bf16) or 2 (fp8)
    constexpr int SB = QUANT ? 2 : EB;          // source element bytes
    const int chunks = a.D / X, vsec = a.D / DV;
    const int nk = a.H_kv * chunks, nv = a.H_kv * vsec;
    const int64_t tile_bytes = (int64_t)a.D * kPage * EB;
    char* kp = (char*)a.k_pages;
    char* vp = (char*)a.v_pages;
    const char* kn = (const char*)a.k_new;
    const char* vn = (const char*)a.v_new;
    for (int base = 0; base < nk + nv; base += kAppendPer * (int)blockDim.x) {
        // the new row's pieces (independent of the page)
        u32x4 lo[kAppendPer], hi[kAppendPer];
#pragma unroll
        for (int j = 0; j < kAppendPer; ++j) {
            const int it = base + j * (int)blockDim.x + (int)threadIdx.x;
            if (it < nk) {
                const int g = it / chunks, c = it - g * chunks;
                const char* src = kn + ((int64_t)b * a.new_sb + (int64_t)g * a.new_sh + (int64_t)c * X) * SB;
                lo[j] = *(const u32x4*)src;
                if (QUANT) hi[j] = *(const u32x4*)(src + 16);
            } else if (it < nk + nv) {
                const int iv = it - nk;
                const int g = iv / vsec, d0 = (iv - g * vsec) * DV;
                const char* src = vn + ((int64_t)b * a.vnew_sb + (int64_t)g * a.vnew_sh + d0) * SB;
                lo[j].x = DV * SB == 4 ? *(const uint32_t*)src : (uint32_t)*(const uint16_t*)src;
            }
        }
        if (!ok) return;
        // the rest of each sector
        u32x4 o0[kAppendPer], o1[kAppendPer];
#pragma unroll
        for (int j = 0; j < kAppendPer; ++j) {
            const int it = base + j * (int)blockDim.x + (int)threadIdx.x;
            if (it < nk) {
                const int g = it / chunks, c = it - g * chunks;
                o0[j] = *(const u32x4*)(kp + ((((int64_t)pg * a.H_kv + g) * chunks + c) * kPage + (slot ^ 1)) * 16);
            } else if (it < nk + nv) {
                const int iv = it - nk;
                const int g = iv / vsec, d0 = (iv - g * vsec) * DV;
                const char* sec = vp + ((int64_t)pg * a.H_kv + g) * tile_bytes + (int64_t)d0 * kPage * EB;
                o0[j] = *(const u32x4*)sec;
                o1[j] = *(const u32x4*)(sec + 16);
            }
        }
#pragma unroll
        for (int j = 0; j < kAppendPer; ++j) {
            const int it = base + j * (int)blockDim.x + (int)threadIdx.x;
            if (it < nk) {
                const int g = it / chunks, c = it - g * chunks;
                char* chunk = kp + (((int64_t)pg * a.H_kv + g) * chunks + c) * kPage * 16;
                u32x4 w = lo[j];
                if (QUANT) {   // 16 bf16 -> 16 e4m3fn codes with the (request, head)'s K scale
                    const float ks = a.k_scale[(int64_t)b * a.H_kv + g];
                    const uint32_t in[8] = {lo[j].x, lo[j].y, lo[j].z, lo[j].w, hi[j].x, hi[j].y, hi[j].z, hi[j].w};
                    uint32_t ow[4];
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const uint32_t l2 = in[2 * k], h2 = in[2 * k + 1];
                        ow[k] = quantize_e4m3fn(__uint_as_float(l2 << 16), ks) |
                                (quantize_e4m3fn(__uint_as_float(l2 & 0xffff0000u), ks) << 8) |
                                (quantize_e4m3fn(__uint_as_float(h2 << 16), ks) << 16) |
                                (quantize_e4m3fn(__uint_as_float(h2 & 0xffff0000u), ks) << 24);
                    }
                    w = u32x4{ow[0], ow[1], ow[2], ow[3]};
                }
                *(u32x4*)(chunk + slot * 16) = w;
                *(u32x4*)(chunk + (slot ^ 1) * 16) = o0[j];
            } else if (it < nk + nv) {
                const int iv = it - nk;
                const int g = iv / vsec, d0 = (iv - g * vsec) * DV;
                char* sec = vp + ((int64_t)pg * a.H_kv + g) * tile_bytes + (int64_t)d0 * kPage * EB;
                u32x4 q0 = o0[j], q1 = o1[j];
                const uint32_t v = lo[j].x;
                if (EB == 2) {
                    put_elem<2>(q0, q1, 2 * slot, v & 0xffffu);
                } else if (QUANT) {   // two bf16 dims -> e4m3fn codes with the V scale
                    const float vs = a.v_scale[(int64_t)b * a.H_kv + g];
                    put_elem<1>(q0, q1, slot, quantize_e4m3fn(__uint_as_float(v << 16), vs));
                    put_elem<1>(q0, q1, 16 + slot, quantize_e4m3fn(__uint_as_float(v & 0xffff0000u), vs));
                } else {
                    put_elem<1>(q0, q1, slot, v & 0xffu);
                    put_elem<1>(q0, q1, 16 + slot, (v >> 8) & 0xffu);
                }
                *(u32x4*)sec = q0;
                *(u32x4*)(sec + 16) = q1;
            }
        }
    }
}

__global__ void __launch_bounds__(512) kv_append_kernel(AppendArgs a) {
    const int b = blockIdx.x;
    const int L = a.seq_lens[b];
    const int pi = L >> 4;
    const bool in_table = L >= 0 && pi < a.max_pages;
    const int pg = in_table ? a.block_table[(int64_t)b * a.bt_stride + pi] : -1;
    const bool ok = pg >= 0 && (int64_t)pg < a.num_pages;
    if (!ok && threadIdx.x == 0) atomicOr(a.err, kErrAppendSlot);
    const int slot = L & (kPage - 1);
    if (a.quant) append_rows<1, true>(a, b, pg, slot, ok);
    else if (a.elem_bytes == 2) append_rows<2, false>(a, b, pg, slot, ok);
    else append_rows<1, false>(a, b, pg, slot, ok);
    if (!ok) return;
    __syncthreads();  // every thread has read seq_lens[b]
    if (threadIdx.x == 0) a.seq_lens[b] = L + 1;
}

// ---------------------------------------------------------- work split ---
// Each wave finds its own range of the flattened step stream (work_split.h)
// from the lengths (no planner launch): it sums the steps of the whole batch,
// then scans the requests' first units up to the one holding its first unit.
// Lengths are clamped to the block-table width.  A step costs the same
// whether it holds PP pages or the last few (its loads are issued for all PP
// pages), so dealing steps rather than pages keeps the waves' times equal
// when many requests end in a short step.  Requests are split only where a
// wave boundary falls inside them, and always between steps.
constexpr int kPlanPerLane = 16;                        // lengths per lane per load batch
constexpr int kPlanBatch = kPlanPerLane * kWaveSize;   // 1024 requests

__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
    for (int o = 1; o < kWaveSize; o <<= 1) {
        const int t = __shfl_up(v, o, kWaveSize);
        if (lane >= o) v += t;
    }
    return v;
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int o = kWaveSize / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWaveSize);
    return v;
}

// ------------------------------------------------ partial attention (MFMA) --
// Each wave walks its contiguous share of the planner's steps, a step being
// PP consecutive pages of one (request b, KV head g); for bf16 pages:
//   S^T[slot, head] = K_page[slot, :] . Q^T[:, head]   (v_mfma 16x16x32 bf16)
//   online softmax per head in base 2, once per step
//   O^T[dim, head] += V_pair^T[dim, token] . P^T[token, head]  (v_mfma 16x16x32)
// Lane l = 16*qg + n.  In the QK product n is the page slot (A row) and the
// query head of the group (B column); the result leaves lane (qg, n) with the
// scores of head n at slots 4qg..4qg+3 of each page of the pair.  Those eight
// scores are exactly the eight B elements the PV product needs from that lane
// (the contraction index is paired with tokens the same way in the A operand),
// so nothing crosses lanes except the max/sum reductions over qg.  P enters
// the PV product as a bf16 pair hi + lo (hi = P truncated to bf16, lo = the
// remainder truncated), which keeps P to about 2^-14 relative.  Slots past the
// request's length are excluded: their scores become -inf and their V
// elements are replaced by zeros.  O is rescaled only when a running max
// grows (exact: otherwise the factor is 1).
// One page of one KV head as this lane holds it.
template <int D, bool FP8>
struct PageK {
    static constexpr int KC = FP8 ? D / 64 : D / 32;  // 16-byte K loads per lane
    u32x4 k[KC];
};
template <int D, bool FP8>
struct PageV {
    typename std::conditional<FP8, uint32_t, u32x2>::type v[D / 16];
};

// K/V pages are read exactly once per step: non-temporal loads keep them from
// displacing reusable lines in the caches, which measurably raises the
// sustained read rate of the gather.
template <typename T>
__device__ __forceinline__ T ld_stream(const char* p) {
    return __builtin_nontemporal_load((const T*)p);
}

template <int D, bool FP8>
__device__ __forceinline__ void load_k(PageK<D, FP8>& r, const char* kbase, int qg, int n) {
    if constexpr (!FP8) {
        // chunk c = 4j + qg (8 dims), slot n: 16 bytes; one instruction covers 1 KiB
#pragma unroll
        for (int j = 0; j < PageK<D, FP8>::KC; ++j)
            r.k[j] = ld_stream<u32x4>(kbase + ((size_t)((4 * j + qg) * kPage + n)) * 16);
    } else {
        // chunk c = qg + 4i (16 dims), slot n: 16 bytes
#pragma unroll
        for (int i = 0; i < PageK<D, FP8>::KC; ++i)
            r.k[i] = ld_stream<u32x4>(kbase + ((size_t)((qg + 4 * i) * kPage + n)) * 16);
    }
}

template <int D, bool FP8>
__device__ __forceinline__ void load_v(PageV<D, FP8>& r, const char* vbase, int qg, int n) {
    // dims 16t + n, slots 4qg..4qg+3; an instruction covers 512 (bf16) or 256 (fp8) bytes
#pragma unroll
    for (int t = 0; t < D / 16; ++t) {
        if constexpr (!FP8)
            r.v[t] = ld_stream<u32x2>(vbase + ((size_t)((16 * t + n) * kPage + 4 * qg)) * 2);
        else
            r.v[t] = ld_stream<uint32_t>(vbase + (size_t)((16 * t + n) * kPage + 4 * qg));
    }
}

// Four-page fp8 steps hold V by page: lane (qg, n) reads the whole 16-slot
// row of dim 16t + n of page qg (16 bytes), so one instruction covers all four
// pages' 256-byte row blocks of tile t.  rv[j].v[t] is the row's dword j
// (slots 4j..4j+3).
template <int D>
__device__ __forceinline__ void load_v_rows(PageV<D, true> (&rv)[4], const char* vbase, int n) {
#pragma unroll
    for (int t = 0; t < D / 16; ++t) {
        const u32x4 w = ld_stream<u32x4>(vbase + (size_t)(16 * t + n) * kPage);
        rv[0].v[t] = w.x;
        rv[1].v[t] = w.y;
        rv[2].v[t] = w.z;
        rv[3].v[t] = w.w;
    }
}

// Scores of one page: lane (qg, n) gets head n at slots 4qg..4qg+3.
template <int D, bool FP8>
__device__ __forceinline__ f32x4 page_scores(const PageK<D, FP8>& r, const bf16x8 (&bq)[D / 32]) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < D / 32; ++j) {
        u32x4 kk;
        if constexpr (!FP8) {
            kk = r.k[j];
        } else {
            const u32x4 w = r.k[j >> 1];
            const uint32_t w0 = (j & 1) ? w.z : w.x;
            const uint32_t w1 = (j & 1) ? w.w : w.y;
            kk.x = fp8x2_to_bf16x2(w0, false);
            kk.y = fp8x2_to_bf16x2(w0, true);
            kk.z = fp8x2_to_bf16x2(w1, false);
            kk.w = fp8x2_to_bf16x2(w1, true);
        }
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kk), bq[j], acc, 0, 0, 0);
    }
    return acc;
}

// Four bf16 V elements (slots 4qg..4qg+3 of dim 16t + n) as the lane's half
// of a PV A operand, zeroed at slots >= nv.
template <int D, bool FP8>
__device__ __forceinline__ u32x2 v_quad(const PageV<D, FP8>& r, int t, int nv, int qg) {
    u32x2 vv;
    if constexpr (!FP8) {
        vv = r.v[t];
    } else {
        vv.x = fp8x2_to_bf16x2(r.v[t], false);
        vv.y = fp8x2_to_bf16x2(r.v[t], true);
    }
    if (nv < kPage) {
        const int k = nv - 4 * qg;  // live elements among this lane's four
        vv.x &= k >= 2 ? 0xffffffffu : (k == 1 ? 0x0000ffffu : 0u);
        vv.y &= k >= 4 ? 0xffffffffu : (k == 3 ? 0x0000ffffu : 0u);
    }
    return vv;
}

// Reductions over the four 16-lane groups (lanes n, n+16, n+32, n+48): a
// 16-lane swap pairs groups 0/1 and 2/3, a 32-lane swap pairs the halves.
// Both are plain VALU permutes, off the LDS path a lane shuffle would take;
// every lane of a column ends with the same bits.
__device__ __forceinline__ float group_max4(float x) {
    const unsigned u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const unsigned v = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float group_sum4(float x) {
    const unsigned u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const unsigned v = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

template <int D>
struct AttnState {
    f32x4 o[D / 16];
    float m;   // running max, log2 units (same in the four qg lanes of a head)
    float l;   // this lane's partial sum of weights
};

// Pack the upper halves of two fp32 bit patterns into one bf16 pair.
__device__ __forceinline__ uint32_t pack_hi16(uint32_t lo, uint32_t hi) {
    return __builtin_amdgcn_perm(hi, lo, 0x07060302u);
}

// Online softmax over one page's scores, then O += V^T P^T for the page.
template <int D, bool FP8>
__device__ __forceinline__ void page_pv(AttnState<D>& st, f32x4 sc, const PageV<D, FP8>& pv, float sl, int nv,
                                        int qg) {
    constexpr int NT = D / 16;
    float x[4];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[i] = (4 * qg + i < nv) ? sc[i] * sl : -INFINITY;
        mx = fmaxf(mx, x[i]);
    }
    mx = group_max4(mx);
    const float m_new = fmaxf(st.m, mx);
    if (__any(m_new > st.m)) {
        const float alpha = fast_exp2(st.m - m_new);
        st.l *= alpha;
#pragma unroll
        for (int t = 0; t < NT; ++t) st.o[t] *= alpha;
        st.m = m_new;
    }
    const float p0 = fast_exp2(x[0] - st.m), p1 = fast_exp2(x[1] - st.m);
    const float p2 = fast_exp2(x[2] - st.m), p3 = fast_exp2(x[3] - st.m);
    st.l += (p0 + p1) + (p2 + p3);
    const uint32_t u0 = __float_as_uint(p0), u1 = __float_as_uint(p1);
    const uint32_t u2 = __float_as_uint(p2), u3 = __float_as_uint(p3);
    const uint32_t r0 = __float_as_uint(p0 - __uint_as_float(u0 & 0xffff0000u));
    const uint32_t r1 = __float_as_uint(p1 - __uint_as_float(u1 & 0xffff0000u));
    const uint32_t r2 = __float_as_uint(p2 - __uint_as_float(u2 & 0xffff0000u));
    const uint32_t r3 = __float_as_uint(p3 - __uint_as_float(u3 & 0xffff0000u));
    const s16x4 bph = __builtin_bit_cast(s16x4, u32x2{pack_hi16(u0, u1), pack_hi16(u2, u3)});
    const s16x4 bpl = __builtin_bit_cast(s16x4, u32x2{pack_hi16(r0, r1), pack_hi16(r2, r3)});
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const s16x4 av = __builtin_bit_cast(s16x4, v_quad<D, FP8>(pv, t, nv, qg));
        st.o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, bph, st.o[t], 0, 0, 0);
        st.o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, bpl, st.o[t], 0, 0, 0);
    }
}

// Online softmax over the scores of PP consecutive pages (PP = 2 or 4), then
// O += V^T P^T with 16x16x32 products over page pairs: in the A operand a
// lane's elements 0..3 are its four slots of the pair's first page and 4..7
// its four slots of the second, the same tokens its eight P elements (B
// operand) carry.
template <int D, bool FP8, int PP>
__device__ __forceinline__ void group_pv(AttnState<D>& st, const f32x4 (&sc)[PP], const PageV<D, FP8> (&pv)[PP],
                                         float sl, const int (&nv)[PP], int qg) {
    constexpr int NT = D / 16;
    float x[4 * PP];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < PP; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            x[4 * i + r] = (4 * qg + r < nv[i]) ? sc[i][r] * sl : -INFINITY;
            mx = fmaxf(mx, x[4 * i + r]);
        }
    mx = group_max4(mx);
    const float m_new = fmaxf(st.m, mx);
    if (__any(m_new > st.m)) {
        const float alpha = fast_exp2(st.m - m_new);
        st.l *= alpha;
#pragma unroll
        for (int t = 0; t < NT; ++t) st.o[t] *= alpha;
        st.m = m_new;
    }
    uint32_t ph[2 * PP], pl[2 * PP];
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < 4 * PP; i += 2) {
        const float p0 = fast_exp2(x[i] - st.m);
        const float p1 = fast_exp2(x[i + 1] - st.m);
        psum += p0 + p1;
        const uint32_t u0 = __float_as_uint(p0), u1 = __float_as_uint(p1);
        const float r0 = p0 - __uint_as_float(u0 & 0xffff0000u);
        const float r1 = p1 - __uint_as_float(u1 & 0xffff0000u);
        ph[i / 2] = pack_hi16(u0, u1);
        pl[i / 2] = pack_hi16(__float_as_uint(r0), __float_as_uint(r1));
    }
    st.l += psum;
#pragma unroll
    for (int j = 0; j < PP / 2; ++j) {
        const bf16x8 bph = __builtin_bit_cast(bf16x8, u32x4{ph[4 * j], ph[4 * j + 1], ph[4 * j + 2], ph[4 * j + 3]});
        const bf16x8 bpl = __builtin_bit_cast(bf16x8, u32x4{pl[4 * j], pl[4 * j + 1], pl[4 * j + 2], pl[4 * j + 3]});
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const u32x2 a0 = v_quad<D, FP8>(pv[2 * j], t, nv[2 * j], qg);
            const u32x2 a1 = v_quad<D, FP8>(pv[2 * j + 1], t, nv[2 * j + 1], qg);
            const bf16x8 av = __builtin_bit_cast(bf16x8, u32x4{a0.x, a0.y, a1.x, a1.y});
            st.o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bph, st.o[t], 0, 0, 0);
            st.o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bpl, st.o[t], 0, 0, 0);
        }
    }
}

// ------------------------------------------------- fp8 pages on fp8 MFMA ---
// v_mfma_scale_f32_16x16x128_f8f6f4 multiplies e4m3 operands directly; each
// lane supplies 32 elements of its 16-lane group's k-block and an E8M0 scale
// (2^(s-127)) for them.  K and V codes enter as loaded.  Q and P are split
// into e4m3 hi + lo terms (residual scaled by 16), about 2^-8 relative, and
// the power-of-two factors of the split ride in the scale operands.
constexpr int kE8M0One = 127;

__device__ __forceinline__ f32x4 mfma_f8(const i32x8& a, const i32x8& b, f32x4 c, int scale_b) {
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, kE8M0One, 0, scale_b);
}

// Codes of two floats into the low (hi = false) or high half of w.
__device__ __forceinline__ uint32_t f32x2_to_fp8(float a, float b, uint32_t w, bool hi) {
    return hi ? (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)w, true)
              : (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)w, false);
}
__device__ __forceinline__ f32x2 fp8x2_to_f32(uint32_t w, bool hi) {
    return hi ? __builtin_amdgcn_cvt_pk_f32_fp8(w, true) : __builtin_amdgcn_cvt_pk_f32_fp8(w, false);
}

// Split four values v (already scaled into the e4m3 range) into hi and lo
// code words: hi = e4m3(v), lo = e4m3(16 (v - hi)).
__device__ __forceinline__ void split4(const float (&v)[4], uint32_t& hi, uint32_t& lo) {
    hi = f32x2_to_fp8(v[0], v[1], 0u, false);
    hi = f32x2_to_fp8(v[2], v[3], hi, true);
    const f32x2 h01 = fp8x2_to_f32(hi, false), h23 = fp8x2_to_f32(hi, true);
    lo = f32x2_to_fp8(16.f * (v[0] - h01.x), 16.f * (v[1] - h01.y), 0u, false);
    lo = f32x2_to_fp8(16.f * (v[2] - h23.x), 16.f * (v[3] - h23.y), lo, true);
}

// Query rows of a (request, head) group as fp8 B operands of the QK product.
// Lane (qg, n) holds head n's dims of chunks qg and qg+4 (the K operand's
// order), scaled by 2^k with k chosen per head so the row's largest
// magnitude lands in [128, 256); 2^-k and 2^-(k+4) go into the E8M0 scales.
struct Q8 {
    i32x8 hi, lo;
    int s_hi, s_lo;
};

template <int D>
__device__ __forceinline__ void q_to_fp8(const bf16x8 (&bq)[D / 32], Q8& q8) {
    constexpr int NV = D / 4;          // values this lane holds: 32 (D = 128) or 16 (D = 64)
    float v[NV];
#pragma unroll
    for (int j = 0; j < D / 32; ++j) {
        const u32x4 w = __builtin_bit_cast(u32x4, bq[j]);
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[8 * j + 2 * i] = __uint_as_float(ws[i] << 16);
            v[8 * j + 2 * i + 1] = __uint_as_float(ws[i] & 0xffff0000u);
        }
    }
    float amax = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) amax = fmaxf(amax, fabsf(v[i]));
    amax = group_max4(amax);
    // 2^e <= amax < 2^(e+1); scale by 2^(7-e); keep the E8M0 exponents in range
    int e = amax > 0.f ? (int)((__float_as_uint(amax) >> 23) & 0xffu) - 127 : 0;
    int k = 7 - e;
    k = max(-120, min(k, 120));
    const float sq = __uint_as_float((uint32_t)(k + 127) << 23);
    uint32_t hw[8], lw[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        hw[i] = 0u;
        lw[i] = 0u;
    }
#pragma unroll
    for (int i = 0; i < NV / 4; ++i) {
        const float t[4] = {v[4 * i] * sq, v[4 * i + 1] * sq, v[4 * i + 2] * sq, v[4 * i + 3] * sq};
        split4(t, hw[i], lw[i]);
    }
    q8.hi = i32x8{(int)hw[0], (int)hw[1], (int)hw[2], (int)hw[3], (int)hw[4], (int)hw[5], (int)hw[6], (int)hw[7]};
    q8.lo = i32x8{(int)lw[0], (int)lw[1], (int)lw[2], (int)lw[3], (int)lw[4], (int)lw[5], (int)lw[6], (int)lw[7]};
    q8.s_hi = kE8M0One - k;
    q8.s_lo = kE8M0One - k - 4;
}

// 4x4 transpose of dwords over the four 16-lane groups: afterwards register j
// of lane group g holds what register g of lane group j held.  A 32-lane swap
// exchanges the off-diagonal 2x2 blocks, a 16-lane swap transposes within them.
__device__ __forceinline__ void transpose4(int (&r)[8]) {
    auto a = __builtin_amdgcn_permlane32_swap((unsigned)r[0], (unsigned)r[2], false, false);
    auto b = __builtin_amdgcn_permlane32_swap((unsigned)r[1], (unsigned)r[3], false, false);
    auto c = __builtin_amdgcn_permlane16_swap(a[0], b[0], false, false);
    auto d = __builtin_amdgcn_permlane16_swap(a[1], b[1], false, false);
    r[0] = (int)c[0];
    r[1] = (int)c[1];
    r[2] = (int)d[0];
    r[3] = (int)d[1];
}

// One step of PP fp8 pages: scores on fp8 MFMA, online softmax, then
// O += V^T P^T with the step's 4*PP tokens per lane group (zero-padded to the
// instruction's 32-element blocks).  Unless the step is `full` (PP pages of
// 16 tokens, the common case), scores of slots >= nv are masked and the V
// codes of those slots are zeroed in place (vx is a ring slot that is
// reloaded before its next use).
template <int D, int PP>
__device__ __forceinline__ void fp8_step(AttnState<D>& st, const PageK<D, true> (&kx)[PP],
                                         PageV<D, true> (&vx)[PP], const Q8& q8, float sl,
                                         const int (&nv)[PP], int qg, bool full) {
    constexpr int NT = D / 16;
    float x[4 * PP];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < PP; ++i) {
        // pages past the step's end were loaded from a valid page; their
        // scores are masked below, so the products run unconditionally
        i32x8 ka;
        if constexpr (D == 128)
            ka = i32x8{(int)kx[i].k[0].x, (int)kx[i].k[0].y, (int)kx[i].k[0].z, (int)kx[i].k[0].w,
                       (int)kx[i].k[1].x, (int)kx[i].k[1].y, (int)kx[i].k[1].z, (int)kx[i].k[1].w};
        else  // upper half meets the zero half of the query operand; a copy of
              // the lower half keeps the register file free of a wide memory view
            ka = i32x8{(int)kx[i].k[0].x, (int)kx[i].k[0].y, (int)kx[i].k[0].z, (int)kx[i].k[0].w,
                       (int)kx[i].k[0].x, (int)kx[i].k[0].y, (int)kx[i].k[0].z, (int)kx[i].k[0].w};
        f32x4 s4 = {0.f, 0.f, 0.f, 0.f};
        s4 = mfma_f8(ka, q8.hi, s4, q8.s_hi);
        s4 = mfma_f8(ka, q8.lo, s4, q8.s_lo);
#pragma unroll
        for (int r = 0; r < 4; ++r) x[4 * i + r] = s4[r] * sl;
    }
    if (!full) {
#pragma unroll
        for (int i = 0; i < PP; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) x[4 * i + r] = (4 * qg + r < nv[i]) ? x[4 * i + r] : -INFINITY;
    }
#pragma unroll
    for (int i = 0; i < 4 * PP; ++i) mx = fmaxf(mx, x[i]);
    mx = group_max4(mx);
    const float m_new = fmaxf(st.m, mx);
    if (__any(m_new > st.m)) {
        const float alpha = fast_exp2(st.m - m_new);
        st.l *= alpha;
#pragma unroll
        for (int t = 0; t < NT; ++t) st.o[t] *= alpha;
        st.m = m_new;
    }
    // P in [0, 1] scaled by 2^8: hi carries 2^-8, lo 2^-12 in the scale operand
    int ph[8], pl[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        ph[i] = 0;
        pl[i] = 0;
    }
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < PP; ++i) {
        float p[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            p[r] = fast_exp2(x[4 * i + r] - st.m);
            psum += p[r];
            p[r] *= 256.f;
        }
        uint32_t h, l;
        split4(p, h, l);
        ph[i] = (int)h;
        pl[i] = (int)l;
    }
    st.l += psum;
    if constexpr (PP == 4) {
        // Lane group qg holds dword i = slots 4qg..4qg+3 of page i; V rows are
        // held by page (lane group qg: page qg, dword j = slots 4j..4j+3), so P
        // is transposed over the four lane groups: two 32-lane and two 16-lane
        // swaps per operand.
        transpose4(ph);
        transpose4(pl);
        const i32x8 bph = {ph[0], ph[1], ph[2], ph[3], 0, 0, 0, 0};
        const i32x8 bpl = {pl[0], pl[1], pl[2], pl[3], 0, 0, 0, 0};
        // codes of slots >= nv are zeroed (a tail slot may hold any byte)
        if (!full) {
            const int nvl = qg == 0 ? nv[0] : qg == 1 ? nv[1] : qg == 2 ? nv[2] : nv[3];
            uint32_t mk[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int k = nvl - 4 * j;
                mk[j] = k >= 4 ? 0xffffffffu : (k <= 0 ? 0u : (1u << (8 * k)) - 1u);
            }
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int j = 0; j < 4; ++j) vx[j].v[t] &= mk[j];
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const i32x8 av = {(int)vx[0].v[t], (int)vx[1].v[t], (int)vx[2].v[t], (int)vx[3].v[t], 0, 0, 0, 0};
            st.o[t] = mfma_f8(av, bph, st.o[t], kE8M0One - 8);
            st.o[t] = mfma_f8(av, bpl, st.o[t], kE8M0One - 12);
        }
        return;
    }
    const i32x8 bph = {ph[0], ph[1], ph[2], ph[3], ph[4], ph[5], ph[6], ph[7]};
    const i32x8 bpl = {pl[0], pl[1], pl[2], pl[3], pl[4], pl[5], pl[6], pl[7]};
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        int va[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) va[i] = 0;
#pragma unroll
        for (int i = 0; i < PP; ++i) {
            uint32_t w = vx[i].v[t];
            if (!full) {
                const int k = nv[i] - 4 * qg;  // live codes among this lane's four
                w &= k >= 4 ? 0xffffffffu : (k <= 0 ? 0u : (1u << (8 * k)) - 1u);
            }
            va[i] = (int)w;
        }
        const i32x8 av = {va[0], va[1], va[2], va[3], va[4], va[5], va[6], va[7]};
        st.o[t] = mfma_f8(av, bph, st.o[t], kE8M0One - 8);
        st.o[t] = mfma_f8(av, bpl, st.o[t], kE8M0One - 12);
    }
}

// ----------------------------------------------------------------- merge ---
// Online merge of partial pieces (m_i, l_i, o_i) of one (request, head):
//   M = max_i m_i,  l = sum_i 2^(m_i - M) l_i,  out = sum_i 2^(m_i - M) o_i / l
// Lane (qg, n) holds head n at dims 16 t + 4 qg .. + 3.  Pieces come in
// batches whose loads are all issued before any is used; a piece marked dead
// gets weight 0.
template <int D>
struct MergeAcc {
    static constexpr int NT = D / 16;
    float M = -INFINITY, l = 0.f;
    f32x4 acc[NT];
    __device__ __forceinline__ MergeAcc() {
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    template <int K>
    __device__ __forceinline__ void fold(float2 (&ml)[K], const f32x4 (&o)[K][NT], const bool (&live)[K]) {
        float Mb = M;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            if (!live[j]) ml[j] = make_float2(-INFINITY, 0.f);
            Mb = fmaxf(Mb, ml[j].x);
        }
        if (Mb > M) {             // exact: otherwise the factor is 1
            const float r = fast_exp2(M - Mb);
            l *= r;
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[t] *= r;
            M = Mb;
        }
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const bool ok = ml[j].x != -INFINITY;
            const float wt = ok ? fast_exp2(ml[j].x - M) : 0.f;
            l += ok ? wt * ml[j].y : 0.f;
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[t] += ok ? wt * o[j][t] : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    }
    // the pieces of waves wf .. wl: wave wf's is its kind-1 slot (the request
    // starts inside its range), every later wave's its kind-0 slot; waves
    // with no units left none.  Two pieces per round trip, in wave order;
    // the first batch may already be in `ml0`, `o0` (loaded with the record).
    static __device__ __forceinline__ int64_t slot_of(const AttnArgs& a, int v, int wf, int nh) {
        return (int64_t)(2 * v + (v == wf ? 1 : 0)) * a.G + nh;
    }
    static __device__ __forceinline__ void load2(const AttnArgs& a, int v0, int wf, int wl, int nh, int qg,
                                                 float2 (&ml)[2], f32x4 (&o)[2][NT]) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int v = min(v0 + j, wl);          // past wl: a re-read of wl's piece, dead below
            const int64_t slot = slot_of(a, v, wf, nh);
            ml[j] = a.part_ml[slot];
#pragma unroll
            for (int t = 0; t < NT; ++t) o[j][t] = *(const f32x4*)(a.part_o + slot * D + 16 * t + 4 * qg);
        }
    }
    __device__ __forceinline__ void fold_waves(const AttnArgs& a, int wf, int wl, int P, int skew, int nh, int qg,
                                               float2 (&ml0)[2], f32x4 (&o0)[2][NT]) {
        const int W = a.waves;
        // every wave holds units when the lightest weight's share of P is
        // above one unit: (256 - k) P > C(W), C(W) <= (256 + k) W
        const bool all_units = (int64_t)(256 - skew) * P > (int64_t)(256 + skew) * W;
        auto has_units = [&](int v) {
            return v <= wl && (all_units || share_bound(v, P, W, skew) < share_bound(v + 1, P, W, skew));
        };
        {
            const bool live[2] = {has_units(wf), has_units(wf + 1)};
            fold<2>(ml0, o0, live);
        }
        for (int v0 = wf + 2; v0 <= wl; v0 += 2) {
            float2 ml[2];
            f32x4 o[2][NT];
            load2(a, v0, wf, wl, nh, qg, ml, o);
            const bool live[2] = {has_units(v0), has_units(v0 + 1)};
            fold<2>(ml, o, live);
        }
    }
    // out[b, g G + n, dims of this lane] = acc / l, rounded to bf16
    __device__ __forceinline__ void store(const AttnArgs& a, int b, int h, int qg) const {
        const float inv = 1.f / l;
        uint16_t* orow = a.out + (int64_t)b * a.o_sb + (int64_t)h * a.o_sh;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            u32x2 pk;
            pk.x = (uint32_t)f32_to_bf16_rne(acc[t][0] * inv) | ((uint32_t)f32_to_bf16_rne(acc[t][1] * inv) << 16);
            pk.y = (uint32_t)f32_to_bf16_rne(acc[t][2] * inv) | ((uint32_t)f32_to_bf16_rne(acc[t][3] * inv) << 16);
            *(u32x2*)(orow + 16 * t + 4 * qg) = pk;
        }
    }
};

// Mark loaded registers as read.  A step reads some of its loads only on some
// paths (the query only at a segment change, the second page only when the
// step has one); a register whose load was never waited for on the path taken
// counts as still in flight when a later step reuses it, and the vector-memory
// counter is in order, so that later wait would drain every load issued
// before it.  Reading the whole slot once, after the next slot's loads are
// out, settles all of them together.
__device__ __forceinline__ void consume(const u32x4& x) { asm volatile("" ::"v"(x)); }
__device__ __forceinline__ void consume(const u32x2& x) { asm volatile("" ::"v"(x)); }
__device__ __forceinline__ void consume(uint32_t x) { asm volatile("" ::"v"(x)); }
__device__ __forceinline__ void consume(float x) { asm volatile("" ::"v"(x)); }
__device__ __forceinline__ void consume(const bf16x8& x) { consume(__builtin_bit_cast(u32x4, x)); }
template <typename T, int N>
__device__ __forceinline__ void consume(const T (&x)[N]) {
#pragma unroll
    for (int i = 0; i < N; ++i) consume(x[i]);
}
template <int D, bool FP8>
__device__ __forceinline__ void consume(const PageK<D, FP8>& r) { consume(r.k); }
template <int D, bool FP8>
__device__ __forceinline__ void consume(const PageV<D, FP8>& r) { consume(r.v); }

// The length the attention reads for request b's stored length L (b < B):
// clamped to the table, plus the new token in a decode step whose append
// fits the table (a position outside the pool is flagged where it is read).
template <bool STEP>
__device__ __forceinline__ int attn_len(const AttnArgs& a, int L) {
    const int maxL = a.max_pages * kPage;
    if (STEP && L >= 0 && L < maxL) return L + 1;
    return min(max(L, 0), maxL);
}

// Decode step: request b's new K and V rows of KV head g, to be written at
// position L (the stored length) by the whole wave, as kv_append_kernel
// does: K as 16-byte chunks (lanes 0 .. D/X - 1), V as D / 64 consecutive
// dims a lane; fp8 pools take codes as they are or bf16 rows quantised with
// the (request, head)'s scales.  row_load issues every read (block-table
// entry, rows, scales) at once; row_store writes them, skipping a position
// outside the pool (the merge pass flags it).
struct NewRow {
    int pg, slot, g;
    u32x4 w, h;      // K chunk (and its second half when quantising)
    uint32_t vv;     // this lane's V dims
    float ks, vs;    // quantising scales
};

template <int D, bool FP8>
__device__ __forceinline__ NewRow row_load(const AttnArgs& a, int b, int g, int L, int lane) {
    constexpr int EB = FP8 ? 1 : 2;
    constexpr int X = 16 / EB;                   // pool elements per K chunk
    constexpr int VD = D / 64;                   // V dims a lane
    NewRow r;
    r.pg = a.block_table[(int64_t)b * a.bt_stride + (L >> 4)];
    r.slot = L & (kPage - 1);
    r.g = g;
    const bool quant = FP8 && a.quant;
    const int SB = quant ? 2 : EB;               // source element bytes
    const char* kn = (const char*)a.k_new + ((int64_t)b * a.new_sb + (int64_t)g * a.new_sh) * SB;
    const char* vn = (const char*)a.v_new + ((int64_t)b * a.vnew_sb + (int64_t)g * a.vnew_sh) * SB;
    r.w = u32x4{0u, 0u, 0u, 0u};
    r.h = u32x4{0u, 0u, 0u, 0u};
    if (lane < D / X) {
        r.w = *(const u32x4*)(kn + (int64_t)lane * X * SB);
        if (quant) r.h = *(const u32x4*)(kn + (int64_t)lane * X * SB + 16);
    }
    if (quant || EB == 2) r.vv = VD == 2 ? *(const uint32_t*)(vn + (int64_t)lane * 4) : *(const uint16_t*)(vn + (int64_t)lane * 2);
    else r.vv = VD == 2 ? *(const uint16_t*)(vn + (int64_t)lane * 2) : *(const uint8_t*)(vn + lane);
    r.ks = quant ? a.k_scale[(int64_t)b * a.H_kv + g] : 0.f;
    r.vs = quant ? a.v_scale[(int64_t)b * a.H_kv + g] : 0.f;
    return r;
}

template <int D, bool FP8>
__device__ __forceinline__ void row_store(const AttnArgs& a, const NewRow& r, int lane) {
    constexpr int EB = FP8 ? 1 : 2;
    constexpr int X = 16 / EB;
    constexpr int VD = D / 64;
    if ((unsigned)r.pg >= (unsigned)a.num_pages) return;
    const bool quant = FP8 && a.quant;
    char* kp = (char*)a.k_pages + ((int64_t)r.pg * a.H_kv + r.g) * ((int64_t)D * kPage * EB);
    char* vp = (char*)a.v_pages + ((int64_t)r.pg * a.H_kv + r.g) * ((int64_t)D * kPage * EB);
    if (lane < D / X) {
        u32x4 w = r.w;
        if (quant) {   // 16 bf16 -> 16 e4m3fn codes with the K scale
            const uint32_t in[8] = {r.w.x, r.w.y, r.w.z, r.w.w, r.h.x, r.h.y, r.h.z, r.h.w};
            uint32_t ow[4];
#pragma unroll
            for (int k = 0; k < 4; ++k)
                ow[k] = quantize_e4m3fn(__uint_as_float(in[2 * k] << 16), r.ks) |
                        (quantize_e4m3fn(__uint_as_float(in[2 * k] & 0xffff0000u), r.ks) << 8) |
                        (quantize_e4m3fn(__uint_as_float(in[2 * k + 1] << 16), r.ks) << 16) |
                        (quantize_e4m3fn(__uint_as_float(in[2 * k + 1] & 0xffff0000u), r.ks) << 24);
            w = u32x4{ow[0], ow[1], ow[2], ow[3]};
        }
        *(u32x4*)(kp + ((int64_t)lane * kPage + r.slot) * 16) = w;
    }
#pragma unroll
    for (int i = 0; i < VD; ++i) {
        char* dst = vp + ((int64_t)(lane * VD + i) * kPage + r.slot) * EB;
        if (quant) {
            const uint32_t bits = (r.vv >> (16 * i)) & 0xffffu;
            *(uint8_t*)dst = (uint8_t)quantize_e4m3fn(__uint_as_float(bits << 16), r.vs);
        } else if (EB == 2) {
            *(uint16_t*)dst = (uint16_t)(r.vv >> (16 * i));
        } else {
            *(uint8_t*)dst = (uint8_t)(r.vv >> (8 * i));
        }
    }
}

// A position in a wave's stream: step x, the `len` consecutive pages from
// page p of request b, KV head g.  Wave-uniform.
struct Cursor {
    int b, g, p;   // request, KV head, first page of the step within the request
    int np, L;     // the request's pages and clamped length
    int x;         // flattened unit (step) index
    int len;       // pages in the step (1..PP; never crosses a request)
    bool live;     // false once past the wave's range
};

template <int PP>
__device__ __forceinline__ void cursor_len(Cursor& c) {
    c.len = min(PP, c.np - c.p);
}

// Step to the next unit.  A cursor that would leave the range keeps its last
// position (so loads issued for it stay in bounds) and stops being live.
template <int PP, bool STEP>
__device__ __forceinline__ void cursor_next(Cursor& c, const AttnArgs& a, int r1) {
    if (!c.live) return;
    if (c.x + 1 >= r1) {
        c.live = false;
        return;
    }
    c.x += 1;
    c.p += PP;
    if (c.p >= c.np) {
        c.p = 0;
        if (++c.g >= a.H_kv) {
            c.g = 0;
            // units remain, so a later request with pages exists
            do {
                ++c.b;
                c.L = attn_len<STEP>(a, a.seq_lens[c.b]);
                c.np = (c.L + kPage - 1) / kPage;
            } while (c.np == 0 && c.b + 1 < a.B);
        }
    }
    cursor_len<PP>(c);
}

// The hardware registers a traced wave records (s_getreg_b32 operands:
// register id, bit offset 0, field width): the XCD it runs on, and its
// wave / SIMD / CU / shader-engine ids.
constexpr int kHwRegXccId = 20 | (3 << 11);    // XCC_ID, bits 3:0
constexpr int kHwRegHwId = 4 | (31 << 11);     // HW_ID, bits 31:0

// DEPTH steps of PP pages are in flight per wave while it computes one.  With
// DEPTH = 1 two waves share each SIMD; with DEPTH = 2 each SIMD runs one wave
// (its issue is not arbitrated against a second, older wave, which otherwise
// runs ahead and leaves the younger one to finish alone).
//
// TRACE: each wave also records, in a.wave_times[3w .. 3w + 2], the
// real-time clock (100 MHz) when it starts and when it has written its last
// result, and (XCD id << 32) | HW_ID: a timing record, not a change of the
// computation.
template <int D, bool FP8, int PP, int DEPTH, bool TRACE, bool STEP>
__global__ void __launch_bounds__(kAttnBlock) __attribute__((amdgpu_waves_per_eu(DEPTH == 1 ? 2 : 1, DEPTH == 1 ? 2 : 1)))
attn_mfma_kernel(AttnArgs a) {
    constexpr int NT = D / 16;
    constexpr int KS = D / 32;
    constexpr int EB = FP8 ? 1 : 2;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int qg = lane >> 4;
    const int n = lane & 15;
    // wave index, made provably uniform so that all stream bookkeeping is scalar
    const int w = __builtin_amdgcn_readfirstlane(blockIdx.x * (kAttnBlock / kWaveSize) + (threadIdx.x >> 6));
    if (w >= a.waves) return;
    uint64_t t_start = 0;
    if constexpr (TRACE) t_start = __builtin_amdgcn_s_memrealtime();
    auto trace_end = [&]() {
        if constexpr (TRACE) {
            const uint64_t t_end = __builtin_amdgcn_s_memrealtime();
            const uint64_t ids = ((uint64_t)(__builtin_amdgcn_s_getreg(kHwRegXccId) & 15) << 32) |
                                 (uint32_t)__builtin_amdgcn_s_getreg(kHwRegHwId);
            if (lane == 0) {
                a.wave_times[3 * (int64_t)w] = (int64_t)t_start;
                a.wave_times[3 * (int64_t)w + 1] = (int64_t)t_end;
                a.wave_times[3 * (int64_t)w + 2] = (int64_t)ids;
            }
        }
    };

    // This wave's range of the P units (see the work split above).  Lane l
    // holds requests b0 + 16 l .. b0 + 16 l + 15 of each batch of lengths, so
    // one scan over the lanes gives every lane's first unit.
    const int maxL = a.max_pages * kPage;
    int Lk[kPlanPerLane], uk[kPlanPerLane];
    bool bad_len = false;
    auto load_lens = [&](int b0) -> int {   // this lane's units in the batch
        int sum = 0;
#pragma unroll
        for (int k = 0; k < kPlanPerLane; ++k) {
            const int b = b0 + kPlanPerLane * lane + k;
            // slots past the batch hold no request: length 0, no units
            const int Ls = b < a.B ? a.seq_lens[b] : 0;
            if (Ls < 0 || Ls > maxL) bad_len = true;
            const int L = b < a.B ? attn_len<STEP>(a, Ls) : 0;
            Lk[k] = L;
            uk[k] = ((L + kPage - 1) / kPage + PP - 1) / PP * a.H_kv;
            sum += uk[k];
        }
        return sum;
    };
    // Requests of length 0 attend nothing and get rows of zeros: request b's
    // rows are written by wave b mod W, all lanes together.
    auto zero_empty = [&](int b0) {
#pragma unroll
        for (int k = 0; k < kPlanPerLane; ++k) {
            const int b = b0 + kPlanPerLane * lane + k;
            uint64_t m = __ballot(b < a.B && Lk[k] == 0 && b % a.waves == w);
            while (m) {
                const int src = __ffsll((unsigned long long)m) - 1;
                m &= m - 1;
                const int bz = b0 + kPlanPerLane * src + k;
                // each head row is D bf16 = D / 4 8-byte units (rows are 8-byte aligned)
                for (int u = lane; u < a.H_q * (D / 4); u += kWaveSize) {
                    const int h = u / (D / 4), c = u - h * (D / 4);
                    *(u32x2*)(a.out + (int64_t)bz * a.o_sb + (int64_t)h * a.o_sh + 4 * c) = u32x2{0u, 0u};
                }
            }
        }
    };
    int lsum = load_lens(0);
    zero_empty(0);
    int incl = wave_incl_scan(lsum, lane);
    int P = __builtin_amdgcn_readlane(incl, kWaveSize - 1);
    for (int b0 = kPlanBatch; b0 < a.B; b0 += kPlanBatch) {
        P += __builtin_amdgcn_readfirstlane(wave_sum(load_lens(b0)));
        zero_empty(b0);
    }
    const int skew = share_skew(a.skew, P, a.waves, PP);
    const int r0 = share_bound(w, P, a.waves, skew);
    const int r1 = share_bound(w + 1, P, a.waves, skew);
    // wave 0 raises the length flag
    if (w == 0 && __any(bad_len) && lane == 0) atomicOr(a.err, kErrLength);
    if (r0 >= r1) {
        if (lane == 0) a.cuts[w] = make_int4(-1, 0, 0, 0);
        trace_end();
        return;
    }
    int sb = -1, sg = 0, sp = 0, sL = 0;   // request, KV head, page, length at unit r0
    int carry = 0;                         // units of the requests before this batch
    for (int b0 = 0; b0 < a.B; b0 += kPlanBatch) {
        if (b0 > 0) {
            lsum = load_lens(b0);
            incl = wave_incl_scan(lsum, lane);
        } else if (a.B > kPlanBatch) {
            lsum = load_lens(0);
            incl = wave_incl_scan(lsum, lane);
        }
        const int excl = carry + incl - lsum;
        const uint64_t hit = __ballot(lsum > 0 && excl <= r0 && r0 < excl + lsum);
        if (sb < 0 && hit != 0) {
            // walk the 16 requests of the lane that holds unit r0
            const int src = __ffsll((unsigned long long)hit) - 1;
            int x = __builtin_amdgcn_readlane(excl, src);
#pragma unroll
            for (int k = 0; k < kPlanPerLane; ++k) {
                const int u = __builtin_amdgcn_readlane(uk[k], src);
                if (sb < 0 && r0 < x + u) {
                    const int ns = u / a.H_kv;
                    const int off = r0 - x;
                    sb = b0 + kPlanPerLane * src + k;
                    sL = __builtin_amdgcn_readlane(Lk[k], src);
                    sg = off / ns;
                    sp = off % ns * PP;
                }
                x += u;
            }
        }
        carry += __builtin_amdgcn_readlane(incl, kWaveSize - 1);
        if (sb >= 0) break;
    }

    const size_t tile_bytes = (size_t)D * kPage * EB;
    const size_t page_stride = (size_t)a.H_kv * tile_bytes;
    const bool hv = n < a.G;

    // DEPTH + 2 cursors walk the wave's stream: cur[0] is computed,
    // cur[1..DEPTH] have their pages (and query rows) in flight, and
    // cur[DEPTH+1] has its block-table entries in flight.
    sb = __builtin_amdgcn_readfirstlane(sb);
    sg = __builtin_amdgcn_readfirstlane(sg);
    sp = __builtin_amdgcn_readfirstlane(sp);
    sL = __builtin_amdgcn_readfirstlane(sL);

    // Decode step: this wave writes the new row of every (request, head)
    // whose last unit (the one holding the new position) lies in its range,
    // before it issues any page load, walking segment by segment from the
    // range's start.  A segment that ends inside the range is followed by
    // another unit of the range, so the walk stays inside the batch.  The
    // stored length is the attention length less one below the table's end;
    // only a full-width attention length needs the stored one read back.
    if constexpr (STEP) {
        int b = sb, g = sg, L = sL, x0 = r0 - sp / PP;   // segment (b, g), its first unit x0
        for (;;) {
            const int last = x0 + ((L + kPage - 1) / kPage + PP - 1) / PP - 1;
            if (last >= r1) break;                        // runs past the range: another wave's
            const int Ls = L < maxL ? L - 1 : a.seq_lens[b];
            if (Ls >= 0 && Ls < maxL) row_store<D, FP8>(a, row_load<D, FP8>(a, b, g, Ls, lane), lane);
            x0 = last + 1;
            if (x0 >= r1) break;
            if (++g == a.H_kv) {
                g = 0;
                do {                                      // the next request with units
                    ++b;
                    L = attn_len<STEP>(a, a.seq_lens[b]);
                } while (L == 0 && b + 1 < a.B);
                if (L == 0) break;
            }
        }
        // the rows are in memory before this wave reads any page
        __builtin_amdgcn_s_waitcnt(0);
    }

    Cursor cur[DEPTH + 2];
    {
        cur[0].b = sb;
        cur[0].g = sg;
        cur[0].p = sp;
        cur[0].L = sL;
        cur[0].np = (cur[0].L + kPage - 1) / kPage;
        cur[0].x = r0;
        cur[0].live = true;
        cursor_len<PP>(cur[0]);
    }
#pragma unroll
    for (int j = 1; j < DEPTH + 2; ++j) {
        cur[j] = cur[j - 1];
        cursor_next<PP, STEP>(cur[j], a, r1);
    }

    // Block-table entries of a step: lane i < PP reads page p + i, clamped to
    // the step's last page (for one-page steps lane 1 reads an in-row
    // neighbour, unused).  The lane-dependent address keeps this a vector
    // load, ordered with the page loads, instead of a scalar one.
    auto bt_load = [&](const Cursor& c) -> int {
        // page i of the step sits in lane i, or in lane group i when fp8 V
        // rows are read by page (each lane then addresses its own page)
        constexpr bool kRows = FP8 && PP == 4;
        const int i = kRows ? (lane >> 4) : PP == 1 ? (lane & 1) : (lane & (PP - 1));
        const int idx = min(c.p + i, (PP == 1 ? c.np : c.p + c.len) - 1);
        return a.block_table[(int64_t)c.b * a.bt_stride + idx];
    };
    // Query rows of a unit's group as the QK B operand: lane (qg, n) holds
    // head g*G + n.  Lanes n >= G hold a copy of the group's last head; their
    // columns of S and O are computed and discarded, which keeps this load
    // free of lane masks.
    auto q_load = [&](const Cursor& c, bf16x8 (&bq)[KS]) {
        const uint16_t* qrow = a.q + (int64_t)c.b * a.q_sb + (int64_t)(c.g * a.G + min(n, a.G - 1)) * a.q_sh;
#pragma unroll
        for (int j = 0; j < KS; ++j) {
            const int dim0 = FP8 ? 16 * (qg + 4 * (j >> 1)) + 8 * (j & 1) : 8 * (4 * j + qg);
            bq[j] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qrow + dim0));
        }
    };
    // fp8 only: lanes 0..31 read the K scale, lanes 32..63 the V scale.
    auto scale_load = [&](const Cursor& c) -> float {
        const float* src = lane < 32 ? a.k_scale : a.v_scale;
        return src[(int64_t)c.b * a.H_kv + c.g];
    };
    int bad_pages = 0;  // wave-uniform: set when a block-table entry is outside the pool
    // K and V of a step's pages.  An entry outside the pool is never
    // dereferenced: page 0 is read instead and the piece's output is poisoned.
    // A one-page step of a two-page stream re-reads its page (a cache hit).
    auto kv_load = [&](const Cursor& c, int btv, PageK<D, FP8> (&rk)[PP], PageV<D, FP8> (&rv)[PP], bool& bad) {
        bad = false;
        constexpr bool kRows = FP8 && PP == 4;
#pragma unroll
        for (int i = 0; i < PP; ++i) {
            int pg = __builtin_amdgcn_readlane(btv, kRows ? 16 * i : i);
            if ((unsigned)pg >= (unsigned)a.num_pages) {
                pg = 0;
                bad = true;
                bad_pages = 1;
            }
            const size_t off = (size_t)pg * page_stride + (size_t)c.g * tile_bytes;
            load_k<D, FP8>(rk[i], (const char*)a.k_pages + off, qg, n);
            if constexpr (!kRows) load_v<D, FP8>(rv[i], (const char*)a.v_pages + off, qg, n);
        }
        if constexpr (kRows) {
            // this lane's page (lane group qg), invalid entries read page 0 as above
            const int pl = (unsigned)btv < (unsigned)a.num_pages ? btv : 0;
            load_v_rows<D>(rv, (const char*)a.v_pages + (size_t)pl * page_stride + (size_t)c.g * tile_bytes, n);
        }
    };

    AttnState<D> st;
    auto reset = [&]() {
#pragma unroll
        for (int t = 0; t < NT; ++t) st.o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        st.m = -INFINITY;
        st.l = 0.f;
    };
    reset();
    bool seg_bad = false;

    // Write the finished piece of C's (request, head): the whole output if the
    // request's head lies entirely in this wave's range, else a partial in
    // the wave's slot of its kind.  A range cuts at most two: the (request,
    // head) it starts in, if that began before it (kind 0), and the one it
    // ends in, if that began inside it and runs past its end (kind 1).
    auto finish = [&](const Cursor& c, float vs) {
        const float l_tot = group_sum4(st.l);
        const int seg_x0 = c.x - c.p / PP;
        const bool whole = seg_x0 >= r0 && seg_x0 + (c.np + PP - 1) / PP <= r1;
        const int kind = seg_x0 < r0 ? 0 : 1;
        if (hv) {
            const int h = c.g * a.G + n;
            if (whole) {
                const float f = seg_bad ? NAN : vs / l_tot;
                uint16_t* orow = a.out + (int64_t)c.b * a.o_sb + (int64_t)h * a.o_sh;
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    u32x2 pk;
                    pk.x = (uint32_t)f32_to_bf16_rne(st.o[t][0] * f) | ((uint32_t)f32_to_bf16_rne(st.o[t][1] * f) << 16);
                    pk.y = (uint32_t)f32_to_bf16_rne(st.o[t][2] * f) | ((uint32_t)f32_to_bf16_rne(st.o[t][3] * f) << 16);
                    *(u32x2*)(orow + 16 * t + 4 * qg) = pk;
                }
            } else {
                const int64_t slot = (int64_t)(2 * w + kind) * a.G + n;
                float* po = a.part_o + slot * D;
                const float f = seg_bad ? NAN : vs;
#pragma unroll
                for (int t = 0; t < NT; ++t) *(f32x4*)(po + 16 * t + 4 * qg) = st.o[t] * f;
                if (qg == 0) a.part_ml[slot] = make_float2(seg_bad ? NAN : st.m, l_tot);
            }
        }
        reset();
        seg_bad = false;
    };

    // Operands live in rings of DEPTH + 1 slots: pages, query rows, fp8
    // scales.  Each step issues cur[DEPTH+1]'s block-table entries and
    // cur[DEPTH]'s query rows and pages into the slot freed by the previous
    // step, then computes cur[0].  Every step issues the same loads, in the
    // same order, so each wait covers exactly the data it needs and DEPTH
    // steps stay in flight.
    PageK<D, FP8> kb[DEPTH + 1][PP];
    PageV<D, FP8> vb[DEPTH + 1][PP];
    bf16x8 qb[DEPTH + 1][KS];
    float scb[DEPTH + 1];
    bool badb[DEPTH + 1];
    // All block-table entries of the prologue go out before its pages: the
    // loop's first wait for btn then leaves as many loads in flight as every
    // later one (the counter is in order, and the wait is shared by all
    // iterations of the loop).
    int bts[DEPTH + 1];
#pragma unroll
    for (int j = 0; j <= DEPTH; ++j) bts[j] = bt_load(cur[j]);
#pragma unroll
    for (int j = 0; j < DEPTH; ++j) {
        q_load(cur[j], qb[j]);
        scb[j] = 0.f;
        if constexpr (FP8) scb[j] = scale_load(cur[j]);
        kv_load(cur[j], bts[j], kb[j], vb[j], badb[j]);
    }
    int btn = bts[DEPTH];
    Q8 q8;                 // fp8 only: query rows of (q8_b, q8_g) as fp8 operands
    int q8_b = -1, q8_g = -1;

    auto step = [&](auto slot) {
        constexpr int sc_ = decltype(slot)::value;                // slot computed now
        constexpr int ld_ = (sc_ + DEPTH) % (DEPTH + 1);          // slot loaded now
        const int btT = bt_load(cur[DEPTH + 1]);
        q_load(cur[DEPTH], qb[ld_]);
        if constexpr (FP8) scb[ld_] = scale_load(cur[DEPTH]);
        kv_load(cur[DEPTH], btn, kb[ld_], vb[ld_], badb[ld_]);
        btn = btT;
        if constexpr (FP8 && DEPTH > 1) consume(qb[sc_]);

        const Cursor& C = cur[0];
        float sl = a.scale_log2, vs = 1.f;
        if constexpr (FP8) {
            sl *= __int_as_float(__builtin_amdgcn_readlane(__float_as_int(scb[sc_]), 0));
            vs = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(scb[sc_]), 32));
        }
        seg_bad = seg_bad || badb[sc_];
        if constexpr (FP8) {
            if (C.b != q8_b || C.g != q8_g) {  // new (request, head): convert its query rows
                q_to_fp8<D>(qb[sc_], q8);
                q8_b = C.b;
                q8_g = C.g;
            }
            int nv[PP];
#pragma unroll
            for (int i = 0; i < PP; ++i) nv[i] = (i == 0 || C.len > i) ? min(kPage, C.L - (C.p + i) * kPage) : 0;
            fp8_step<D, PP>(st, kb[sc_], vb[sc_], q8, sl, nv, qg, C.len == PP && C.L >= (C.p + PP) * kPage);
        } else if constexpr (PP == 1) {
            const f32x4 s4 = page_scores<D, FP8>(kb[sc_][0], qb[sc_]);
            page_pv<D, FP8>(st, s4, vb[sc_][0], sl, min(kPage, C.L - C.p * kPage), qg);
        } else {
            f32x4 sc4[PP];
            int nv[PP];
#pragma unroll
            for (int i = 0; i < PP; ++i) {
                // pages past the step's end hold a valid page of the request
                // (the block-table read is clamped); all their slots are masked
                sc4[i] = page_scores<D, FP8>(kb[sc_][i], qb[sc_]);
                nv[i] = (i == 0 || C.len > i) ? min(kPage, C.L - (C.p + i) * kPage) : 0;
            }
            group_pv<D, FP8, PP>(st, sc4, vb[sc_], sl, nv, qg);
        }
        if (C.live && (C.p + C.len >= C.np || C.x + 1 >= r1)) finish(C, vs);
#pragma unroll
        for (int j = 0; j < DEPTH + 1; ++j) cur[j] = cur[j + 1];
        cursor_next<PP, STEP>(cur[DEPTH + 1], a, r1);
    };

    // One exit, after a whole round of DEPTH + 1 steps.  An exit between
    // steps would leave that step's prefetches in flight on an edge that the
    // compiler joins with the continuing edge ahead of the loop header, and
    // the header would then wait for every load in flight on each iteration.
    // The last round may run up to DEPTH steps past the range: their cursors
    // are dead (re-reading the last pages of the range, writing nothing).
    for (;;) {
        step(std::integral_constant<int, 0>{});
        step(std::integral_constant<int, 1>{});
        if constexpr (DEPTH >= 2) step(std::integral_constant<int, 2>{});
        if constexpr (DEPTH >= 3) step(std::integral_constant<int, 3>{});
        if (!cur[0].live) break;
        if constexpr (DEPTH == 1) {
            // Two workgroups share each CU at this depth (one wave of each per
            // SIMD), and the wave arbiter favours the older: it finished well
            // ahead and left the other alone on its CU (per-wave timing
            // records, 512-request fp8 batch).  A wave with more of its range
            // left now issues first.
            const int q = (int)((int64_t)(cur[0].x - r0) * 4 / (r1 - r0));
            if (q <= 0) __builtin_amdgcn_s_setprio(3);
            else if (q == 1) __builtin_amdgcn_s_setprio(2);
            else if (q == 2) __builtin_amdgcn_s_setprio(1);
            else __builtin_amdgcn_s_setprio(0);
        }
    }
    if (bad_pages) atomicOr(a.err, kErrPage);
    // The request this wave's range ends in, if it began inside the range and
    // runs past it (its kind-1 piece; the dead cursors stopped at the last
    // unit): the merge kernel's wave w combines it with the later waves'
    // pieces.
    const Cursor& e = cur[0];
    const int ex0 = e.x - e.p / PP;
    const int en = (e.np + PP - 1) / PP;
    if (lane == 0) {
        const bool cut = ex0 >= r0 && ex0 + en > r1;
        const int wl = cut ? wave_of(ex0 + en - 1, P, a.waves, skew) : 0;
        a.cuts[w] = cut ? make_int4(e.b, e.g, wl, P) : make_int4(-1, 0, 0, 0);
    }
    trace_end();
}

// One wave per attention wave w: if w's range ended inside a (request, head)
// that began in it, combine that request's pieces.
template <int D>
__global__ void __launch_bounds__(256) merge_kernel(AttnArgs a) {
    if (a.k_new != nullptr) {
        // decode step: advance the length of every request whose new row
        // fitted (as kv_append_kernel does); flag the others
        const int maxL = a.max_pages * kPage;
        for (int64_t b = (int64_t)blockIdx.x * 256 + threadIdx.x; b < a.B; b += (int64_t)gridDim.x * 256) {
            const int L = a.lens_rw[b];
            bool ok = L >= 0 && L < maxL;
            if (ok) {
                const int pg = a.block_table[b * a.bt_stride + (L >> 4)];
                ok = (unsigned)pg < (unsigned)a.num_pages;
            }
            if (ok) a.lens_rw[b] = L + 1;
            else atomicOr(a.err, kErrAppendSlot);
        }
    }
    const int w = __builtin_amdgcn_readfirstlane(blockIdx.x * (256 / kWaveSize) + (threadIdx.x >> 6));
    if (w >= a.waves) return;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int qg = lane >> 4, n = lane & 15, nh = min(n, a.G - 1);
    // the record and, in the same round trip, the first two pieces a cut
    // starting in wave w would have (slots 2w + 1 and 2w + 2; past the
    // workspace's last wave a re-read of 2w + 1)
    const int4 c = a.cuts[w];
    float2 ml0[2];
    f32x4 o0[2][D / 16];
    MergeAcc<D>::load2(a, w, w, min(w + 1, a.waves - 1), nh, qg, ml0, o0);
    if (c.x < 0) return;
    const int b = __builtin_amdgcn_readfirstlane(c.x), g = __builtin_amdgcn_readfirstlane(c.y);
    const int wl = __builtin_amdgcn_readfirstlane(c.z), P = __builtin_amdgcn_readfirstlane(c.w);
    MergeAcc<D> m;
    m.fold_waves(a, w, wl, P, share_skew(a.skew, P, a.waves, a.pp), nh, qg, ml0, o0);
    if (n < a.G) m.store(a, b, g * a.G + n, qg);
}

}  // namespace

// ------------------------------------------------------------- launchers ---

void launch_kv_append(const AppendArgs& a, hipStream_t s) {
    if (a.B == 0) return;
    hipLaunchKernelGGL(kv_append_kernel, dim3(a.B), dim3(512), 0, s, a);
}

// The shapes built with a traced twin: head_dim 128 at the library's default
// steps (bf16: one or two pages, depth 2; fp8: four pages, depth 1).
template <int D, bool FP8, int PP, int DEPTH>
constexpr bool kTraced = D == 128 && (FP8 ? (PP == 4 && DEPTH == 1) : (PP <= 2 && DEPTH == 2));

// The shapes built with a decode-step twin (the append fused in): the
// library's default steps, both head sizes.
template <bool FP8, int PP, int DEPTH>
constexpr bool kStepBuilt = FP8 ? (PP == 4 && DEPTH == 1) : (PP <= 2 && DEPTH == 2);

template <int D, bool FP8, int PP, int DEPTH>
struct Variant {
    static void launch(const AttnArgs& a, int grid, hipStream_t s) {
        if (a.k_new != nullptr) {   // the host launches the step only where it is built
            if constexpr (kStepBuilt<FP8, PP, DEPTH>)
                hipLaunchKernelGGL((attn_mfma_kernel<D, FP8, PP, DEPTH, false, true>), dim3(grid), dim3(kAttnBlock),
                                   0, s, a);
            return;
        }
        if constexpr (kTraced<D, FP8, PP, DEPTH>) {
            if (a.wave_times) {
                hipLaunchKernelGGL((attn_mfma_kernel<D, FP8, PP, DEPTH, true, false>), dim3(grid), dim3(kAttnBlock),
                                   0, s, a);
                return;
            }
        }
        hipLaunchKernelGGL((attn_mfma_kernel<D, FP8, PP, DEPTH, false, false>), dim3(grid), dim3(kAttnBlock), 0, s,
                           a);
    }
    static int occupancy() {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, attn_mfma_kernel<D, FP8, PP, DEPTH, false, false>,
                                                         kAttnBlock, 0) != hipSuccess ||
            nb < 1)
            nb = 1;
        return nb;
    }
};

// Dispatch on (head_dim, fp8, pages per step, depth): 1 or 2 pages for bf16
// pools, 1, 2 or 4 for fp8 pools; depth 1 or 2.
template <int D, bool FP8, int PP>
static int dispatch_depth(int depth, bool occ, const AttnArgs* a, int grid, hipStream_t s) {
    if (depth == 2) {
        if (occ) return Variant<D, FP8, PP, 2>::occupancy();
        Variant<D, FP8, PP, 2>::launch(*a, grid, s);
    } else {
        if (occ) return Variant<D, FP8, PP, 1>::occupancy();
        Variant<D, FP8, PP, 1>::launch(*a, grid, s);
    }
    return 0;
}

template <int D, bool FP8>
static int dispatch_pp(int pp, int depth, bool occ, const AttnArgs* a, int grid, hipStream_t s) {
    if constexpr (FP8) {
        if (pp == 4) return dispatch_depth<D, FP8, 4>(depth, occ, a, grid, s);
    }
    if (pp == 2) return dispatch_depth<D, FP8, 2>(depth, occ, a, grid, s);
    return dispatch_depth<D, FP8, 1>(depth, occ, a, grid, s);
}

static int dispatch(int D, bool fp8, int pp, int depth, bool occ, const AttnArgs* a, int grid, hipStream_t s) {
    if (D == 128) return fp8 ? dispatch_pp<128, true>(pp, depth, occ, a, grid, s)
                             : dispatch_pp<128, false>(pp, depth, occ, a, grid, s);
    return fp8 ? dispatch_pp<64, true>(pp, depth, occ, a, grid, s) : dispatch_pp<64, false>(pp, depth, occ, a, grid, s);
}

void launch_attention(const AttnArgs& a, int pages_per_step, int depth, bool fp8, int grid, hipStream_t s) {
    if (a.B == 0 || a.H_q == 0) return;
    dispatch(a.D, fp8, pages_per_step, depth, false, &a, grid, s);
}

bool attention_traced(int pages_per_step, int depth, bool fp8, int D) {
    if (D != 128) return false;
    return fp8 ? (pages_per_step == 4 && depth == 1) : (pages_per_step <= 2 && depth == 2);
}

bool attention_step_built(int pages_per_step, int depth, bool fp8) {
    return fp8 ? (pages_per_step == 4 && depth == 1) : (pages_per_step <= 2 && depth == 2);
}

int attention_blocks_per_cu(int pages_per_step, int depth, bool fp8, int D) {
    return dispatch(D, fp8, pages_per_step, depth, true, nullptr, 0, nullptr);
}

void launch_merge(const AttnArgs& a, hipStream_t s) {
    const dim3 g((a.waves + 3) / 4), blk(256);
    if (a.D == 128)
        hipLaunchKernelGGL(merge_kernel<128>, g, blk, 0, s, a);
    else
        hipLaunchKernelGGL(merge_kernel<64>, g, blk, 0, s, a);
}

}  // namespace bellman
