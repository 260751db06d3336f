// HIP kernels for gfx950: KV append, split planning, split-K partial decode
// attention on the matrix cores, and the log-sum-exp merge of the partials.
//
// The computation is one decode step of the serving loop that beLLMan
// (arXiv 2510.15330, Sec. 3) controls: every request attends its one new
// query token over its own KV cache (prompt plus tokens generated so far).
#include "internal.h"

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
// One workgroup per request: copy the new K row into its 16-byte chunks and
// the new V row into its slot column, then advance the request's length.
__global__ void __launch_bounds__(256) kv_append_kernel(AppendArgs a) {
    const int b = blockIdx.x;
    const int L = a.seq_lens[b];
    const int pi = L >> 4;
    bool ok = L >= 0 && pi < a.max_pages;
    int pg = ok ? a.block_table[(int64_t)b * a.bt_stride + pi] : -1;
    ok = ok && pg >= 0 && (int64_t)pg < a.num_pages;
    if (!ok) {
        if (threadIdx.x == 0) atomicOr(a.err, kErrAppendSlot);
        return;
    }
    const int slot = L & (kPage - 1);
    const int eb = a.elem_bytes;
    const int x = 16 / eb;
    const int chunks = a.D / x;
    const int64_t tile_elems = (int64_t)a.D * kPage;

    char* kp = (char*)a.k_pages;
    const char* kn = (const char*)a.k_new;
    for (int i = threadIdx.x; i < a.H_kv * chunks; i += blockDim.x) {
        const int g = i / chunks, c = i - g * chunks;
        const int64_t src = (int64_t)b * a.new_sb + (int64_t)g * a.new_sh + (int64_t)c * x;
        const int64_t dst = (((int64_t)pg * a.H_kv + g) * chunks + c) * kPage + slot;  // 16-byte units
        *(u32x4*)(kp + dst * 16) = *(const u32x4*)(kn + src * eb);
    }
    char* vp = (char*)a.v_pages;
    const char* vn = (const char*)a.v_new;
    for (int i = threadIdx.x; i < a.H_kv * a.D; i += blockDim.x) {
        const int g = i / a.D, d = i - g * a.D;
        const int64_t src = (int64_t)b * a.vnew_sb + (int64_t)g * a.vnew_sh + d;
        const int64_t dst = ((int64_t)pg * a.H_kv + g) * tile_elems + (int64_t)d * kPage + slot;
        if (eb == 2)
            *(uint16_t*)(vp + dst * 2) = *(const uint16_t*)(vn + src * 2);
        else
            *(uint8_t*)(vp + dst) = *(const uint8_t*)(vn + src);
    }
    __syncthreads();  // every thread has read seq_lens[b]
    if (threadIdx.x == 0) a.seq_lens[b] = L + 1;
}

// -------------------------------------------------------------- planner ---
// One workgroup: split each request into chunks of split_pages pages, lay
// the (request, split, clamped length) jobs out request-major with an
// exclusive scan, and reset the work-stealing cursor.
__global__ void __launch_bounds__(1024) plan_kernel(AttnArgs a) {
    __shared__ int scan[1024];
    __shared__ int carry;
    const int tid = threadIdx.x;
    const int maxL = a.max_pages * kPage;
    if (tid == 0) carry = 0;
    __syncthreads();
    for (int base = 0; base < a.B; base += 1024) {
        const int b = base + tid;
        int ns = 0, L = 0;
        if (b < a.B) {
            L = a.seq_lens[b];
            if (L < 0 || L > maxL) {
                atomicOr(&a.hdr->err_flags, kErrLength);
                L = L < 0 ? 0 : maxL;
            }
            const int np = (L + kPage - 1) / kPage;
            ns = (np + a.split_pages - 1) / a.split_pages;
        }
        scan[tid] = ns;
        __syncthreads();
        for (int off = 1; off < 1024; off <<= 1) {
            const int v = tid >= off ? scan[tid - off] : 0;
            __syncthreads();
            scan[tid] += v;
            __syncthreads();
        }
        const int excl = carry + scan[tid] - ns;
        if (b < a.B) {
            a.job_start[b] = excl;
            for (int s = 0; s < ns; ++s) a.jobs[excl + s] = make_int4(b, s, L, 0);
        }
        __syncthreads();
        if (tid == 1023) carry += scan[1023];
        __syncthreads();
    }
    if (tid == 0) {
        a.job_start[a.B] = carry;
        a.hdr->njobs = carry;
        a.hdr->counter = 0;
    }
}

// ------------------------------------------------ partial attention (MFMA) --
// Each wave takes work items = (request b, split s, KV head g) in turn and
// streams each split's pages two at a time:
//   S^T[slot, head] = K_page[slot, :] . Q^T[:, head]   (v_mfma 16x16x32 bf16)
//   online softmax per head in base 2, once per 32 tokens
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
template <int D, bool FP8>
struct PageRegs {
    static constexpr int NT = D / 16;
    static constexpr int KS = D / 32;
    static constexpr int KC = FP8 ? D / 64 : KS;  // 16-byte K loads per lane
    u32x4 k[KC];
    typename std::conditional<FP8, uint32_t, u32x2>::type v[NT];
};

// K/V pages are read exactly once per step: non-temporal loads keep them from
// displacing reusable lines in the caches, which measurably raises the
// sustained read rate of the gather.
template <typename T>
__device__ __forceinline__ T ld_stream(const char* p) {
    return __builtin_nontemporal_load((const T*)p);
}

template <int D, bool FP8>
__device__ __forceinline__ void load_page(PageRegs<D, FP8>& r, const char* kbase, const char* vbase,
                                          int qg, int n) {
    constexpr int NT = D / 16;
    if constexpr (!FP8) {
        // K chunk c = 4j + qg (8 dims), slot n: 16 bytes; one load instruction
        // covers 1 KiB contiguous.
#pragma unroll
        for (int j = 0; j < PageRegs<D, FP8>::KC; ++j)
            r.k[j] = ld_stream<u32x4>(kbase + ((size_t)((4 * j + qg) * kPage + n)) * 16);
        // V dims 16t + n, slots 4qg..4qg+3: 8 bytes; 512 bytes contiguous per instruction.
#pragma unroll
        for (int t = 0; t < NT; ++t)
            r.v[t] = ld_stream<u32x2>(vbase + ((size_t)((16 * t + n) * kPage + 4 * qg)) * 2);
    } else {
        // K chunk c = qg + 4i (16 dims), slot n: 16 bytes.
#pragma unroll
        for (int i = 0; i < PageRegs<D, FP8>::KC; ++i)
            r.k[i] = ld_stream<u32x4>(kbase + ((size_t)((qg + 4 * i) * kPage + n)) * 16);
#pragma unroll
        for (int t = 0; t < NT; ++t)
            r.v[t] = ld_stream<uint32_t>(vbase + (size_t)((16 * t + n) * kPage + 4 * qg));
    }
}

// Scores of one page: lane (qg, n) gets head n at slots 4qg..4qg+3.
template <int D, bool FP8>
__device__ __forceinline__ f32x4 page_scores(const PageRegs<D, FP8>& r, const bf16x8 (&bq)[D / 32]) {
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
__device__ __forceinline__ u32x2 v_quad(const PageRegs<D, FP8>& r, int t, int nv, int qg) {
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

template <int D, bool FP8>
__device__ __forceinline__ void attend_pair(AttnState<D>& st, const PageRegs<D, FP8>& ra, const PageRegs<D, FP8>& rb,
                                            const bf16x8 (&bq)[D / 32], float sl, int nva, int nvb, int qg) {
    constexpr int NT = D / 16;
    const f32x4 sa = page_scores<D, FP8>(ra, bq);
    f32x4 sb = {0.f, 0.f, 0.f, 0.f};
    if (nvb > 0) sb = page_scores<D, FP8>(rb, bq);

    float x[8];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[i] = (4 * qg + i < nva) ? sa[i] * sl : -INFINITY;
        x[4 + i] = (4 * qg + i < nvb) ? sb[i] * sl : -INFINITY;
        mx = fmaxf(mx, fmaxf(x[i], x[4 + i]));
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(st.m, mx);
    if (__any(m_new > st.m)) {
        const float alpha = fast_exp2(st.m - m_new);
        st.l *= alpha;
#pragma unroll
        for (int t = 0; t < NT; ++t) st.o[t] *= alpha;
        st.m = m_new;
    }

    uint32_t ph[4], pl[4];
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
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
    const bf16x8 bph = __builtin_bit_cast(bf16x8, u32x4{ph[0], ph[1], ph[2], ph[3]});
    const bf16x8 bpl = __builtin_bit_cast(bf16x8, u32x4{pl[0], pl[1], pl[2], pl[3]});

#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const u32x2 va = v_quad<D, FP8>(ra, t, nva, qg);
        const u32x2 vb = v_quad<D, FP8>(rb, t, nvb, qg);
        const bf16x8 av = __builtin_bit_cast(bf16x8, u32x4{va.x, va.y, vb.x, vb.y});
        st.o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bph, st.o[t], 0, 0, 0);
        st.o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bpl, st.o[t], 0, 0, 0);
    }
}

template <int D, bool FP8>
__global__ void __launch_bounds__(kAttnBlock) __attribute__((amdgpu_waves_per_eu(2))) attn_mfma_kernel(AttnArgs a) {
    constexpr int NT = D / 16;
    constexpr int KS = D / 32;
    constexpr int EB = FP8 ? 1 : 2;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int qg = lane >> 4;
    const int n = lane & 15;
    const int total = a.hdr->njobs * a.H_kv;
    const size_t tile_bytes = (size_t)D * kPage * EB;
    const size_t page_stride = (size_t)a.H_kv * tile_bytes;

    // Items are dealt round-robin over all resident waves: wave w takes items
    // w, w + W, w + 2W, ...  Consecutive items are the KV heads of one
    // (request, split) job, so neighbouring waves get equal-sized items and
    // every wave's share averages over many jobs.
    const int waves = gridDim.x * (kAttnBlock / kWaveSize);
    for (int item = blockIdx.x * (kAttnBlock / kWaveSize) + (threadIdx.x >> 6); item < total; item += waves) {

        const int job = item / a.H_kv;
        const int g = item - job * a.H_kv;
        const int4 js = a.jobs[job];
        const int b = js.x, s = js.y, L = js.z;
        const int np_total = (L + kPage - 1) / kPage;
        const int nsplit = (np_total + a.split_pages - 1) / a.split_pages;
        const int p_begin = s * a.split_pages;
        const int np = min(a.split_pages, np_total - p_begin);

        // this split's block-table entries, one per lane
        int my_pg = 0;
        if (lane < np) my_pg = a.block_table[(int64_t)b * a.bt_stride + p_begin + lane];
        const bool lane_bad = lane < np && (my_pg < 0 || (int64_t)my_pg >= a.num_pages);
        const bool bad = __any(lane_bad);
        if (bad && lane == 0) atomicOr(&a.hdr->err_flags, kErrPage);

        // query operand: lane (qg, n) holds head g*G+n (zeros past the group)
        const int h = g * a.G + n;
        const bool hv = n < a.G;
        bf16x8 bq[KS];
        {
            const uint16_t* qrow = a.q + (int64_t)b * a.q_sb + (int64_t)h * a.q_sh;
#pragma unroll
            for (int j = 0; j < KS; ++j) {
                const int dim0 = FP8 ? 16 * (qg + 4 * (j >> 1)) + 8 * (j & 1) : 8 * (4 * j + qg);
                u32x4 w = {0u, 0u, 0u, 0u};
                if (hv) w = *(const u32x4*)(qrow + dim0);
                bq[j] = __builtin_bit_cast(bf16x8, w);
            }
        }
        const float sl = FP8 ? a.scale_log2 * a.k_scale[(int64_t)b * a.H_kv + g] : a.scale_log2;

        AttnState<D> st;
#pragma unroll
        for (int t = 0; t < NT; ++t) st.o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        st.m = -INFINITY;
        st.l = 0.f;

        if (!bad) {
            const char* kpool = (const char*)a.k_pages + (size_t)g * tile_bytes;
            const char* vpool = (const char*)a.v_pages + (size_t)g * tile_bytes;
            const int tok0 = p_begin * kPage;
            const int npairs = (np + 1) >> 1;
            // Every iteration issues the same 24 loads (two pages of K and V)
            // so that the wait before each pair covers only that pair's loads;
            // indices are clamped, so the odd tail page and the prefetch past
            // the last pair re-read an in-bounds page of this split (cache
            // hits) whose slots are masked or never used.
            PageRegs<D, FP8> r0a, r0b, r1a, r1b;
            auto load_pair = [&](PageRegs<D, FP8>& ra, PageRegs<D, FP8>& rb, int pair) {
                const int pa = __builtin_amdgcn_readlane(my_pg, min(2 * pair, np - 1));
                const int pb = __builtin_amdgcn_readlane(my_pg, min(2 * pair + 1, np - 1));
                load_page<D, FP8>(ra, kpool + pa * page_stride, vpool + pa * page_stride, qg, n);
                load_page<D, FP8>(rb, kpool + pb * page_stride, vpool + pb * page_stride, qg, n);
            };
            auto live = [&](int page) { return page < np ? min(kPage, L - tok0 - page * kPage) : 0; };
            load_pair(r0a, r0b, 0);
            for (int pr = 0;;) {
                load_pair(r1a, r1b, pr + 1);
                attend_pair<D, FP8>(st, r0a, r0b, bq, sl, live(2 * pr), live(2 * pr + 1), qg);
                if (++pr >= npairs) break;
                load_pair(r0a, r0b, pr + 1);
                attend_pair<D, FP8>(st, r1a, r1b, bq, sl, live(2 * pr), live(2 * pr + 1), qg);
                if (++pr >= npairs) break;
            }
        }

        float l_tot = st.l + __shfl_xor(st.l, 16);
        l_tot += __shfl_xor(l_tot, 32);
        const float vs = FP8 ? a.v_scale[(int64_t)b * a.H_kv + g] : 1.f;
        if (hv) {
            if (nsplit == 1) {
                const float f = bad ? NAN : vs / l_tot;
                uint16_t* orow = a.out + (int64_t)b * a.o_sb + (int64_t)h * a.o_sh;
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    u32x2 pk;
                    pk.x = (uint32_t)f32_to_bf16_rne(st.o[t][0] * f) | ((uint32_t)f32_to_bf16_rne(st.o[t][1] * f) << 16);
                    pk.y = (uint32_t)f32_to_bf16_rne(st.o[t][2] * f) | ((uint32_t)f32_to_bf16_rne(st.o[t][3] * f) << 16);
                    *(u32x2*)(orow + 16 * t + 4 * qg) = pk;
                }
            } else {
                const int64_t pidx = (int64_t)job * a.H_q + h;
                float* po = a.part_o + pidx * D;
                const float f = bad ? NAN : vs;
#pragma unroll
                for (int t = 0; t < NT; ++t) *(f32x4*)(po + 16 * t + 4 * qg) = st.o[t] * f;
                if (qg == 0) a.part_ml[pidx] = make_float2(bad ? NAN : st.m, l_tot);
            }
        }
    }
}

// ----------------------------------------------------------------- merge ---
// One wave per (request, query head): combine the splits' partial results
//   M = max_s m_s,  l = sum_s 2^(m_s - M) l_s,  out = sum_s 2^(m_s - M) o_s / l
// in split order (deterministic).  Requests with a single split were written
// by the partial kernel; requests of length 0 get zeros.
template <int D>
__global__ void __launch_bounds__(256) merge_kernel(AttnArgs a) {
    const int wid = blockIdx.x * (256 / kWaveSize) + (threadIdx.x >> 6);
    const int lane = threadIdx.x & (kWaveSize - 1);
    if (wid >= a.B * a.H_q) return;
    const int b = wid / a.H_q, h = wid - b * a.H_q;
    const int maxL = a.max_pages * kPage;
    const int L = min(max(a.seq_lens[b], 0), maxL);
    const int np_total = (L + kPage - 1) / kPage;
    const int nsplit = (np_total + a.split_pages - 1) / a.split_pages;
    uint16_t* orow = a.out + (int64_t)b * a.o_sb + (int64_t)h * a.o_sh;
    if (nsplit == 1) return;
    if (nsplit == 0) {
        for (int d = lane; d < D; d += kWaveSize) orow[d] = 0;
        return;
    }
    const int j0 = a.job_start[b];
    float M = -INFINITY;
    for (int s = 0; s < nsplit; ++s) M = fmaxf(M, a.part_ml[(int64_t)(j0 + s) * a.H_q + h].x);
    float l = 0.f;
    float acc[D / kWaveSize];
#pragma unroll
    for (int k = 0; k < D / kWaveSize; ++k) acc[k] = 0.f;
    for (int s = 0; s < nsplit; ++s) {
        const int64_t pidx = (int64_t)(j0 + s) * a.H_q + h;
        const float2 ml = a.part_ml[pidx];
        const float w = fast_exp2(ml.x - M);
        l += w * ml.y;
        const float* po = a.part_o + pidx * D;
#pragma unroll
        for (int k = 0; k < D / kWaveSize; ++k) acc[k] += w * po[lane + kWaveSize * k];
    }
    const float inv = 1.f / l;
#pragma unroll
    for (int k = 0; k < D / kWaveSize; ++k) orow[lane + kWaveSize * k] = f32_to_bf16_rne(acc[k] * inv);
}

}  // namespace

// ------------------------------------------------------------- launchers ---

void launch_kv_append(const AppendArgs& a, hipStream_t s) {
    if (a.B == 0) return;
    hipLaunchKernelGGL(kv_append_kernel, dim3(a.B), dim3(256), 0, s, a);
}

void launch_plan(const AttnArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(1024), 0, s, a);
}

void launch_attention(const AttnArgs& a, int impl, bool fp8, int grid, hipStream_t s) {
    (void)impl;
    if (a.B == 0 || a.H_q == 0) return;
    const dim3 g(grid), blk(kAttnBlock);
    if (a.D == 128) {
        if (fp8)
            hipLaunchKernelGGL((attn_mfma_kernel<128, true>), g, blk, 0, s, a);
        else
            hipLaunchKernelGGL((attn_mfma_kernel<128, false>), g, blk, 0, s, a);
    } else {
        if (fp8)
            hipLaunchKernelGGL((attn_mfma_kernel<64, true>), g, blk, 0, s, a);
        else
            hipLaunchKernelGGL((attn_mfma_kernel<64, false>), g, blk, 0, s, a);
    }
}

int attention_blocks_per_cu(int impl, bool fp8, int D) {
    (void)impl;
    int nb = 0;
    hipError_t e;
    if (D == 128)
        e = fp8 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, attn_mfma_kernel<128, true>, kAttnBlock, 0)
                : hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, attn_mfma_kernel<128, false>, kAttnBlock, 0);
    else
        e = fp8 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, attn_mfma_kernel<64, true>, kAttnBlock, 0)
                : hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, attn_mfma_kernel<64, false>, kAttnBlock, 0);
    if (e != hipSuccess || nb < 1) nb = 1;
    return nb;
}

void launch_merge(const AttnArgs& a, hipStream_t s) {
    const int pairs = a.B * a.H_q;
    if (pairs == 0) return;
    const dim3 g((pairs + 3) / 4), blk(256);
    if (a.D == 128)
        hipLaunchKernelGGL(merge_kernel<128>, g, blk, 0, s, a);
    else
        hipLaunchKernelGGL(merge_kernel<64>, g, blk, 0, s, a);
}

}  // namespace bellman
