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
// the (request, split) jobs out request-major with an exclusive scan, and
// reset the work-stealing cursor.
__global__ void __launch_bounds__(1024) plan_kernel(AttnArgs a) {
    __shared__ int scan[1024];
    __shared__ int carry;
    const int tid = threadIdx.x;
    const int maxL = a.max_pages * kPage;
    if (tid == 0) carry = 0;
    __syncthreads();
    for (int base = 0; base < a.B; base += 1024) {
        const int b = base + tid;
        int ns = 0;
        if (b < a.B) {
            int L = a.seq_lens[b];
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
            for (int s = 0; s < ns; ++s) a.jobs[excl + s] = make_int2(b, s);
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
// Each wave repeatedly takes one work item = (request b, split s, KV head g)
// from a device-wide cursor and streams the split's pages:
//   S^T[slot, head] = K_page[slot, :] . Q^T[:, head]   (v_mfma 16x16x32 bf16)
//   online softmax per head in base 2
//   O^T[dim, head] += V_page^T[dim, slot] . P^T[slot, head]   (v_mfma 16x16x16)
// Lane l = 16*qg + n.  In the QK product n is the page slot (A row) and the
// query head of the group (B column); the result leaves lane (qg, n) with the
// scores of head n at slots 4qg..4qg+3, which are exactly the four B
// elements the PV product needs from that lane, so no data crosses lanes
// except the max/sum reductions over qg.  P enters the PV product as a bf16
// pair hi + lo (hi = truncation, lo = rounded remainder), which keeps P to
// about 2^-16 relative.  Slots past the request's length are excluded: their
// scores become -inf and their V elements are replaced by zeros.
template <int D, bool FP8>
struct PageRegs {
    static constexpr int NT = D / 16;
    static constexpr int KS = D / 32;
    static constexpr int KC = FP8 ? D / 64 : KS;  // 16-byte K loads per lane
    u32x4 k[KC];
    typename std::conditional<FP8, uint32_t, u32x2>::type v[NT];
};

template <int D, bool FP8>
__device__ __forceinline__ void load_page(PageRegs<D, FP8>& r, const char* kbase, const char* vbase,
                                          int qg, int n) {
    constexpr int NT = D / 16;
    if constexpr (!FP8) {
        // K chunk c = 4j + qg (8 dims), slot n: 16 bytes; one load instruction
        // covers 1 KiB contiguous.
#pragma unroll
        for (int j = 0; j < PageRegs<D, FP8>::KC; ++j)
            r.k[j] = *(const u32x4*)(kbase + ((size_t)((4 * j + qg) * kPage + n)) * 16);
        // V dims 16t + n, slots 4qg..4qg+3: 8 bytes.
#pragma unroll
        for (int t = 0; t < NT; ++t)
            r.v[t] = *(const u32x2*)(vbase + ((size_t)((16 * t + n) * kPage + 4 * qg)) * 2);
    } else {
        // K chunk c = qg + 4i (16 dims), slot n: 16 bytes.
#pragma unroll
        for (int i = 0; i < PageRegs<D, FP8>::KC; ++i)
            r.k[i] = *(const u32x4*)(kbase + ((size_t)((qg + 4 * i) * kPage + n)) * 16);
#pragma unroll
        for (int t = 0; t < NT; ++t)
            r.v[t] = *(const uint32_t*)(vbase + (size_t)((16 * t + n) * kPage + 4 * qg));
    }
}

template <int D, bool FP8>
struct AttnState {
    f32x4 o[D / 16];
    float m;   // running max, log2 units
    float l;   // this lane's partial sum of weights
};

template <int D, bool FP8>
__device__ __forceinline__ void attend_page(AttnState<D, FP8>& st, const PageRegs<D, FP8>& r,
                                            const bf16x8 (&bq)[D / 32], float sl, int nv, int qg) {
    constexpr int NT = D / 16;
    constexpr int KS = D / 32;
    f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < KS; ++j) {
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
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kk), bq[j], sacc, 0, 0, 0);
    }

    float x[4];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[i] = (4 * qg + i < nv) ? sacc[i] * sl : -INFINITY;
        mx = fmaxf(mx, x[i]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(st.m, mx);
    const float alpha = fast_exp2(st.m - m_new);
    st.m = m_new;

    s16x4 ph, pl;
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float p = fast_exp2(x[i] - m_new);
        psum += p;
        const uint32_t u = __float_as_uint(p);
        const float hi = __uint_as_float(u & 0xffff0000u);
        ph[i] = (short)(u >> 16);
        pl[i] = (short)f32_to_bf16_rne(p - hi);
    }
    st.l = st.l * alpha + psum;

#pragma unroll
    for (int t = 0; t < NT; ++t) {
        st.o[t] *= alpha;
        u32x2 vv;
        if constexpr (!FP8) {
            vv = r.v[t];
        } else {
            vv.x = fp8x2_to_bf16x2(r.v[t], false);
            vv.y = fp8x2_to_bf16x2(r.v[t], true);
        }
        s16x4 av = __builtin_bit_cast(s16x4, vv);
        if (nv < kPage) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (4 * qg + i >= nv) av[i] = 0;
        }
        st.o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, ph, st.o[t], 0, 0, 0);
        st.o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, pl, st.o[t], 0, 0, 0);
    }
}

template <int D, bool FP8>
__global__ void __launch_bounds__(kAttnBlock) attn_mfma_kernel(AttnArgs a) {
    constexpr int NT = D / 16;
    constexpr int KS = D / 32;
    constexpr int EB = FP8 ? 1 : 2;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int qg = lane >> 4;
    const int n = lane & 15;
    const int total = a.hdr->njobs * a.H_kv;
    const int maxL = a.max_pages * kPage;
    const size_t tile_bytes = (size_t)D * kPage * EB;

    for (;;) {
        int item = 0;
        if (lane == 0) item = atomicAdd(&a.hdr->counter, 1);
        item = __builtin_amdgcn_readfirstlane(item);
        if (item >= total) break;
        const int job = item / a.H_kv;
        const int g = item - job * a.H_kv;
        const int2 js = a.jobs[job];
        const int b = js.x, s = js.y;
        const int L = min(max(a.seq_lens[b], 0), maxL);
        const int np_total = (L + kPage - 1) / kPage;
        const int nsplit = (np_total + a.split_pages - 1) / a.split_pages;
        const int p_begin = s * a.split_pages;
        const int np = min(a.split_pages, np_total - p_begin);

        // this split's block-table entries, one per lane
        int my_pg = 0;
        if (lane < np) my_pg = a.block_table[(int64_t)b * a.bt_stride + p_begin + lane];
        const bool lane_bad = lane < np && (my_pg < 0 || (int64_t)my_pg >= a.num_pages);
        const bool bad = __ballot(lane_bad) != 0;
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

        AttnState<D, FP8> st;
#pragma unroll
        for (int t = 0; t < NT; ++t) st.o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        st.m = -INFINITY;
        st.l = 0.f;

        if (!bad && np > 0) {
            const char* kpool = (const char*)a.k_pages + (size_t)g * tile_bytes;
            const char* vpool = (const char*)a.v_pages + (size_t)g * tile_bytes;
            const size_t page_stride = (size_t)a.H_kv * tile_bytes;
            const int tok0 = p_begin * kPage;
            PageRegs<D, FP8> ra, rb;
            {
                const int pg = __builtin_amdgcn_readlane(my_pg, 0);
                load_page<D, FP8>(ra, kpool + pg * page_stride, vpool + pg * page_stride, qg, n);
            }
            for (int i = 0; i < np; i += 2) {
                if (i + 1 < np) {
                    const int pg = __builtin_amdgcn_readlane(my_pg, i + 1);
                    load_page<D, FP8>(rb, kpool + pg * page_stride, vpool + pg * page_stride, qg, n);
                }
                attend_page<D, FP8>(st, ra, bq, sl, min(kPage, L - tok0 - i * kPage), qg);
                if (i + 1 < np) {
                    if (i + 2 < np) {
                        const int pg = __builtin_amdgcn_readlane(my_pg, i + 2);
                        load_page<D, FP8>(ra, kpool + pg * page_stride, vpool + pg * page_stride, qg, n);
                    }
                    attend_page<D, FP8>(st, rb, bq, sl, min(kPage, L - tok0 - (i + 1) * kPage), qg);
                }
            }
        }

        float l_tot = st.l + __shfl_xor(st.l, 16);
        l_tot += __shfl_xor(l_tot, 32);
        const float vs = FP8 ? a.v_scale[(int64_t)b * a.H_kv + g] : 1.f;
        if (!hv) continue;
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
