// Prompt (prefill) path over the paged KV cache: the write of a prompt's
// keys and values into its pages, and causal prompt attention (each query
// token attends every cached token up to its own position), for gfx950.
//
// The paper's serving loop (Sec. 3 "Our key proposal", Sec. 4 "Setup and
// trace") prefills each queued request's prompt before decoding; the
// prefill's cost sets the time to first token.  The attention is a dense
// contraction (QK^T and PV over head_dim and keys), so it runs on
// v_mfma_f32_32x32x16_bf16, with the keys and values staged through LDS and
// shared by the workgroup's four waves.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "../../include/bellman.h"
#include "internal.h"

namespace bellman {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float swap_halves(float x) {  // value of lane l ^ 32
    const unsigned u = __float_as_uint(x);
    // the swap exchanges the first operand's lanes 32..63 with the second
    // operand's lanes 0..31: the upper half finds its partner in r[0], the
    // lower half in r[1]
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}

// ----------------------------------------------------------- prompt write --
// Work is cut by (request, page the request's new positions touch, KV head):
// write_plan_kernel scans the touched-page counts of the requests into
// page_start[0..B]; kv_write_kernel takes one item per workgroup.  A K page
// [D/x chunks][16 slots][x] takes 16-byte units with consecutive threads on
// consecutive slots; the V rows of the page's tokens go through LDS and
// leave as 16-byte runs of the dim-major V page [D][16 slots] (element by
// element where the page is only partly written).  Lengths are advanced
// afterwards by lens_kernel, so every item sees its request's old length.
constexpr int kPlanThreads = 1024;

// Inclusive scan of one value per thread over a kPlanThreads block.
__device__ __forceinline__ int block_scan(int v, int* part) {
    const int tid = threadIdx.x;
    part[tid] = v;
    __syncthreads();
    for (int off = 1; off < kPlanThreads; off <<= 1) {
        const int x = tid >= off ? part[tid - off] : 0;
        __syncthreads();
        part[tid] += x;
        __syncthreads();
    }
    return part[tid];
}

// Pages request b's new positions touch, or -1 for a malformed request
// (negative or reversed range, rows past T, negative length).
__device__ __forceinline__ int pages_touched(const WriteArgs& a, int b) {
    const int s0 = a.q_start[b], s1 = a.q_start[b + 1];
    const int L = a.seq_lens[b];
    if (s0 < 0 || s1 < s0 || s1 > a.T || L < 0) return -1;
    if (s1 == s0) return 0;
    const int64_t last = (int64_t)L + (s1 - s0) - 1;
    return (int)(last / kPage - L / kPage + 1);
}

__global__ void __launch_bounds__(kPlanThreads) write_plan_kernel(WriteArgs a, int32_t* page_start) {
    __shared__ int part[kPlanThreads];
    __shared__ int malformed;
    const int tid = threadIdx.x;
    if (tid == 0) malformed = (a.q_start[0] < 0 || a.q_start[a.B] > a.T) ? 1 : 0;
    __syncthreads();
    const int per = (a.B + kPlanThreads - 1) / kPlanThreads;
    const int b0 = tid * per;
    int sum = 0, bad = 0;
    for (int k = 0; k < per; ++k) {
        const int b = b0 + k;
        if (b >= a.B) break;
        if (a.q_start[b + 1] < a.q_start[b]) atomicOr(&malformed, 1);
        const int t = pages_touched(a, b);
        if (t < 0) bad = 1;
        else sum += t;
    }
    if (bad) atomicOr(a.err, kErrAppendSlot);
    const int incl = block_scan(sum, part);
    if (malformed) {
        for (int k = 0; k < per; ++k)
            if (b0 + k < a.B) page_start[b0 + k] = 0;
        if (tid == 0) {
            page_start[a.B] = 0;
            atomicOr(a.err, kErrAppendSlot);
        }
        return;
    }
    int run = incl - sum;
    for (int k = 0; k < per; ++k) {
        const int b = b0 + k;
        if (b < a.B) {
            page_start[b] = run;
            run += max(pages_touched(a, b), 0);
        }
    }
    if (tid == kPlanThreads - 1) {
        page_start[a.B] = incl;
        if (a.q_start[a.B] < a.T) atomicOr(a.err, kErrAppendSlot);   // rows no request owns
    }
}

template <int EB>
__global__ void __launch_bounds__(256) kv_write_kernel(WriteArgs a, const int32_t* page_start) {
    __shared__ __attribute__((aligned(16))) uint8_t vst[kPage * 128 * 2];   // the page's V rows, one head
    const int item = blockIdx.x, g = blockIdx.y, tid = threadIdx.x;
    if (item >= page_start[a.B]) return;
    int lo = 0, hi = a.B - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (page_start[mid] <= item) lo = mid;
        else hi = mid - 1;
    }
    const int b = lo;
    const int s0 = a.q_start[b], L = a.seq_lens[b];
    const int n = a.q_start[b + 1] - s0;
    const int pi = L / kPage + (item - page_start[b]);
    const int64_t first = (int64_t)kPage * pi;              // position of slot 0
    const int slot_lo = (int)(max((int64_t)L, first) - first);
    const int slot_hi = (int)(min((int64_t)L + n, first + kPage) - first);
    int pg = -1;
    if (pi < a.max_pages) pg = a.block_table[(int64_t)b * a.bt_stride + pi];
    if (pg < 0 || pg >= a.num_pages) {
        if (g == 0 && tid == 0) atomicOr(a.err, kErrAppendSlot);
        return;
    }
    const int64_t row0 = s0 + (first - L);                   // token row of slot 0
    constexpr int x = 16 / EB;                               // elements per 16-byte unit
    const int chunks = a.D / x;
    const char* kn = (const char*)a.k_new;
    const char* vn = (const char*)a.v_new;
    char* kp = (char*)a.k_pages + ((int64_t)pg * a.H_kv + g) * (int64_t)a.D * kPage * EB;
    char* vp = (char*)a.v_pages + ((int64_t)pg * a.H_kv + g) * (int64_t)a.D * kPage * EB;
    for (int u = tid; u < chunks * kPage; u += 256) {
        const int c = u / kPage, sl = u % kPage;
        if (sl < slot_lo || sl >= slot_hi) continue;
        const char* src = kn + ((row0 + sl) * a.k_st + (int64_t)g * a.k_sh + (int64_t)c * x) * EB;
        *(u32x4*)(kp + (int64_t)u * 16) = *(const u32x4*)src;
    }
    const int row_units = a.D * EB / 16;                     // 16-byte units of one token's V row
    for (int u = tid; u < kPage * row_units; u += 256) {
        const int sl = u / row_units, k = u % row_units;
        if (sl < slot_lo || sl >= slot_hi) continue;
        *(u32x4*)&vst[u * 16] = *(const u32x4*)(vn + ((row0 + sl) * a.v_st + (int64_t)g * a.v_sh) * EB + k * 16);
    }
    __syncthreads();
    // V page rows: unit (d, h) holds slots h x .. h x + x - 1 of dim d
    const int row_bytes = a.D * EB;
    for (int u = tid; u < a.D * EB; u += 256) {
        const int d = u / EB, h = u % EB;
        const int sa = h * x;
        char* dst = vp + (int64_t)u * 16;
        if (sa >= slot_lo && sa + x <= slot_hi) {
            uint8_t buf[16];
#pragma unroll
            for (int e = 0; e < x; ++e)
#pragma unroll
                for (int q = 0; q < EB; ++q) buf[e * EB + q] = vst[(sa + e) * row_bytes + d * EB + q];
            *(u32x4*)dst = *(const u32x4*)buf;
        } else {
            for (int sl = max(sa, slot_lo); sl < min(sa + x, slot_hi); ++sl)
                for (int q = 0; q < EB; ++q) dst[(sl - sa) * EB + q] = (char)vst[sl * row_bytes + d * EB + q];
        }
    }
}

// Each request's length grows by its token count (when its last position
// fits the table).
__global__ void lens_kernel(WriteArgs a) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= a.B) return;
    const int n = a.q_start[b + 1] - a.q_start[b];
    const int L = a.seq_lens[b];
    if (n < 0 || L < 0 || (int64_t)L + n > (int64_t)a.max_pages * kPage || a.q_start[b + 1] > a.T) {
        atomicOr(a.err, kErrAppendSlot);
        return;
    }
    a.seq_lens[b] = L + n;
}

// --------------------------------------------------------------- planning --
// Exclusive scan of the requests' query-tile counts, ceil(n_b / 128), into
// tile_start[0..B].  A request whose range is malformed (longer than its
// length, or a length past the table) gets no tiles and a flag; a q_start
// that is not non-decreasing from a non-negative start up to at most T gives
// no request any tile (so the tiles always fit the grid of
// ceil(T / 128) + B workgroups).
__device__ __forceinline__ int tiles_of(const PrefillArgs& a, int b) {
    const int n = a.q_start[b + 1] - a.q_start[b], L = a.seq_lens[b];
    if (n < 0 || n > L || (int64_t)L > (int64_t)a.max_pages * kPage) return -1;
    return (n + kPrefillRows - 1) / kPrefillRows;
}

// pages of request b whose values the attention reads: all ceil(L_b / 16)
// when it has query tiles, none otherwise
__device__ __forceinline__ int vpages_of(const PrefillArgs& a, int b) {
    return tiles_of(a, b) > 0 ? (a.seq_lens[b] + kPage - 1) / kPage : 0;
}

__global__ void __launch_bounds__(kPlanThreads) prefill_plan_kernel(PrefillArgs a) {
    __shared__ int part[kPlanThreads];
    __shared__ int malformed;
    __shared__ int total_pages;
    const int tid = threadIdx.x;
    if (tid == 0) malformed = (a.q_start[0] < 0 || a.q_start[a.B] > a.T) ? 1 : 0;
    __syncthreads();
    const int per = (a.B + kPlanThreads - 1) / kPlanThreads;
    const int b0 = tid * per;
    int sum = 0, bad = 0;
    for (int k = 0; k < per; ++k) {
        const int b = b0 + k;
        if (b >= a.B) break;
        if (a.q_start[b + 1] < a.q_start[b]) atomicOr(&malformed, 1);
        const int t = tiles_of(a, b);
        if (t < 0) bad = 1;
        else sum += t;
    }
    if (bad) atomicOr(a.err, kErrLength);
    const int incl = block_scan(sum, part);
    if (!a.fp8) {
        // bf16 pools: the pages the value copy holds (every page of a request
        // with query tiles, none of the others; none at all when malformed)
        int pages = 0;
        for (int k = 0; k < per; ++k)
            if (b0 + k < a.B && !malformed) pages += vpages_of(a, b0 + k);
        const int pincl = block_scan(pages, part);
        int prun = pincl - pages;
        for (int k = 0; k < per; ++k) {
            const int b = b0 + k;
            if (b < a.B) {
                a.page_off[b] = prun;
                prun += malformed ? 0 : vpages_of(a, b);
            }
        }
        if (tid == kPlanThreads - 1) {
            a.page_off[a.B] = pincl;
            total_pages = pincl;
        }
        __syncthreads();   // page_off is read back below by every thread
        // the request of every copied page: the last b with page_off[b] <= p
        for (int p = tid; p < total_pages; p += kPlanThreads) {
            int lo = 0, hi = a.B - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (a.page_off[mid] <= p) lo = mid;
                else hi = mid - 1;
            }
            a.page_req[p] = lo;
        }
    }
    if (malformed) {
        for (int k = 0; k < per; ++k)
            if (b0 + k < a.B) a.tile_start[b0 + k] = 0;
        if (tid == 0) {
            a.tile_start[a.B] = 0;
            atomicOr(a.err, kErrLength);
        }
        return;
    }
    int run = incl - sum;
    for (int k = 0; k < per; ++k) {
        const int b = b0 + k;
        if (b < a.B) {
            a.tile_start[b] = run;
            run += max(tiles_of(a, b), 0);
        }
    }
    if (tid == kPlanThreads - 1) a.tile_start[a.B] = incl;
}

// ------------------------------------------------ fp16 copy of bf16 values --
// Over bf16 pools PV runs in fp16, in one pass (P, below 2^8, keeps 11
// significant bits in fp16; rounded to bf16 once it would spend the bf16
// error budget).  Each (request, KV head)'s values are copied into the
// workspace as fp16 at a power-of-two scale 2^e that puts their largest
// magnitude M in [2^14, 2^15): bf16's 8 significant bits fit fp16's 11, so
// every value of at least M 2^-28 converts exactly and none overflows, and
// the rest keep an absolute error below M 2^-40.  The copy keeps the pool's
// page layout [page][D][16 slots], a request's pages consecutive from
// page_off[b], slots past its length zero.  Three passes, none with
// atomics: vmax_kernel takes the largest magnitude of every (page, head)
// tile, vreduce_kernel M of every (request, KV head), and vcopy_kernel
// writes the copy.

// the scale exponent e for a largest magnitude whose float bits are mb
// (e = 0 when every value is zero or the maximum is not finite)
__device__ __forceinline__ int vcopy_exp(uint32_t mb) {
    if (mb == 0u || mb >= 0x7f800000u) return 0;
    const int E = max((int)(mb >> 23), 1);          // floor(log2 M) + 127
    return min(max(141 - E, -126), 126);
}
__device__ __forceinline__ float pow2f(int e) {   // 2^e, -126 <= e <= 127
    return __uint_as_float((uint32_t)(e + 127) << 23);
}

// The copy passes run a fixed grid of waves over the flat (page, KV head)
// tiles of all requests; page p of the copy belongs to request page_req[p]
// (written by the planner).  Each lane takes 4 (D = 128) or 2 16-byte units
// (8 slots of one dim row) of a tile, all loaded before any is used.
template <int D>
struct VTile {
    static constexpr int U = 2 * D / 64;   // units per lane
    int b, j, g, pg, L;
    u32x4 w[U];
    // load tile t (p = t / H_kv, g = t % H_kv); slots past the length read as 0
    __device__ __forceinline__ void load(const PrefillArgs& a, int64_t t, int lane) {
        const int64_t p = t / a.H_kv;
        g = (int)(t % a.H_kv);
        b = a.page_req[p];
        j = (int)(p - a.page_off[b]);
        L = a.seq_lens[b];
        pg = a.block_table[(int64_t)b * a.bt_stride + j];
        const bool ok = (unsigned)pg < (unsigned)a.num_pages;
        const uint16_t* src = (const uint16_t*)a.v_pages + ((int64_t)(ok ? pg : 0) * a.H_kv + g) * (D * kPage);
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int r = 64 * k + lane, s0 = 8 * (r & 1);
            w[k] = (ok && L - kPage * j - s0 > 0) ? *(const u32x4*)(src + (r >> 1) * kPage + s0) : u32x4{0u, 0u, 0u, 0u};
        }
    }
    // value i of unit k, 0 past the length
    __device__ __forceinline__ float value(int k, int i, int lane) const {
        const int r = 64 * k + lane, live = L - kPage * j - 8 * (r & 1);
        const uint32_t bits = (i & 1) ? (w[k][i >> 1] & 0xffff0000u) : (w[k][i >> 1] << 16);
        return i < live ? __uint_as_float(bits) : 0.f;
    }
};

__device__ __forceinline__ int64_t vcopy_tiles(const PrefillArgs& a) {
    return (int64_t)a.page_off[a.B] * a.H_kv;
}

// largest |v| of each (page, head) tile, in tmax[tile]
template <int D>
__global__ void __launch_bounds__(256) vmax_kernel(PrefillArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * 4, n = vcopy_tiles(a);
    for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < n; t += waves) {
        VTile<D> v;
        v.load(a, t, lane);
        float m = 0.f;
#pragma unroll
        for (int k = 0; k < VTile<D>::U; ++k)
#pragma unroll
            for (int i = 0; i < 8; ++i) m = fmaxf(m, fabsf(v.value(k, i, lane)));
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
        if (lane == 0) a.tmax[t] = m;
    }
}

// one wave per (request, KV head): vmax = float bits of the largest tile
// maximum over the request's pages (0 for a request without copied pages)
__global__ void __launch_bounds__(256) vreduce_kernel(PrefillArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= (int64_t)a.B * a.H_kv) return;
    const int b = (int)(i / a.H_kv), g = (int)(i % a.H_kv);
    const int p0 = a.page_off[b], np = a.page_off[b + 1] - p0;
    float m = 0.f;
    for (int j = lane; j < np; j += 64) m = fmaxf(m, a.tmax[((int64_t)p0 + j) * a.H_kv + g]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
    if (lane == 0) a.vmax[i] = __float_as_uint(m);
}

template <int D>
__global__ void __launch_bounds__(256) vcopy_kernel(PrefillArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * 4, n = vcopy_tiles(a);
    for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < n; t += waves) {
        VTile<D> v;
        v.load(a, t, lane);
        const float sc = pow2f(vcopy_exp(a.vmax[(int64_t)v.b * a.H_kv + v.g]));
        uint16_t* dst = a.vcopy + t * (int64_t)(D * kPage);   // tile t = (page, head) of the copy
#pragma unroll
        for (int k = 0; k < VTile<D>::U; ++k) {
            const int r = 64 * k + lane;
            u32x4 h;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const f32x2 x = {v.value(k, 2 * i, lane) * sc, v.value(k, 2 * i + 1, lane) * sc};
                h[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector(x, f16x2));   // round to nearest even
            }
            *(u32x4*)(dst + (r >> 1) * kPage + 8 * (r & 1)) = h;
        }
    }
}

// -------------------------------------------------------------- attention --
// Workgroup = 128 query rows of one request and one query head; wave w owns
// rows 32w..32w+31.  Keys go by steps of 64 (four pages).  The step's K and V
// tiles are copied from the pool straight into LDS (global_load_lds, 16 bytes
// a lane) in the pool's own layout (K [page][D/8 chunks][16 slots][8],
// V [page][D][16 slots], both XOR-swizzled against bank conflicts by the
// choice of unit each lane fetches), double-buffered in four separate arrays
// (so no read of one buffer waits on a copy into another), with K one step
// ahead of V, and read by all four waves.
//
// S^T = K Q^T on 32x32x16 MFMAs: A = 32 keys x 16 dims from LDS, B = the
// wave's 32 query columns, held in registers for the whole kernel.  A's row i
// holds key pi(i) = 16 (i / 16) + 8 ((i / 4) % 2) + 4 ((i / 8) % 2) + i % 4,
// which leaves lane (h, c) (h = lane / 32) of the result with query c and the
// keys 16 u + 8 h + 0..7 for u = 0, 1: the row max needs only the partner lane
// c + 32, and the lane's probabilities are exactly the B operand of
// O^T += V^T P^T for the 16 keys of page u, whose V^T elements are one
// 16-byte run of each dim-major V row.  Online softmax in base 2 with a lazy
// max: O and l are rescaled only when some column's max grows by more than
// 2^8, so P stays below 2^8.  P enters as bf16 (hi) plus the bf16 remainder
// (lo), carrying it to ~2^-17: P rounded to bf16 once would add up to 2^-9
// of every weight on top of the output's own 2^-9 rounding, more than the
// bf16 error budget allows.
//
// The loop is software-pipelined: step s masks and takes the max of S(s)
// (computed one step earlier), then issues the MFMAs of S(s + 1)
// interleaved with the exponentials of P(s), then the PV MFMAs of step s.
constexpr float kLazyMax = 8.0f;
constexpr int kPageWindow = 1024;   // block-table entries staged in LDS
constexpr int kXcds = 8;            // accelerator complexes; workgroup i runs on XCD i % 8
// VALU instructions of the softmax placed between consecutive S MFMAs
constexpr int kValuPerMfma = 7;

// FP8: pools of e4m3fn codes with per-(request, KV head) dequantisation
// scales.  The tiles reach LDS as codes (half the bytes) and each operand is
// widened exactly to bf16 before the same bf16 MFMAs; the K scale folds into
// the score scale and the V scale into the final normalisation.  A lane
// reads one whole 16-byte unit and feeds two MFMAs with its halves:
//  * S: A row i holds key pi8(i) = 16 ((i / 4) % 2) + 8 (i / 16) +
//    4 ((i / 8) % 2) + i % 4, so lane (h, c) of the result holds the keys
//    16 h + 8 e + 0..7 (e = 0, 1) of each 32-key half: page h of the half.
//    MFMA pair (2 m, 2 m + 1) reads, in lane (h, c), the unit of chunk
//    2 m + h of key pi8(c) and takes its codes 8 e .. 8 e + 7 into MFMA
//    2 m + e; the query operand of MFMA 2 m + e holds dims 32 m + 16 h + 8 e.
//  * PV: lane (h, c) reads row 32 t + c of page h of the half (16 keys) and
//    takes keys 8 e .. 8 e + 7 into MFMA e, whose P operand is then exactly
//    the lane's probabilities of group e.  PV runs in fp16, one pass: the
//    codes (at most 448 in magnitude, subnormals from 2^-9) are exact in
//    fp16, and P (below 2^8 with the lazy max) keeps 11 significant bits
//    there, against the bf16 hi + lo pair's two passes.
// Pages sit PB + 128 bytes apart in LDS and odd pages hold K slot s at
// s ^ 4, so every 8 (and 16) consecutive lanes of a read touch distinct
// banks.
template <int D, int NH, bool FP8>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
prefill_attn_kernel(PrefillArgs a) {
    constexpr int KS = 32 * NH;         // keys per step
    constexpr int PPS = KS / kPage;     // pages per step
    constexpr int EB = FP8 ? 1 : 2;     // bytes per pool element
    constexpr int PE = D * kPage;       // elements of one page of one head (K or V)
    constexpr int PB = PE * EB;         // its bytes
    constexpr int KT = PPS * PE;        // a step's K (or V) tile, elements
    constexpr int PBP = FP8 ? PB + 128 : PB;   // LDS bytes from one page of a tile to the next
    constexpr int KTW = PPS * PBP / 2;  // the tile in 16-bit words
    constexpr int UPP = PB / 16;        // 16-byte units per page
    constexpr int PER = 2 * PPS * UPP / 256;   // units of K + V per thread per step
    constexpr int WIN = kPageWindow / PPS;     // steps per block-table window
    __shared__ __attribute__((aligned(16))) uint16_t kb0[KTW];
    __shared__ __attribute__((aligned(16))) uint16_t kb1[KTW];
    __shared__ __attribute__((aligned(16))) uint16_t vb0[KTW];
    __shared__ __attribute__((aligned(16))) uint16_t vb1[KTW];
    __shared__ int pages[kPageWindow];

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 31, hl = lane >> 5;
    // work item r = ((g * tiles) + i) * G + j: KV head g, the i-th tile from
    // the end (the longest first), query head g G + j.  Each of the 8 XCDs
    // (workgroups go to XCD blockIdx % 8) takes a contiguous share of the
    // items, so the G query heads and the neighbouring tiles that stream the
    // same keys and values run together and share that XCD's L2.
    const int tiles = a.tile_start[a.B];
    const int items = tiles * a.H_q;
    const int share = (items + kXcds - 1) / kXcds;
    const int kq = (int)blockIdx.x / kXcds;
    const int r = ((int)blockIdx.x % kXcds) * share + kq;
    if (kq >= share || r >= items) return;
    const int g = r / (tiles * a.G);
    const int x = tiles - 1 - (r % (tiles * a.G)) / a.G;
    const int h = g * a.G + r % a.G;
    int lo = 0, hi = a.B - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.tile_start[mid] <= x) lo = mid;
        else hi = mid - 1;
    }
    const int b = lo;
    const int t0 = a.q_start[b];
    const int n = a.q_start[b + 1] - t0;
    const int L = a.seq_lens[b];
    const int p0 = L - n;                          // position of query token 0
    const int r0 = (x - a.tile_start[b]) * kPrefillRows;
    const int kv_end = p0 + min(r0 + kPrefillRows, n);   // keys [0, kv_end)
    const int nsteps = (kv_end + KS - 1) / KS;
    const int np = (L + kPage - 1) / kPage;
    const int32_t* bt = a.block_table + (int64_t)b * a.bt_stride;

    const int rw = r0 + 32 * w;                    // this wave's first row
    const int row = min(rw + c, n - 1);            // padding columns repeat the last row
    const int pos = p0 + row;                      // keys 0..pos are visible to this column
    const int wave_steps = rw < n ? (p0 + min(rw + 31, n - 1)) / KS + 1 : 0;

    // softmax(scale * s) = softmax(|scale| * (-s)): for a negative scale the
    // query's sign bits are flipped (the host keeps |scale| >= FLT_MIN).
    // fp8 pools: the scores are dequantised by the (request, head)'s K scale.
    float s_eff = a.scale_log2, v_scale = 1.f;
    if constexpr (FP8) {
        s_eff *= a.k_scale[(int64_t)b * a.H_kv + g];
        v_scale = a.v_scale[(int64_t)b * a.H_kv + g];
    }
    const float sl = fabsf(s_eff);
    bf16x8 qv[D / 16];
    {
        const uint32_t flip = s_eff < 0.f ? 0x80008000u : 0u;
        // the B operand of MFMA kb: dims 16 kb + 8 hl (fp8: 32 (kb / 2) + 16 hl + 8 (kb % 2))
        const uint16_t* qrow = a.q + (int64_t)(t0 + row) * a.q_st + (int64_t)h * a.q_sh + (FP8 ? 16 : 8) * hl;
#pragma unroll
        for (int kb = 0; kb < D / 16; ++kb) {
            u32x4 v = *(const u32x4*)(qrow + (FP8 ? 32 * (kb >> 1) + 8 * (kb & 1) : 16 * kb));
            v ^= flip;
            qv[kb] = __builtin_bit_cast(bf16x8, v);
        }
    }
    f32x16 o[D / 32];
#pragma unroll
    for (int t = 0; t < D / 32; ++t) o[t] = f32x16{};
    float m = -INFINITY, l = 0.f;
    bool bad = false;

    // the block-table entries of WIN steps at a time sit in LDS, refilled when
    // no copy is in flight, so a step's pages cost LDS reads only
    auto refill = [&](int j) {
        for (int e = tid; e < kPageWindow; e += 256) pages[e] = bt[min(PPS * j + e, np - 1)];
        __syncthreads();
    };
    // unit u = 256 k + tid of a step: tensor u / (PPS UPP) (K, V), page
    // (u / UPP) % PPS, 16-byte unit u % UPP of that page; a wave's 64 units
    // are consecutive and lie in one page.  K runs one step ahead of V: while
    // step s computes, K of step s + 2 and V of step s + 1 are loaded into
    // registers, and written to LDS after it.
    constexpr int PERH = PER / 2;      // units of one tensor per thread per step
    const char* kbase = (const char*)a.k_pages + (int64_t)g * PB;
    const char* vbase = (const char*)a.v_pages + (int64_t)g * PB;
    const int64_t page_bytes = (int64_t)a.H_kv * PB;
    // bf16 pools: the values come from the fp16 copy, whose pages of request
    // b are consecutive from page_off[b] (same bytes per page as bf16)
    const char* vbase16 = FP8 ? nullptr : (const char*)a.vcopy + (int64_t)g * PB;
    const int64_t vpb = FP8 ? 0 : (int64_t)a.page_off[b];
    int64_t off1[PPS], off2[PPS];      // page byte offsets of steps s + 1 and s + 2
    auto pages_of = [&](int j, int64_t (&off)[PPS]) {
        const int e = PPS * (j % WIN);
#pragma unroll
        for (int q = 0; q < PPS; ++q) {
            int pg = pages[e + q];
            if ((unsigned)pg >= (unsigned)a.num_pages) {
                pg = 0;
                bad = true;
            }
            off[q] = (int64_t)pg * page_bytes;
        }
    };
    // direct copies into LDS: lane l of a wave lands at unit (wave base + l);
    // it fetches the global unit the swizzle maps there (the swizzles are
    // involutions within a page; fp8 tiles are not swizzled)
    auto dma = [&](const char* base, const int64_t (&off)[PPS], uint16_t* dst, bool isv) {
#pragma unroll
        for (int k = 0; k < PERH; ++k) {
            int64_t o_pg;
            if constexpr (FP8) {
                const int u0 = 256 * k + 64 * w;    // this wave's 64 units: one page's units u0 % UPP ..
                const int pp = u0 / UPP;
                // page (256 k) / UPP + (w / (4 / BPP)) of the step, chosen by
                // selects on the wave's bits (no indexed access of off[],
                // which the compiler would stage through memory)
                constexpr int BPP = 256 / UPP;  // pages a round of 256 units covers: 2 (D 128) or 4 (D 64)
                const int p0k = (256 * k) / UPP;
                if constexpr (BPP == 2) {
                    o_pg = (w >> 1) ? off[p0k + 1] : off[p0k];
                } else {
                    const int64_t lo2 = (w & 1) ? off[p0k + 1] : off[p0k];
                    const int64_t hi2 = (w & 1) ? off[p0k + 3] : off[p0k + 2];
                    o_pg = (w & 2) ? hi2 : lo2;
                }
                const int v = u0 % UPP + lane;
                const int vg = (!isv && (pp & 1)) ? v ^ 4 : v;
                __builtin_amdgcn_global_load_lds(base + o_pg + vg * 16, dst + (pp * PBP + (u0 % UPP) * 16) / 2, 16, 0,
                                                 0);
                continue;
            } else {
                constexpr int BPP = 256 / UPP;
                const int pp = (256 * k) / UPP;
                o_pg = off[pp];
                if constexpr (BPP == 2) o_pg = (w >> 1) ? off[pp + 1] : o_pg;
            }
            const int v = ((256 * k + 64 * w) % UPP) + lane;          // LDS unit within its page
            const int vg = FP8 ? v : isv ? v ^ (((v >> 3) ^ (v >> 4)) & 1) : v ^ (((v >> 3) & 1) << 2);
            __builtin_amdgcn_global_load_lds(base + o_pg + vg * 16, dst + 8 * (256 * k + 64 * w), 16, 0, 0);
        }
    };
    // the fp16 value copy of step j (bf16 pools), laid out and swizzled as V;
    // a step past the request's pages re-reads its last page
    auto dma_v16 = [&](int j, uint16_t* dst) {
#pragma unroll
        for (int k = 0; k < PERH; ++k) {
            constexpr int BPP = 256 / UPP;
            const int pp = (256 * k) / UPP + (BPP == 2 ? (w >> 1) : 0);
            const int64_t o_pg = (vpb + min(PPS * j + pp, np - 1)) * page_bytes;
            const int v = ((256 * k + 64 * w) % UPP) + lane;
            const int vg = v ^ (((v >> 3) ^ (v >> 4)) & 1);
            __builtin_amdgcn_global_load_lds(vbase16 + o_pg + vg * 16, dst + 8 * (256 * k + 64 * w), 16, 0, 0);
        }
    };
    // V slots of keys >= L hold no token (NaN in a pool); P is 0 there, and
    // 0 * NaN must not reach O, so the tail step's slots are cleared
    auto clear_tail = [&](int s, uint16_t* V) {
        if constexpr (FP8) {
            // codes [page][D][16 slots], pages PBP bytes apart
            uint8_t* Vb = (uint8_t*)V;
            for (int e = tid; e < KT; e += 256) {
                const int key = KS * s + 16 * (e / PE) + (e & 15);
                if (key >= L) Vb[(e / PE) * PBP + e % PE] = 0;
            }
        } else {
            for (int e = tid; e < KT; e += 256) {
                const int d = (e % PE) >> 4;
                const int half = ((e >> 3) & 1) ^ (((d >> 2) ^ (d >> 3)) & 1);
                const int key = KS * s + 16 * (e / PE) + 8 * half + (e & 7);
                if (key >= L) V[e] = 0;
            }
        }
    };

    // lane (h, c) reads A row c = key pi(c) of each 32-key half
    const int kk = 16 * (c >> 4) + 8 * ((c >> 2) & 1) + 4 * ((c >> 3) & 1) + (c & 3);
    const int kslot = (kk & 15) ^ (((kk >> 3) & 1) << 2);
    const int k_off = (kk >> 4) * PE + hl * (kPage * 8) + kslot * 8;
    const int v_off = c * kPage + 8 * (hl ^ (((c >> 2) ^ (c >> 3)) & 1));
    // fp8 (byte offsets): the K unit (chunk 2 m + hl, slot) of key pi8(c),
    // and row c of V page hl, of each 32-key half
    const int kk8 = 16 * ((c >> 2) & 1) + 8 * ((c >> 4) & 1) + 4 * ((c >> 3) & 1) + (c & 3);
    const int k_off8 = (kk8 >> 4) * PBP + hl * 256 + ((kk8 & 15) ^ (4 * (kk8 >> 4))) * 16;
    const int v_off8 = hl * PBP + c * 16;
    // eight codes -> eight bf16, exactly
    auto widen = [](const u32x2 w8) -> bf16x8 {
        const bf16x2 p0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w8.x, 1.0f, false);
        const bf16x2 p1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w8.x, 1.0f, true);
        const bf16x2 p2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w8.y, 1.0f, false);
        const bf16x2 p3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w8.y, 1.0f, true);
        return __builtin_bit_cast(bf16x8, u32x4{__builtin_bit_cast(uint32_t, p0), __builtin_bit_cast(uint32_t, p1),
                                                __builtin_bit_cast(uint32_t, p2), __builtin_bit_cast(uint32_t, p3)});
    };
    // eight codes -> eight fp16, exactly
    auto widen16 = [](const u32x2 w8) -> f16x8 {
        const f16x2 p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w8.x, 1.0f, false);
        const f16x2 p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w8.x, 1.0f, true);
        const f16x2 p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w8.y, 1.0f, false);
        const f16x2 p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w8.y, 1.0f, true);
        return __builtin_bit_cast(f16x8, u32x4{__builtin_bit_cast(uint32_t, p0), __builtin_bit_cast(uint32_t, p1),
                                               __builtin_bit_cast(uint32_t, p2), __builtin_bit_cast(uint32_t, p3)});
    };
    auto k_operand = [&](const uint16_t* Kt, int hh, int kb) -> bf16x8 {
        return *(const bf16x8*)(Kt + k_off + hh * 2 * PE + kb * (2 * kPage * 8));
    };
    auto v_operand = [&](const uint16_t* Vt0, int hh, int u, int t) -> bf16x8 {
        return *(const bf16x8*)(Vt0 + v_off + hh * 2 * PE + (u * D + 32 * t) * kPage);
    };
    // fp8: the 16-byte unit of K pair m, and row 32 t + c of V, of half hh
    auto k_unit8 = [&](const uint16_t* Kt, int hh, int m) -> u32x4 {
        return *(const u32x4*)((const char*)Kt + hh * 2 * PBP + m * 512 + k_off8);
    };
    auto v_row8 = [&](const uint16_t* Vt0, int hh, int t) -> u32x4 {
        return *(const u32x4*)((const char*)Vt0 + hh * 2 * PBP + (32 * t) * 16 + v_off8);
    };

    auto qk = [&](const uint16_t* Kt, f32x16 (&sc)[NH]) {
#pragma unroll
        for (int hh = 0; hh < NH; ++hh) sc[hh] = f32x16{};
        if constexpr (FP8) {
#pragma unroll
            for (int m = 0; m < D / 32; ++m) {
                u32x4 ku[NH];
#pragma unroll
                for (int hh = 0; hh < NH; ++hh) ku[hh] = k_unit8(Kt, hh, m);
#pragma unroll
                for (int e = 0; e < 2; ++e)
#pragma unroll
                    for (int hh = 0; hh < NH; ++hh) {
                        const bf16x8 ka = widen(e ? u32x2{ku[hh].z, ku[hh].w} : u32x2{ku[hh].x, ku[hh].y});
                        sc[hh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qv[2 * m + e], sc[hh], 0, 0, 0);
                    }
            }
        } else {
#pragma unroll
            for (int kb = 0; kb < D / 16; ++kb)
#pragma unroll
                for (int hh = 0; hh < NH; ++hh) {
                    const bf16x8 ka = k_operand(Kt, hh, kb);
                    sc[hh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qv[kb], sc[hh], 0, 0, 0);
                }
        }
    };

    // prologue: K and V of step 0, K of step 1, S of step 0
    refill(0);
    pages_of(0, off2);
    dma(kbase, off2, kb0, false);
    if constexpr (FP8) dma(vbase, off2, vb0, true);
    else dma_v16(0, vb0);
    if (nsteps > 1) {
        pages_of(1, off1);
        dma(kbase, off1, kb1, false);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (FP8 && KS > L) {   // (the fp16 copy holds zeros past the length)
        clear_tail(0, vb0);
        __syncthreads();
    }
    f32x16 sca[NH], scb[NH];
    if (0 < wave_steps) qk(kb0, sca);
    // step 0 copies K(2) over K(0): every wave's reads of K(0) come first
    __syncthreads();

    // one step; sc holds S(s), scn receives S(s + 1)
    auto step = [&](auto par, const int s, f32x16 (&sc)[NH], f32x16 (&scn)[NH]) {
        constexpr int P = decltype(par)::value;   // s % 2
        uint16_t* k_rd = P ? kb0 : kb1;   // K(s + 1)
        uint16_t* k_wr = P ? kb1 : kb0;   // K(s + 2), over K(s)
        uint16_t* v_rd = P ? vb1 : vb0;   // V(s)
        uint16_t* v_wr = P ? vb0 : vb1;   // V(s + 1), over V(s - 1)
        const bool more_k = s + 2 < nsteps, more_v = s + 1 < nsteps;
        if (more_v) {
            if constexpr (FP8) dma(vbase, off1, v_wr, true);
            else dma_v16(s + 1, v_wr);
        }
        if (more_k) {
            if ((s + 2) % WIN == 0) refill(s + 2);
            pages_of(s + 2, off2);
            dma(kbase, off2, k_wr, false);
        }
        uint32_t ph[NH][8];   // P as fp16 pairs
        if (s < wave_steps) {
            // keys above a column's position are masked only on the steps
            // the wave's diagonal crosses
            if (KS * s + KS - 1 > p0 + rw) {
#pragma unroll
                for (int hh = 0; hh < NH; ++hh)
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        const int key = KS * s + 32 * hh + (j & 7) + (FP8 ? 16 * hl + 8 * (j >> 3) : 16 * (j >> 3) + 8 * hl);
                        sc[hh][j] = key <= pos ? sc[hh][j] : -INFINITY;
                    }
            }
            float mx = -INFINITY;
#pragma unroll
            for (int hh = 0; hh < NH; ++hh)
#pragma unroll
                for (int j = 0; j < 16; ++j) mx = fmaxf(mx, sc[hh][j]);
            mx = fmaxf(mx, swap_halves(mx));
            const float m_new = fmaxf(m, mx * sl);     // scaled units
            if (__any(m_new > m + kLazyMax)) {
                const float alpha = __builtin_amdgcn_exp2f(m - m_new);
                l *= alpha;
#pragma unroll
                for (int t = 0; t < D / 32; ++t) o[t] *= alpha;
                m = m_new;
            }
            // S of step s + 1 on the matrix cores while P of step s is formed
            // (past a wave's last step the result is not used)
            qk(k_rd, scn);
            float psum = 0.f;
#pragma unroll
            for (int hh = 0; hh < NH; ++hh)
#pragma unroll
                for (int j = 0; j < 16; j += 2) {
                    const f32x2 pq = {__builtin_amdgcn_exp2f(__builtin_fmaf(sc[hh][j], sl, -m)),
                                      __builtin_amdgcn_exp2f(__builtin_fmaf(sc[hh][j + 1], sl, -m))};
                    psum += pq.x + pq.y;
                    ph[hh][j / 2] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pq, f16x2));   // RNE
                }
            l += psum;
            // K reads run two MFMAs ahead of the S MFMAs, with the softmax
            // VALU work spread between them
            // (fp8: one K read per two MFMAs)
            constexpr int KR = FP8 ? 2 : 1;
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
            for (int i = 0; i < 8 * NH; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);        // an MFMA of S
                if (i % KR == KR - 1 && i / KR + 2 < 8 * NH / KR)
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // a K read
                __builtin_amdgcn_sched_group_barrier(0x002, kValuPerMfma, 0);   // softmax VALU
            }
            // O^T += V^T P^T, per 16-key group u of each half and 32-dim tile t
            // (bf16: group u is page u; fp8: keys 8 u .. 8 u + 7 of the
            // lane's page, both groups from one 16-byte V row)
            auto p_operand = [](const uint32_t (&p)[8], int u) {
                return __builtin_bit_cast(f16x8, u32x4{p[4 * u], p[4 * u + 1], p[4 * u + 2], p[4 * u + 3]});
            };
            if constexpr (FP8) {
#pragma unroll
                for (int hh = 0; hh < NH; ++hh)
#pragma unroll
                    for (int t = 0; t < D / 32; ++t) {
                        const u32x4 vr = v_row8(v_rd, hh, t);
#pragma unroll
                        for (int u = 0; u < 2; ++u) {
                            const f16x8 va = widen16(u ? u32x2{vr.z, vr.w} : u32x2{vr.x, vr.y});
                            o[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, p_operand(ph[hh], u), o[t], 0, 0, 0);
                        }
                    }
            } else {
#pragma unroll
                for (int hh = 0; hh < NH; ++hh)
#pragma unroll
                    for (int u = 0; u < 2; ++u) {
                        const f16x8 pa = p_operand(ph[hh], u);
#pragma unroll
                        for (int t = 0; t < D / 32; ++t) {
                            const f16x8 va = __builtin_bit_cast(f16x8, v_operand(v_rd, hh, u, t));
                            o[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, pa, o[t], 0, 0, 0);
                        }
                    }
            }
            // V reads run four MFMAs ahead of the PV MFMAs (fp8: two reads
            // ahead, each feeding two)
            constexpr int MF = FP8 ? 2 : 1;
            constexpr int NV = (FP8 ? 1 : 2) * NH * (D / 32);
            constexpr int VA = FP8 ? 2 : 4;
            __builtin_amdgcn_sched_group_barrier(0x100, VA, 0);
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, MF, 0);
                if (i + VA < NV) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
        }
        if (more_v) {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
            if (FP8 && KS * (s + 2) > L) {
                clear_tail(s + 1, v_wr);
                __syncthreads();
            }
        }
#pragma unroll
        for (int q = 0; q < PPS; ++q) off1[q] = off2[q];
    };
    // unrolled by two so that S(s) and S(s + 1) alternate between register sets
    for (int s = 0; s < nsteps; s += 2) {
        step(std::integral_constant<int, 0>{}, s, sca, scb);
        if (s + 1 < nsteps) step(std::integral_constant<int, 1>{}, s + 1, scb, sca);
    }
    if (bad && lane == 0) atomicOr(a.err, kErrPage);
    if (rw >= n) return;
    const float l_tot = l + swap_halves(l);
    // fp8: the V scale; bf16: undo the value copy's 2^e
    if constexpr (!FP8) v_scale = pow2f(-vcopy_exp(a.vmax[(int64_t)b * a.H_kv + g]));
    const float f = v_scale / l_tot;
    if (rw + c < n) {
        uint16_t* orow = a.out + (int64_t)(t0 + rw + c) * a.o_st + (int64_t)h * a.o_sh;
#pragma unroll
        for (int t = 0; t < D / 32; ++t)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const f32x2 v01 = {o[t][4 * r4] * f, o[t][4 * r4 + 1] * f};
                const f32x2 v23 = {o[t][4 * r4 + 2] * f, o[t][4 * r4 + 3] * f};
                u32x2 pk;
                pk.x = __builtin_bit_cast(uint32_t, __builtin_convertvector(v01, bf16x2));
                pk.y = __builtin_bit_cast(uint32_t, __builtin_convertvector(v23, bf16x2));
                *(u32x2*)(orow + 32 * t + 8 * r4 + 4 * hl) = pk;
            }
    }
}

}  // namespace

void launch_kv_write(const WriteArgs& a, int32_t* page_start, hipStream_t s) {
    hipLaunchKernelGGL(write_plan_kernel, dim3(1), dim3(kPlanThreads), 0, s, a, page_start);
    // an upper bound on the pages touched: ceil(n_b / 16) + 1 per request
    const unsigned items = (unsigned)(a.T / kPage + 2 * a.B + 1);
    if (a.elem_bytes == 2)
        hipLaunchKernelGGL(kv_write_kernel<2>, dim3(items, (unsigned)a.H_kv), dim3(256), 0, s, a, (const int32_t*)page_start);
    else
        hipLaunchKernelGGL(kv_write_kernel<1>, dim3(items, (unsigned)a.H_kv), dim3(256), 0, s, a, (const int32_t*)page_start);
    hipLaunchKernelGGL(lens_kernel, dim3((a.B + 255) / 256), dim3(256), 0, s, a);
}

constexpr int kHalves = 2;   // 32-key halves per step: 64 keys, four pages
void launch_prefill_prep(const PrefillArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(prefill_plan_kernel, dim3(1), dim3(kPlanThreads), 0, s, a);
    if (!a.fp8) {
        const dim3 vgrid((unsigned)a.vgrid);
        if (a.D == 128) {
            hipLaunchKernelGGL(vmax_kernel<128>, vgrid, dim3(256), 0, s, a);
        } else {
            hipLaunchKernelGGL(vmax_kernel<64>, vgrid, dim3(256), 0, s, a);
        }
        hipLaunchKernelGGL(vreduce_kernel, dim3((unsigned)(((int64_t)a.B * a.H_kv + 3) / 4)), dim3(256), 0, s, a);
        if (a.D == 128) {
            hipLaunchKernelGGL(vcopy_kernel<128>, vgrid, dim3(256), 0, s, a);
        } else {
            hipLaunchKernelGGL(vcopy_kernel<64>, vgrid, dim3(256), 0, s, a);
        }
    }
}

void launch_prefill_attn(const PrefillArgs& a, hipStream_t s) {
    // an upper bound on tiles x query heads, rounded up to whole XCD rows
    const int64_t items = ((int64_t)(a.T + kPrefillRows - 1) / kPrefillRows + a.B) * a.H_q;
    const dim3 grid((unsigned)((items + kXcds - 1) / kXcds * kXcds));
    if (a.fp8) {
        if (a.D == 128)
            hipLaunchKernelGGL((prefill_attn_kernel<128, kHalves, true>), grid, dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((prefill_attn_kernel<64, kHalves, true>), grid, dim3(256), 0, s, a);
    } else if (a.D == 128) {
        hipLaunchKernelGGL((prefill_attn_kernel<128, kHalves, false>), grid, dim3(256), 0, s, a);
    } else {
        hipLaunchKernelGGL((prefill_attn_kernel<64, kHalves, false>), grid, dim3(256), 0, s, a);
    }
}

}  // namespace bellman
