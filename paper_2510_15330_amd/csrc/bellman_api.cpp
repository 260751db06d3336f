// Host side of the C ABI: descriptor validation, the per-device workspace,
// and the launch sequence of one decode-attention call.
#include <hip/hip_runtime.h>

#include <float.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "../../include/bellman.h"
#include "internal.h"
#include "work_split.h"

using namespace bellman;

namespace {

thread_local char g_last_error[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return code;
}

// ------------------------------------------------------------- workspace ---

constexpr int kXcdSkew = 10;          // share weights 266 : 246, even : odd XCDs (measured best of 0-28)
constexpr int kXcdSkew2 = 6;          // the same with two workgroups per CU (fp8 stress batch: best of 0, 6, 12, 20)
constexpr int kMaxAttnBatch = 8192;  // lengths every attention wave reads to find its share
constexpr double kShortSharePages = 512;   // below this many table pages a wave: one page per step

// The growable per-device workspace.  Growing it allocates a larger block
// and keeps the old one alive until bellman_shutdown, so kernels already
// enqueued and graphs captured earlier still write into valid memory; no
// growth happens while the stream is being captured.
struct Workspace {
    char* base = nullptr;
    size_t cap = 0;
    std::vector<char*> retired;
};

std::mutex g_ws_mutex;
Workspace g_ws[kMaxDevices];
int g_cu_count[kMaxDevices];
int g_blocks_per_cu[kMaxDevices][2][2][5][3];  // [dev][fp8][D==128][pages per step][depth], 0 = unknown

int current_device(int* dev) {
    hipError_t e = hipGetDevice(dev);
    if (e != hipSuccess) return fail(BELLMAN_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (*dev < 0 || *dev >= kMaxDevices) return fail(BELLMAN_ERR_UNSUPPORTED, "device index %d", *dev);
    return BELLMAN_OK;
}

// Grow the current device's workspace to at least `bytes` (no region of it
// needs initialising).
int ensure_workspace(int dev, size_t bytes, hipStream_t stream, char** base) {
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    Workspace& w = g_ws[dev];
    if (bytes < kWsHeader) bytes = kWsHeader;
    if (w.cap < bytes) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        hipError_t e = hipStreamIsCapturing(stream, &cs);
        if (e != hipSuccess) return fail(BELLMAN_ERR_HIP, "hipStreamIsCapturing: %s", hipGetErrorString(e));
        if (cs != hipStreamCaptureStatusNone)
            return fail(BELLMAN_ERR_UNSUPPORTED,
                        "the workspace would have to grow to %zu bytes during graph capture; make the same call, "
                        "or bellman_reserve_workspace, before capturing", bytes);
        size_t want = bytes + bytes / 4;
        want = (want + 0xFFFFF) & ~(size_t)0xFFFFF;
        void* p = nullptr;
        e = hipMalloc(&p, want);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(BELLMAN_ERR_OOM, "workspace hipMalloc(%zu): %s", want, hipGetErrorString(e));
        }
        if (w.base) w.retired.push_back(w.base);
        w.base = (char*)p;
        w.cap = want;
    }
    *base = w.base;
    return BELLMAN_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// --------------------------------------------------------- descriptors ----

int elem_size(int32_t dt) {
    switch (dt) {
        case BELLMAN_BF16: return 2;
        case BELLMAN_FP8_E4M3FN: return 1;
        case BELLMAN_INT32: return 4;
        case BELLMAN_FP32: return 4;
        default: return 0;
    }
}

const char* dtype_name(int32_t dt) {
    switch (dt) {
        case BELLMAN_BF16: return "bf16";
        case BELLMAN_FP8_E4M3FN: return "fp8_e4m3fn";
        case BELLMAN_INT32: return "int32";
        case BELLMAN_FP32: return "fp32";
        default: return "unknown";
    }
}

int check_tensor(const bellman_tensor_t* t, const char* name, int ndim) {
    if (!t) return fail(BELLMAN_ERR_INVALID_ARG, "%s: null descriptor", name);
    if (t->ndim != ndim) return fail(BELLMAN_ERR_INVALID_ARG, "%s: expected %d dims, got %d", name, ndim, t->ndim);
    if (elem_size(t->dtype) == 0) return fail(BELLMAN_ERR_INVALID_ARG, "%s: unknown dtype %d", name, t->dtype);
    int64_t numel = 1;
    for (int i = 0; i < ndim; ++i) {
        if (t->shape[i] < 0) return fail(BELLMAN_ERR_INVALID_ARG, "%s: negative size in dim %d", name, i);
        numel *= t->shape[i];
    }
    if (numel > 0 && !t->data) return fail(BELLMAN_ERR_INVALID_ARG, "%s: null data pointer", name);
    return BELLMAN_OK;
}

int check_dtype(const bellman_tensor_t* t, const char* name, int32_t want) {
    if (t->dtype != want)
        return fail(BELLMAN_ERR_INVALID_ARG, "%s: dtype %s, expected %s", name, dtype_name(t->dtype), dtype_name(want));
    return BELLMAN_OK;
}

bool is_contiguous(const bellman_tensor_t* t) {
    int64_t expect = 1;
    for (int i = t->ndim - 1; i >= 0; --i) {
        if (t->shape[i] != 1 && t->stride[i] != expect) return false;
        expect *= t->shape[i];
    }
    return true;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

struct PoolShape {
    int64_t num_pages;
    int H_kv, D, x;
    bool fp8;
};

// K [NP, H_kv, D/x, 16, x], V [NP, H_kv, D, 16], same dtype, contiguous.
int check_pools(const bellman_tensor_t* k, const bellman_tensor_t* v, PoolShape* ps, bool need_scales) {
    int rc;
    if ((rc = check_tensor(k, "k_pages", 5))) return rc;
    if ((rc = check_tensor(v, "v_pages", 4))) return rc;
    if (k->dtype != BELLMAN_BF16 && k->dtype != BELLMAN_FP8_E4M3FN)
        return fail(BELLMAN_ERR_INVALID_ARG, "k_pages: dtype %s, expected bf16 or fp8_e4m3fn", dtype_name(k->dtype));
    if (v->dtype != k->dtype)
        return fail(BELLMAN_ERR_INVALID_ARG, "v_pages: dtype %s differs from k_pages %s", dtype_name(v->dtype),
                    dtype_name(k->dtype));
    const bool fp8 = k->dtype == BELLMAN_FP8_E4M3FN;
    const int64_t x = fp8 ? 16 : 8;
    if (k->shape[3] != kPage) return fail(BELLMAN_ERR_UNSUPPORTED, "k_pages: page size %lld, only 16 is supported", (long long)k->shape[3]);
    if (k->shape[4] != x)
        return fail(BELLMAN_ERR_INVALID_ARG, "k_pages: innermost chunk %lld, expected %lld (16 bytes)", (long long)k->shape[4], (long long)x);
    const int64_t D = k->shape[2] * x;
    if (v->shape[0] != k->shape[0] || v->shape[1] != k->shape[1] || v->shape[2] != D || v->shape[3] != kPage)
        return fail(BELLMAN_ERR_INVALID_ARG, "v_pages: shape [%lld,%lld,%lld,%lld] does not match k_pages (expected [%lld,%lld,%lld,16])",
                    (long long)v->shape[0], (long long)v->shape[1], (long long)v->shape[2], (long long)v->shape[3],
                    (long long)k->shape[0], (long long)k->shape[1], (long long)D);
    if (D != 64 && D != 128) return fail(BELLMAN_ERR_UNSUPPORTED, "head_dim %lld: only 64 and 128 are supported", (long long)D);
    if (k->shape[1] < 1) return fail(BELLMAN_ERR_INVALID_ARG, "k_pages: no KV heads");
    if (k->shape[0] < 1) return fail(BELLMAN_ERR_INVALID_ARG, "k_pages: the pool has no pages");
    if (k->shape[0] > INT32_MAX) return fail(BELLMAN_ERR_UNSUPPORTED, "more than 2^31-1 pages");
    if (!is_contiguous(k)) return fail(BELLMAN_ERR_UNSUPPORTED, "k_pages: must be contiguous");
    if (!is_contiguous(v)) return fail(BELLMAN_ERR_UNSUPPORTED, "v_pages: must be contiguous");
    if (!aligned(k->data, 16) || !aligned(v->data, 16))
        return fail(BELLMAN_ERR_UNSUPPORTED, "k_pages/v_pages: data must be 16-byte aligned");
    if (need_scales) {
        if (fp8 && (!k->dequant_scale || !v->dequant_scale))
            return fail(BELLMAN_ERR_INVALID_ARG, "fp8 pools need dequant_scale on both k_pages and v_pages");
        if (!fp8 && (k->dequant_scale || v->dequant_scale))
            return fail(BELLMAN_ERR_INVALID_ARG, "dequant_scale is only meaningful for fp8 pools");
    }
    ps->num_pages = k->shape[0];
    ps->H_kv = (int)k->shape[1];
    ps->D = (int)D;
    ps->x = (int)x;
    ps->fp8 = fp8;
    return BELLMAN_OK;
}

int check_block_table(const bellman_tensor_t* bt, int64_t B) {
    int rc;
    if ((rc = check_tensor(bt, "block_table", 2))) return rc;
    if ((rc = check_dtype(bt, "block_table", BELLMAN_INT32))) return rc;
    if (bt->shape[0] != B)
        return fail(BELLMAN_ERR_INVALID_ARG, "block_table: %lld rows for batch %lld", (long long)bt->shape[0], (long long)B);
    if (B > 0 && bt->shape[1] < 1) return fail(BELLMAN_ERR_INVALID_ARG, "block_table: no page columns");
    if (bt->shape[1] > (INT32_MAX / kPage)) return fail(BELLMAN_ERR_UNSUPPORTED, "block_table: too many columns");
    if (bt->shape[1] > 1 && bt->stride[1] != 1) return fail(BELLMAN_ERR_UNSUPPORTED, "block_table: innermost dim must be contiguous");
    if (bt->shape[0] > 1 && bt->stride[0] < bt->shape[1])
        return fail(BELLMAN_ERR_INVALID_ARG, "block_table: row stride %lld < %lld columns", (long long)bt->stride[0], (long long)bt->shape[1]);
    return BELLMAN_OK;
}

int check_seq_lens(const bellman_tensor_t* sl, int64_t B) {
    int rc;
    if ((rc = check_tensor(sl, "seq_lens", 1))) return rc;
    if ((rc = check_dtype(sl, "seq_lens", BELLMAN_INT32))) return rc;
    if (sl->shape[0] != B) return fail(BELLMAN_ERR_INVALID_ARG, "seq_lens: %lld entries for batch %lld", (long long)sl->shape[0], (long long)B);
    if (B > 1 && sl->stride[0] != 1) return fail(BELLMAN_ERR_UNSUPPORTED, "seq_lens: must be contiguous");
    return BELLMAN_OK;
}

// [B, H, D] with innermost contiguous; row strides keep 16-byte alignment.
int check_rows(const bellman_tensor_t* t, const char* name, int32_t dtype, int64_t B, int64_t H, int64_t D, size_t align) {
    int rc;
    if ((rc = check_tensor(t, name, 3))) return rc;
    if ((rc = check_dtype(t, name, dtype))) return rc;
    if (t->shape[0] != B || t->shape[1] != H || t->shape[2] != D)
        return fail(BELLMAN_ERR_INVALID_ARG, "%s: shape [%lld,%lld,%lld], expected [%lld,%lld,%lld]", name, (long long)t->shape[0],
                    (long long)t->shape[1], (long long)t->shape[2], (long long)B, (long long)H, (long long)D);
    if (t->stride[2] != 1) return fail(BELLMAN_ERR_UNSUPPORTED, "%s: innermost dim must be contiguous", name);
    const size_t eb = (size_t)elem_size(dtype);
    if (!aligned(t->data, align) || ((size_t)t->stride[0] * eb) % align || ((size_t)t->stride[1] * eb) % align)
        return fail(BELLMAN_ERR_UNSUPPORTED, "%s: rows must be %zu-byte aligned", name, align);
    return BELLMAN_OK;
}

int launch_status(const char* what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(BELLMAN_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e));
    return BELLMAN_OK;
}

// One decode-attention call.  `fixed` selects the device's fixed scratch
// array (no allocation; calls whose workspace exceeds it are rejected)
// instead of the growable library workspace.
int decode_attention(const bellman_tensor_t* q, const bellman_tensor_t* k_pages, const bellman_tensor_t* v_pages,
                     const bellman_tensor_t* block_table, const bellman_tensor_t* seq_lens, float scale,
                     bellman_tensor_t* out, const bellman_attn_opts_t* opts, void* stream, bool fixed,
                     const bellman_tensor_t* k_new = nullptr, const bellman_tensor_t* v_new = nullptr) {
    g_last_error[0] = 0;
    int rc;
    PoolShape ps;
    if ((rc = check_pools(k_pages, v_pages, &ps, true))) return rc;
    if ((rc = check_tensor(q, "q", 3))) return rc;
    const int64_t B = q->shape[0];
    const int64_t H_q = q->shape[1];
    if ((rc = check_rows(q, "q", BELLMAN_BF16, B, H_q, ps.D, 16))) return rc;
    if ((rc = check_rows(out, "out", BELLMAN_BF16, B, H_q, ps.D, 8))) return rc;
    if ((rc = check_block_table(block_table, B))) return rc;
    if ((rc = check_seq_lens(seq_lens, B))) return rc;
    if (!isfinite(scale)) return fail(BELLMAN_ERR_INVALID_ARG, "scale must be finite");
    if (H_q < 1 || H_q % ps.H_kv != 0)
        return fail(BELLMAN_ERR_INVALID_ARG, "query heads %lld not a multiple of KV heads %d", (long long)H_q, ps.H_kv);
    // decode step: the new rows, as for bellman_kv_append
    const bool step = k_new != nullptr || v_new != nullptr;
    bool quant = false;
    if (step) {
        if ((rc = check_tensor(k_new, "k_new", 3))) return rc;
        quant = ps.fp8 && k_new->dtype == BELLMAN_BF16;
        const int32_t row_dtype = quant ? (int32_t)BELLMAN_BF16 : k_pages->dtype;
        if ((rc = check_rows(k_new, "k_new", row_dtype, B, ps.H_kv, ps.D, 16))) return rc;
        if ((rc = check_rows(v_new, "v_new", row_dtype, B, ps.H_kv, ps.D, 16))) return rc;
    }
    const int64_t G = H_q / ps.H_kv;
    if (G > 16) return fail(BELLMAN_ERR_UNSUPPORTED, "GQA group %lld > 16", (long long)G);
    if (B > kMaxAttnBatch) return fail(BELLMAN_ERR_UNSUPPORTED, "batch %lld > %d", (long long)B, kMaxAttnBatch);
    const int64_t max_pages = block_table->shape[1];
    if ((double)B * ps.H_kv * (double)max_pages >= 2147483647.0)
        return fail(BELLMAN_ERR_UNSUPPORTED, "batch x KV heads x block-table width must stay below 2^31 pages");
    int max_waves = 0, pps = 0, depth = 0, skew_opt = 0;
    if (opts) {
        max_waves = opts->max_waves;
        skew_opt = opts->xcd_skew;
        pps = opts->pages_per_step;
        depth = opts->pipeline_depth;
        if (depth < 0 || depth > 2) return fail(BELLMAN_ERR_UNSUPPORTED, "pipeline_depth %d not in {0, 1, 2}", depth);
        if (max_waves < 0) return fail(BELLMAN_ERR_INVALID_ARG, "max_waves %d < 0", max_waves);
        if (pps != 0 && pps != 1 && pps != 2 && pps != 4)
            return fail(BELLMAN_ERR_UNSUPPORTED, "pages_per_step %d not in {0, 1, 2, 4}", pps);
        if (skew_opt < -1 || skew_opt > kMaxSkew)
            return fail(BELLMAN_ERR_INVALID_ARG, "xcd_skew %d not in [-1, %d]", skew_opt, kMaxSkew);
    }
    if (pps == 4 && !ps.fp8) return fail(BELLMAN_ERR_UNSUPPORTED, "pages_per_step 4 is built for fp8 pools only");
    if (depth == 0) depth = ps.fp8 ? 1 : 2;  // measured: fp8 steps compute more per byte
    if (B == 0) return BELLMAN_OK;

    int dev;
    if ((rc = current_device(&dev))) return rc;
    if (g_cu_count[dev] == 0) {
        int cu = 0;
        hipError_t e = hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess || cu < 1) return fail(BELLMAN_ERR_HIP, "multiprocessor count: %s", hipGetErrorString(e));
        g_cu_count[dev] = cu;
    }
    if (pps == 0) {
        // bf16: two pages per step, or one when the block table leaves room
        // for few pages per wave (short shares: the finer step shortens the
        // ramp and the tail; measured 121 against 126 us on 64 requests of
        // 1-4k tokens, while 256 requests of 6-13.5k tokens run faster with
        // two).  Decided from the table's width, so no device read is needed.
        int64_t w_est = (int64_t)g_cu_count[dev] * (kAttnBlock / kWaveSize) * (depth == 2 ? 1 : 2);
        if (max_waves > 0 && w_est > max_waves) w_est = max_waves;
        const double table_pages_per_wave = (double)B * ps.H_kv * (double)max_pages / (double)w_est;
        pps = ps.fp8 ? 4 : (table_pages_per_wave < kShortSharePages ? 1 : 2);
    }
    if (step && !attention_step_built(pps, depth, ps.fp8))
        return fail(BELLMAN_ERR_UNSUPPORTED,
                    "decode step: built for the default steps only (bf16: 1 or 2 pages, depth 2; fp8: 4 pages, "
                    "depth 1)");
    int64_t* wave_times = opts ? opts->wave_times : nullptr;
    if (step && wave_times) return fail(BELLMAN_ERR_UNSUPPORTED, "decode step: wave_times is not built for it");
    if (wave_times && !attention_traced(pps, depth, ps.fp8, ps.D))
        return fail(BELLMAN_ERR_UNSUPPORTED,
                    "wave_times: traced kernels are built for head_dim 128 at the default steps only");
    if (wave_times && !aligned(wave_times, 8)) return fail(BELLMAN_ERR_UNSUPPORTED, "wave_times must be 8-byte aligned");
    int& bpc = g_blocks_per_cu[dev][ps.fp8][ps.D == 128][pps][depth];
    if (bpc == 0) {
        bpc = attention_blocks_per_cu(pps, depth, ps.fp8, ps.D);
        if (depth == 2) bpc = 1;  // one wavefront per SIMD
    }
    // Every resident wave takes an equal share of the flattened step stream.
    int64_t waves = (int64_t)g_cu_count[dev] * bpc * (kAttnBlock / kWaveSize);
    if (max_waves > 0 && waves > max_waves) waves = max_waves;
    const int64_t grid = (waves + (kAttnBlock / kWaveSize) - 1) / (kAttnBlock / kWaveSize);

    if (waves > kMaxWaves) return fail(BELLMAN_ERR_UNSUPPORTED, "%lld waves > %d", (long long)waves, kMaxWaves);
    // two partial slots per wave and query head: a wave's range cuts at most
    // the request it starts in and the one it ends in
    const size_t off_cuts = kWsHeader;
    const size_t off_ml = off_cuts + align256(sizeof(int4) * (size_t)waves);
    const size_t slots = 2 * (size_t)waves * (size_t)G;
    const size_t off_o = off_ml + align256(sizeof(float2) * slots);
    const size_t total = off_o + align256(sizeof(float) * slots * (size_t)ps.D);
    hipStream_t s = (hipStream_t)stream;
    char* base;
    if (fixed) {
        if (total > kScratchBytes)
            return fail(BELLMAN_ERR_UNSUPPORTED,
                        "this call needs %zu bytes of scratch; the fixed scratch array holds %zu "
                        "(2 * waves * G partial slots of %zu bytes)",
                        total, kScratchBytes, sizeof(float2) + sizeof(float) * (size_t)ps.D);
        if ((rc = device_scratch(dev, &base))) return rc;
    } else if ((rc = ensure_workspace(dev, total, s, &base))) {
        return rc;
    }
    int32_t* err;
    if ((rc = device_error_word(dev, &err))) return rc;

    AttnArgs a;
    a.q = (const uint16_t*)q->data;
    a.q_sb = q->stride[0];
    a.q_sh = q->stride[1];
    a.k_pages = k_pages->data;
    a.v_pages = v_pages->data;
    a.k_scale = k_pages->dequant_scale;
    a.v_scale = v_pages->dequant_scale;
    a.block_table = (const int32_t*)block_table->data;
    a.bt_stride = B > 1 ? block_table->stride[0] : max_pages;
    a.seq_lens = (const int32_t*)seq_lens->data;
    a.out = (uint16_t*)out->data;
    a.o_sb = out->stride[0];
    a.o_sh = out->stride[1];
    a.num_pages = ps.num_pages;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.B = (int)B;
    a.H_q = (int)H_q;
    a.H_kv = ps.H_kv;
    a.G = (int)G;
    a.D = ps.D;
    a.max_pages = (int)max_pages;
    a.waves = (int)waves;
    a.pp = pps;
    // The default XCD weights were measured on a whole MI355X (256 CUs,
    // workgroup i on XCD i mod 8), with one and with two workgroups per CU;
    // partitioned devices keep equal shares.
    if (skew_opt == 0) a.skew = g_cu_count[dev] == 256 ? (bpc == 1 ? kXcdSkew : kXcdSkew2) : 0;
    else a.skew = skew_opt < 0 ? 0 : skew_opt;
    a.err = err;
    a.cuts = (int4*)(base + off_cuts);
    a.part_ml = (float2*)(base + off_ml);
    a.part_o = (float*)(base + off_o);
    a.wave_times = wave_times;
    a.k_new = step ? k_new->data : nullptr;
    a.v_new = step ? v_new->data : nullptr;
    a.new_sb = step ? k_new->stride[0] : 0;
    a.new_sh = step ? k_new->stride[1] : 0;
    a.vnew_sb = step ? v_new->stride[0] : 0;
    a.vnew_sh = step ? v_new->stride[1] : 0;
    a.quant = quant ? 1 : 0;
    a.lens_rw = step ? (int32_t*)seq_lens->data : nullptr;

    hipEvent_t ev0 = opts ? (hipEvent_t)opts->event_begin : nullptr;
    hipEvent_t ev1 = opts ? (hipEvent_t)opts->event_end : nullptr;
    if (ev0) {
        hipError_t e = hipEventRecord(ev0, s);
        if (e != hipSuccess) return fail(BELLMAN_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    launch_attention(a, pps, depth, ps.fp8, (int)grid, s);
    if ((rc = launch_status("attention"))) return rc;
    if (ev1) {
        hipError_t e = hipEventRecord(ev1, s);
        if (e != hipSuccess) return fail(BELLMAN_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    launch_merge(a, s);
    return launch_status("merge");
}

}  // namespace

namespace bellman {
int set_error(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return code;
}
}  // namespace bellman

// ================================================================== ABI ====

extern "C" {

const char* bellman_last_error(void) { return g_last_error; }

const char* bellman_version(void) { return "0.1.0"; }

int bellman_reserve_workspace(int64_t bytes) {
    g_last_error[0] = 0;
    if (bytes < 0) return fail(BELLMAN_ERR_INVALID_ARG, "negative workspace size");
    int dev, rc;
    if ((rc = current_device(&dev))) return rc;
    char* base;
    return ensure_workspace(dev, (size_t)bytes, nullptr, &base);
}

void bellman_shutdown(void) {
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    int cur = 0;
    (void)hipGetDevice(&cur);
    for (int d = 0; d < kMaxDevices; ++d) {
        Workspace& w = g_ws[d];
        if (!w.base && w.retired.empty()) continue;
        (void)hipSetDevice(d);
        (void)hipDeviceSynchronize();
        for (char* p : w.retired) (void)hipFree(p);
        w.retired.clear();
        if (w.base) (void)hipFree(w.base);
        w.base = nullptr;
        w.cap = 0;
    }
    (void)hipSetDevice(cur);
}

int bellman_device_errors(void* stream, int32_t* flags) {
    g_last_error[0] = 0;
    if (!flags) return fail(BELLMAN_ERR_INVALID_ARG, "flags: null pointer");
    int dev, rc;
    if ((rc = current_device(&dev))) return rc;
    int32_t* err;
    if ((rc = device_error_word(dev, &err))) return rc;
    hipStream_t s = (hipStream_t)stream;
    int32_t v = 0;
    hipError_t e = hipMemcpyAsync(&v, err, sizeof v, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e == hipSuccess) e = hipMemsetAsync(err, 0, sizeof v, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(BELLMAN_ERR_HIP, "reading the device error word: %s", hipGetErrorString(e));
    *flags = v;
    return BELLMAN_OK;
}

int bellman_kv_append(const bellman_tensor_t* k_new, const bellman_tensor_t* v_new, bellman_tensor_t* k_pages,
                      bellman_tensor_t* v_pages, const bellman_tensor_t* block_table, bellman_tensor_t* seq_lens,
                      void* stream) {
    g_last_error[0] = 0;
    int rc;
    PoolShape ps;
    if ((rc = check_pools(k_pages, v_pages, &ps, false))) return rc;
    if ((rc = check_tensor(k_new, "k_new", 3))) return rc;
    const int64_t B = k_new->shape[0];
    // bf16 rows into fp8 pools are quantised with the pools' dequant scales
    const bool quant = ps.fp8 && k_new->dtype == BELLMAN_BF16;
    const int32_t row_dtype = quant ? (int32_t)BELLMAN_BF16 : k_pages->dtype;
    if ((rc = check_rows(k_new, "k_new", row_dtype, B, ps.H_kv, ps.D, 16))) return rc;
    if ((rc = check_rows(v_new, "v_new", row_dtype, B, ps.H_kv, ps.D, 16))) return rc;
    if ((rc = check_block_table(block_table, B))) return rc;
    if ((rc = check_seq_lens(seq_lens, B))) return rc;
    if (quant && (!k_pages->dequant_scale || !v_pages->dequant_scale))
        return fail(BELLMAN_ERR_INVALID_ARG, "quantising bf16 rows into fp8 pools needs dequant_scale on both pools");
    if (B > INT32_MAX) return fail(BELLMAN_ERR_UNSUPPORTED, "batch too large");
    if (B == 0) return BELLMAN_OK;

    int dev;
    if ((rc = current_device(&dev))) return rc;
    int32_t* err;
    if ((rc = device_error_word(dev, &err))) return rc;

    AppendArgs a;
    a.k_new = k_new->data;
    a.v_new = v_new->data;
    a.new_sb = k_new->stride[0];
    a.new_sh = k_new->stride[1];
    a.vnew_sb = v_new->stride[0];
    a.vnew_sh = v_new->stride[1];
    a.k_pages = k_pages->data;
    a.v_pages = v_pages->data;
    a.block_table = (const int32_t*)block_table->data;
    a.bt_stride = block_table->shape[0] > 1 ? block_table->stride[0] : block_table->shape[1];
    a.seq_lens = (int32_t*)seq_lens->data;
    a.err = err;
    a.num_pages = ps.num_pages;
    a.k_scale = k_pages->dequant_scale;
    a.v_scale = v_pages->dequant_scale;
    a.B = (int)B;
    a.H_kv = ps.H_kv;
    a.D = ps.D;
    a.max_pages = (int)block_table->shape[1];
    a.elem_bytes = ps.fp8 ? 1 : 2;
    a.quant = quant ? 1 : 0;
    launch_kv_append(a, (hipStream_t)stream);
    return launch_status("kv_append");
}

int bellman_probe_gather(const void* pool, int64_t pool_bytes, int32_t tile_bytes, int32_t max_waves, uint32_t* sink,
                         void* stream) {
    g_last_error[0] = 0;
    if (!pool || !sink) return fail(BELLMAN_ERR_INVALID_ARG, "pool and sink must be device pointers");
    if (tile_bytes != 2048 && tile_bytes != 4096 && tile_bytes != 8192)
        return fail(BELLMAN_ERR_UNSUPPORTED, "tile_bytes %d not in {2048, 4096, 8192}", tile_bytes);
    if (pool_bytes < tile_bytes || pool_bytes % tile_bytes)
        return fail(BELLMAN_ERR_INVALID_ARG, "pool_bytes %lld is not a positive multiple of tile_bytes",
                    (long long)pool_bytes);
    const int64_t n = pool_bytes / tile_bytes;
    if (n & (n - 1)) return fail(BELLMAN_ERR_INVALID_ARG, "pool_bytes / tile_bytes = %lld is not a power of two",
                                 (long long)n);
    if (!aligned(pool, 16) || !aligned(sink, 4))
        return fail(BELLMAN_ERR_UNSUPPORTED, "pool must be 16-byte and sink 4-byte aligned");
    if (max_waves < 0) return fail(BELLMAN_ERR_INVALID_ARG, "max_waves %d < 0", max_waves);
    int dev, rc;
    if ((rc = current_device(&dev))) return rc;
    int cu = 0;
    hipError_t e = hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess || cu < 1) return fail(BELLMAN_ERR_HIP, "multiprocessor count: %s", hipGetErrorString(e));
    int64_t waves = (int64_t)cu * gather_probe_blocks_per_cu(tile_bytes) * 4;
    if (max_waves > 0 && waves > max_waves) waves = max_waves;
    if (waves > n) waves = n;
    launch_gather_probe(pool, n, tile_bytes, (int)waves, sink, (hipStream_t)stream);
    return launch_status("gather probe");
}

int bellman_decode_attention_opts(const bellman_tensor_t* q, const bellman_tensor_t* k_pages,
                                  const bellman_tensor_t* v_pages, const bellman_tensor_t* block_table,
                                  const bellman_tensor_t* seq_lens, float scale, bellman_tensor_t* out,
                                  const bellman_attn_opts_t* opts, void* stream) {
    return decode_attention(q, k_pages, v_pages, block_table, seq_lens, scale, out, opts, stream, false);
}

int bellman_decode_attention(const bellman_tensor_t* q, const bellman_tensor_t* k_pages, const bellman_tensor_t* v_pages,
                             const bellman_tensor_t* block_table, const bellman_tensor_t* seq_lens, float scale,
                             bellman_tensor_t* out, void* stream) {
    return decode_attention(q, k_pages, v_pages, block_table, seq_lens, scale, out, nullptr, stream, false);
}

int bellman_decode_attention_noalloc(const bellman_tensor_t* q, const bellman_tensor_t* k_pages,
                                     const bellman_tensor_t* v_pages, const bellman_tensor_t* block_table,
                                     const bellman_tensor_t* seq_lens, float scale, bellman_tensor_t* out,
                                     const bellman_attn_opts_t* opts, void* stream) {
    return decode_attention(q, k_pages, v_pages, block_table, seq_lens, scale, out, opts, stream, true);
}

int bellman_decode_step(const bellman_tensor_t* k_new, const bellman_tensor_t* v_new, const bellman_tensor_t* q,
                        bellman_tensor_t* k_pages, bellman_tensor_t* v_pages, const bellman_tensor_t* block_table,
                        bellman_tensor_t* seq_lens, float scale, bellman_tensor_t* out,
                        const bellman_attn_opts_t* opts, void* stream) {
    g_last_error[0] = 0;
    if (!k_new || !v_new) return fail(BELLMAN_ERR_INVALID_ARG, "k_new and v_new are required");
    return decode_attention(q, k_pages, v_pages, block_table, seq_lens, scale, out, opts, stream, false, k_new, v_new);
}

// ------------------------------------------------------------ prompt path --

namespace {
int check_q_start(const bellman_tensor_t* qs, int64_t B) {
    int rc;
    if ((rc = check_tensor(qs, "q_start", 1))) return rc;
    if ((rc = check_dtype(qs, "q_start", BELLMAN_INT32))) return rc;
    if (qs->shape[0] != B + 1)
        return fail(BELLMAN_ERR_INVALID_ARG, "q_start: %lld entries for batch %lld (need B + 1)", (long long)qs->shape[0],
                    (long long)B);
    if (qs->shape[0] > 1 && qs->stride[0] != 1) return fail(BELLMAN_ERR_UNSUPPORTED, "q_start: must be contiguous");
    return BELLMAN_OK;
}
}  // namespace

int bellman_kv_write(const bellman_tensor_t* k_new, const bellman_tensor_t* v_new, bellman_tensor_t* k_pages,
                     bellman_tensor_t* v_pages, const bellman_tensor_t* block_table, bellman_tensor_t* seq_lens,
                     const bellman_tensor_t* q_start, void* stream) {
    g_last_error[0] = 0;
    int rc;
    PoolShape ps;
    if ((rc = check_pools(k_pages, v_pages, &ps, false))) return rc;
    if ((rc = check_tensor(k_new, "k_new", 3))) return rc;
    const int64_t T = k_new->shape[0];
    const size_t eb = ps.fp8 ? 1 : 2;
    if ((rc = check_rows(k_new, "k_new", k_pages->dtype, T, ps.H_kv, ps.D, 16))) return rc;
    if ((rc = check_rows(v_new, "v_new", k_pages->dtype, T, ps.H_kv, ps.D, 16))) return rc;
    if ((rc = check_seq_lens(seq_lens, seq_lens ? seq_lens->shape[0] : 0))) return rc;
    const int64_t B = seq_lens->shape[0];
    if ((rc = check_block_table(block_table, B))) return rc;
    if ((rc = check_q_start(q_start, B))) return rc;
    if (T > INT32_MAX || B > INT32_MAX) return fail(BELLMAN_ERR_UNSUPPORTED, "too many tokens or requests");
    if (T == 0 || B == 0) return BELLMAN_OK;

    if (T / 16 + 2 * B + 1 > (int64_t)UINT32_MAX) return fail(BELLMAN_ERR_UNSUPPORTED, "too many tokens or requests");

    int dev;
    if ((rc = current_device(&dev))) return rc;
    char* base;
    if ((rc = ensure_workspace(dev, kWsHeader + align256((size_t)(B + 1) * 4), (hipStream_t)stream, &base)))
        return rc;
    int32_t* err;
    if ((rc = device_error_word(dev, &err))) return rc;
    WriteArgs a;
    a.k_new = k_new->data;
    a.v_new = v_new->data;
    a.k_st = k_new->stride[0];
    a.k_sh = k_new->stride[1];
    a.v_st = v_new->stride[0];
    a.v_sh = v_new->stride[1];
    a.k_pages = k_pages->data;
    a.v_pages = v_pages->data;
    a.block_table = (const int32_t*)block_table->data;
    a.bt_stride = block_table->shape[0] > 1 ? block_table->stride[0] : block_table->shape[1];
    a.seq_lens = (int32_t*)seq_lens->data;
    a.q_start = (const int32_t*)q_start->data;
    a.err = err;
    a.num_pages = ps.num_pages;
    a.B = (int)B;
    a.T = (int)T;
    a.H_kv = ps.H_kv;
    a.D = ps.D;
    a.max_pages = (int)block_table->shape[1];
    a.elem_bytes = (int)eb;
    launch_kv_write(a, (int32_t*)(base + kWsHeader), (hipStream_t)stream);
    return launch_status("kv_write");
}

int bellman_prefill_attention_opts(const bellman_tensor_t* q, const bellman_tensor_t* k_pages,
                                   const bellman_tensor_t* v_pages, const bellman_tensor_t* block_table,
                                   const bellman_tensor_t* seq_lens, const bellman_tensor_t* q_start, float scale,
                                   bellman_tensor_t* out, const bellman_prefill_opts_t* opts, void* stream) {
    g_last_error[0] = 0;
    int rc;
    PoolShape ps;
    if ((rc = check_pools(k_pages, v_pages, &ps, true))) return rc;
    if ((rc = check_tensor(q, "q", 3))) return rc;
    const int64_t T = q->shape[0];
    const int64_t H_q = q->shape[1];
    if ((rc = check_rows(q, "q", BELLMAN_BF16, T, H_q, ps.D, 16))) return rc;
    if ((rc = check_rows(out, "out", BELLMAN_BF16, T, H_q, ps.D, 8))) return rc;
    if ((rc = check_seq_lens(seq_lens, seq_lens ? seq_lens->shape[0] : 0))) return rc;
    const int64_t B = seq_lens->shape[0];
    if ((rc = check_block_table(block_table, B))) return rc;
    if ((rc = check_q_start(q_start, B))) return rc;
    if (!isfinite(scale)) return fail(BELLMAN_ERR_INVALID_ARG, "scale must be finite");
    if (H_q < 1 || H_q % ps.H_kv != 0)
        return fail(BELLMAN_ERR_INVALID_ARG, "query heads %lld not a multiple of KV heads %d", (long long)H_q, ps.H_kv);
    if (H_q > 65535) return fail(BELLMAN_ERR_UNSUPPORTED, "more than 65535 query heads");
    if (T > INT32_MAX / 2 || B > INT32_MAX / 2) return fail(BELLMAN_ERR_UNSUPPORTED, "too many tokens or requests");
    // tiles x query heads must fit the kernel's 32-bit work index
    if (((T + kPrefillRows - 1) / kPrefillRows + B) * H_q > INT32_MAX / 2)
        return fail(BELLMAN_ERR_UNSUPPORTED, "too many query tiles x heads");
    if (T == 0 || B == 0) return BELLMAN_OK;

    // bf16 pools: the fp16 copy of the values holds at most every table page
    // of every request (B x maxP pages of H_kv heads)
    const int64_t max_pages = block_table->shape[1];
    const size_t page_head_bytes = (size_t)ps.D * 16 * 2;
    if (!ps.fp8 && (double)B * (double)max_pages >= 2147483647.0)
        return fail(BELLMAN_ERR_UNSUPPORTED, "batch x block-table width must stay below 2^31 pages");
    const size_t copy_bytes = ps.fp8 ? 0 : (size_t)B * (size_t)max_pages * (size_t)ps.H_kv * page_head_bytes;
    if (!ps.fp8 && (double)B * (double)max_pages * ps.H_kv * (double)page_head_bytes > 1099511627776.0)
        return fail(BELLMAN_ERR_UNSUPPORTED, "the fp16 value copy of B x maxP pages would exceed 1 TiB");
    const size_t off_tiles = kWsHeader;
    const size_t off_pages = off_tiles + align256((size_t)(B + 1) * 4);
    const size_t off_req = off_pages + align256((size_t)(B + 1) * 4);
    const size_t off_tmax = off_req + align256(ps.fp8 ? 0 : (size_t)B * (size_t)max_pages * 4);
    const size_t off_vmax = off_tmax + align256(ps.fp8 ? 0 : (size_t)B * (size_t)max_pages * ps.H_kv * 4);
    const size_t off_copy = off_vmax + align256((size_t)B * ps.H_kv * 4);
    const size_t total = off_copy + align256(copy_bytes);

    int dev;
    if ((rc = current_device(&dev))) return rc;
    hipStream_t s = (hipStream_t)stream;
    char* base;
    if ((rc = ensure_workspace(dev, total, s, &base))) return rc;
    int32_t* err;
    if ((rc = device_error_word(dev, &err))) return rc;
    PrefillArgs a;
    a.q = (const uint16_t*)q->data;
    a.q_st = q->stride[0];
    a.q_sh = q->stride[1];
    a.k_pages = k_pages->data;
    a.v_pages = v_pages->data;
    a.block_table = (const int32_t*)block_table->data;
    a.bt_stride = block_table->shape[0] > 1 ? block_table->stride[0] : block_table->shape[1];
    a.seq_lens = (const int32_t*)seq_lens->data;
    a.q_start = (const int32_t*)q_start->data;
    a.out = (uint16_t*)out->data;
    a.o_st = out->stride[0];
    a.o_sh = out->stride[1];
    a.num_pages = ps.num_pages;
    // the kernel takes |scale| (with the query's sign flipped for a negative
    // one) and needs it nonzero; a zero scale becomes the smallest normal
    a.scale_log2 = scale * 1.4426950408889634f;
    if (fabsf(a.scale_log2) < FLT_MIN) a.scale_log2 = copysignf(FLT_MIN, a.scale_log2);
    a.B = (int)B;
    a.T = (int)T;
    a.H_q = (int)H_q;
    a.H_kv = ps.H_kv;
    a.G = (int)(H_q / ps.H_kv);
    a.D = ps.D;
    a.max_pages = (int)max_pages;
    a.err = err;
    a.tile_start = (int32_t*)(base + off_tiles);
    a.fp8 = ps.fp8 ? 1 : 0;
    a.k_scale = k_pages->dequant_scale;
    a.v_scale = v_pages->dequant_scale;
    a.page_off = (int32_t*)(base + off_pages);
    a.page_req = (int32_t*)(base + off_req);
    a.tmax = (float*)(base + off_tmax);
    a.vmax = (uint32_t*)(base + off_vmax);
    a.vcopy = (uint16_t*)(base + off_copy);
    // enough waves for every (page, head) tile of B x maxP pages at most
    // once, and at most 2048 workgroups
    a.vgrid = (int)std::max<int64_t>(1, std::min<int64_t>(2048, ((int64_t)B * max_pages * ps.H_kv + 3) / 4));
    launch_prefill_prep(a, s);
    if ((rc = launch_status("prefill_attention (planning)"))) return rc;
    if (opts && opts->event_begin) {
        hipError_t e = hipEventRecord((hipEvent_t)opts->event_begin, s);
        if (e != hipSuccess) return fail(BELLMAN_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    launch_prefill_attn(a, s);
    if ((rc = launch_status("prefill_attention"))) return rc;
    if (opts && opts->event_end) {
        hipError_t e = hipEventRecord((hipEvent_t)opts->event_end, s);
        if (e != hipSuccess) return fail(BELLMAN_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    return BELLMAN_OK;
}

int bellman_prefill_attention(const bellman_tensor_t* q, const bellman_tensor_t* k_pages,
                              const bellman_tensor_t* v_pages, const bellman_tensor_t* block_table,
                              const bellman_tensor_t* seq_lens, const bellman_tensor_t* q_start, float scale,
                              bellman_tensor_t* out, void* stream) {
    return bellman_prefill_attention_opts(q, k_pages, v_pages, block_table, seq_lens, q_start, scale, out, nullptr,
                                          stream);
}

}  // extern "C"
