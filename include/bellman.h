/*
 * libbellman — batched paged decode attention for MI355X (gfx950), with the
 * KV append that feeds it and the host-side output-length controller of
 * beLLMan ("beLLMan: Controlling LLM Congestion", arXiv 2510.15330).
 *
 * The paper (Sec. 3) serves requests through a batching scheduler whose
 * per-token decode latency (TBT) it watches; each decode step attends one new
 * query token per request over that request's KV cache, whose length is the
 * prompt plus the tokens generated so far, and the controller caps each
 * request's output length under load.  This library provides that decode
 * step and the controller.
 *
 * Conventions for every call below
 *  - Tensors are described by bellman_tensor_t: a data pointer, an element
 *    type, a shape and strides in elements.  Device tensors are memory the
 *    caller allocated on the current HIP device; the library never frees,
 *    reallocates or retains them after the call returns.
 *  - stream is a hipStream_t (NULL = the device's null stream).  Every
 *    device call only enqueues work on it and returns without synchronising.
 *  - Return value: 0 on success, otherwise a negative bellman_status_t; the
 *    reason is in bellman_last_error() (per thread).  Arguments are checked
 *    on the host from the descriptors alone, before any HIP call; the call
 *    then enqueues nothing.  Device contents (lengths, block-table entries)
 *    cannot be checked on the host without a sync; the kernels bound-check
 *    them, skip any slot or page outside the pool, and record the violation
 *    in a per-device error word read by bellman_device_errors().  Faults of
 *    the GPU surface at the caller's next synchronisation.
 *  - No C++ exception crosses this interface.
 *
 * Paged KV layout (both pools hold whole 16-token pages; page p of head g is
 * one contiguous tile):
 *    K pool  [NP, H_kv, D/x, 16, x]   x = 16 bytes / element size
 *            (8 for bf16, 16 for fp8): for each page and head, the keys are
 *            stored as D/x chunks of x consecutive dims, each chunk holding
 *            all 16 slots.
 *    V pool  [NP, H_kv, D, 16]        values stored dim-major: for each
 *            page, head and dim, the 16 slots are consecutive.
 *  Token t of request b lives in page block_table[b][t / 16], slot t % 16.
 *  Element types: bf16, or OCP fp8 e4m3fn with one fp32 dequantisation
 *  scale per (request, KV head) for K and one for V (real value =
 *  e4m3fn(code) * scale).  Supported: head_dim D in {64, 128}; H_q a
 *  multiple of H_kv with G = H_q / H_kv <= 16; query head h reads KV head
 *  h / G.
 */
#ifndef BELLMAN_H
#define BELLMAN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum bellman_status {
    BELLMAN_OK = 0,
    BELLMAN_ERR_INVALID_ARG = -1,  /* null pointer, bad shape/stride/dtype, non-finite scale */
    BELLMAN_ERR_UNSUPPORTED = -2,  /* well-formed but outside what the kernels implement */
    BELLMAN_ERR_HIP = -3,          /* a HIP runtime call or kernel launch failed */
    BELLMAN_ERR_OOM = -4           /* workspace allocation failed */
} bellman_status_t;

typedef enum bellman_dtype {
    BELLMAN_BF16 = 1,
    BELLMAN_FP8_E4M3FN = 2,
    BELLMAN_INT32 = 3,
    BELLMAN_FP32 = 4
} bellman_dtype_t;

#define BELLMAN_MAX_DIMS 5
#define BELLMAN_PAGE_TOKENS 16

typedef struct bellman_tensor {
    void *data;                       /* device pointer */
    int32_t dtype;                    /* bellman_dtype_t */
    int32_t ndim;                     /* used entries of shape/stride */
    int64_t shape[BELLMAN_MAX_DIMS];
    int64_t stride[BELLMAN_MAX_DIMS]; /* in elements */
    const float *dequant_scale;       /* fp8 K/V pools only: device fp32 [B, H_kv],
                                         contiguous; NULL otherwise */
} bellman_tensor_t;

/*
 * Append one token per request to the paged KV cache (the step that grows
 * each request's KV length by one token per decode step, Sec. 3).
 *   k_new, v_new  [B, H_kv, D], innermost dim contiguous, rows 16-byte
 *                 aligned.  Either the
 *                 pools' element type (codes copied as they are), or bf16
 *                 rows for fp8 pools: then each value x of KV head g is
 *                 stored as e4m3fn(x / scale[b, g]) with the pool's
 *                 dequant_scale (K's for k_new, V's for v_new), the quotient
 *                 one correctly rounded binary32 division, rounded to
 *                 nearest with ties to the even mantissa, saturating at
 *                 +-448, NaN kept.
 *   k_pages       [NP, H_kv, D/x, 16, x] contiguous (written).
 *   v_pages       [NP, H_kv, D, 16] contiguous (written).
 *   block_table   int32 [B, maxP], innermost contiguous; the page that will
 *                 receive the token must already be assigned.
 *   seq_lens      int32 [B] contiguous, read and written: the token of
 *                 request b goes to position L = seq_lens[b]
 *                 (page block_table[b][L/16], slot L%16), then seq_lens[b]
 *                 becomes L + 1.
 * The write is bit-exact (a byte copy, or the quantisation above) and
 * changes nothing else: the bytes around the new slot that share a 32-byte
 * sector with it (the neighbouring slot's K chunk, the rest of each V dim
 * row) are read and written back unchanged, so that every sector is written
 * whole.  Hence no two requests of one call may append into the same page.
 * A request whose slot lies outside the block table or the pool is skipped
 * (no byte written, length unchanged) and flagged in the device error word.
 */
int bellman_kv_append(const bellman_tensor_t *k_new, const bellman_tensor_t *v_new,
                      bellman_tensor_t *k_pages, bellman_tensor_t *v_pages,
                      const bellman_tensor_t *block_table, bellman_tensor_t *seq_lens,
                      void *stream);

/*
 * Decode attention for one step: for request b and query head h,
 *   out[b,h,:] = sum_t softmax_t(scale * <q[b,h,:], k_t>) * v_t,  t < seq_lens[b]
 * over the request's KV pages (query head h uses KV head h / G).
 *   q            bf16 [B, H_q, D], innermost contiguous.
 *   k_pages      [NP, H_kv, D/x, 16, x] contiguous, bf16 or fp8 (with
 *                dequant_scale set).
 *   v_pages      [NP, H_kv, D, 16] contiguous, same element type.
 *   block_table  int32 [B, maxP], innermost contiguous.
 *   seq_lens     int32 [B]: attention lengths (after this step's append).
 *   scale        finite fp32 softmax scale (usually 1/sqrt(D)).
 *   out          bf16 [B, H_q, D], innermost contiguous (written; rounded to
 *                nearest even).  A request of length 0 gets zeros.
 * The work of the batch, as (request, KV head, step of consecutive pages)
 * units, is dealt to the GPU's resident wavefronts in equal contiguous
 * shares; a request cut by a share boundary has its partial softmax
 * statistics merged in a second pass.  The shares are planned on the device,
 * so the call never waits for the GPU.
 * Limits: B <= 8192 and B * H_kv * maxP < 2^31.  Scratch memory is a
 * per-device library workspace (partial results of the cut requests),
 * grown on demand (hipMalloc) and released by bellman_shutdown(); calls on
 * different streams of one device must not overlap in time.  Growing
 * allocates a larger block and keeps the previous one until
 * bellman_shutdown(), so work already enqueued and HIP graphs captured
 * earlier keep valid scratch; a call that would have to grow the workspace
 * while its stream is being captured fails with BELLMAN_ERR_UNSUPPORTED
 * (make the same call, or bellman_reserve_workspace, before capturing).
 * Once the workspace has grown to a call's size, the call enqueues only
 * kernels on `stream`: no memset, copy or host wait, so it can be captured
 * in a HIP graph and replayed.
 */
int bellman_decode_attention(const bellman_tensor_t *q, const bellman_tensor_t *k_pages,
                             const bellman_tensor_t *v_pages,
                             const bellman_tensor_t *block_table,
                             const bellman_tensor_t *seq_lens, float scale,
                             bellman_tensor_t *out, void *stream);

typedef struct bellman_attn_opts {
    int32_t max_waves;    /* cap on the waves that share the work; 0 = every wave the
                             GPU can keep resident.  Fewer waves split fewer
                             requests (results agree within rounding). */
    int32_t xcd_skew;     /* share weights of the waves of even- and odd-numbered
                             XCDs (workgroup i runs on XCD i mod 8), applied only
                             when every wave gets at least 384 pages (steps x
                             pages per step):
                             0 = the library's choice (on a whole 256-CU device
                             k = 10 with one workgroup per CU, k = 6 with two;
                             equal shares otherwise); -1 = equal shares; k in
                             1..255 = weights 256 + k : 256 - k.  Results agree
                             within rounding. */
    int32_t pages_per_step; /* 16-token pages per softmax update: 1 or 2 (bf16),
                               1, 2 or 4 (fp8); 0 = the library's choice
                               (4 for fp8 pools; for bf16 pools 1 when
                               B * H_kv * maxP is below 512 pages per wave,
                               else 2) */
    int32_t pipeline_depth; /* steps of pages in flight per wavefront while it
                               computes one: 1 (two wavefronts per SIMD) or 2 (one
                               per SIMD); 0 = the library's choice (2 for bf16,
                               1 for fp8 pools) */
    void *event_begin;    /* optional hipEvent_t recorded on the stream right before
                             the main attention kernel (profiling); NULL = none */
    void *event_end;      /* optional hipEvent_t recorded right after it (before the
                             merge of the cut requests) */
    int64_t *wave_times;  /* optional device array of 3 * W int64 (W = the waves the
                             call uses: every resident wave, or max_waves): wave w
                             writes [3w] = the 100 MHz real-time clock when it
                             starts, [3w+1] = the clock when it has written its
                             last result, [3w+2] = (XCD id << 32) | HW_ID of its
                             SIMD.  A timing record: the results are those of the
                             untraced call.  Built for head_dim 128 at the default
                             steps (bf16: pages_per_step 1 or 2 with
                             pipeline_depth 2; fp8: 4 pages, depth 1); other
                             shapes return BELLMAN_ERR_UNSUPPORTED.  NULL = none */
} bellman_attn_opts_t;

/* bellman_decode_attention with explicit tuning options (NULL = defaults).
 * Results of different options agree within floating-point reordering. */
int bellman_decode_attention_opts(const bellman_tensor_t *q, const bellman_tensor_t *k_pages,
                                  const bellman_tensor_t *v_pages,
                                  const bellman_tensor_t *block_table,
                                  const bellman_tensor_t *seq_lens, float scale,
                                  bellman_tensor_t *out, const bellman_attn_opts_t *opts,
                                  void *stream);

/* Bytes of the fixed per-device scratch array of
 * bellman_decode_attention_noalloc. */
#define BELLMAN_FIXED_SCRATCH_BYTES (32 << 20)

/*
 * bellman_decode_attention_opts for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, kernels and results as
 * bellman_decode_attention_opts (NULL opts = defaults); the call allocates
 * nothing (no hipMalloc, hipFree or allocating library routine).  The
 * scratch lives in a fixed array of BELLMAN_FIXED_SCRATCH_BYTES that the
 * library's code object holds on every GPU it runs on until the process
 * ends, instead of the growable workspace.  A call needs
 *     256 + 16 W + 8 S + 4 D S   bytes (regions rounded up to 256 B),
 *     S = 2 W G partial slots,
 * W the waves it uses (1024 for bf16 and 2048 for fp8 pools on a whole
 * MI355X, or max_waves if smaller): up to G = 16 at D = 128 for bf16 pools
 * and G = 8 for fp8 pools by default; fp8 pools with G = 16 need
 * max_waves <= 1900.  A call that needs more is rejected with
 * BELLMAN_ERR_UNSUPPORTED before anything is enqueued.  Every call on one
 * GPU shares that GPU's array and leaves its contents behind (nothing in it
 * has to start at any value); calls that overlap in time on one device, on
 * any streams, race and give wrong results.
 */
int bellman_decode_attention_noalloc(const bellman_tensor_t *q, const bellman_tensor_t *k_pages,
                                     const bellman_tensor_t *v_pages,
                                     const bellman_tensor_t *block_table,
                                     const bellman_tensor_t *seq_lens, float scale,
                                     bellman_tensor_t *out, const bellman_attn_opts_t *opts,
                                     void *stream);

/* One decode step in one call: bellman_kv_append(k_new, v_new, ...) followed
 * by bellman_decode_attention_opts(q, ...), with the same arguments, results
 * and pool bytes, but no append launch (and no kernel boundary) between
 * them.  The attention reads length seq_lens[b] + 1 for every request with
 * 0 <= seq_lens[b] < maxP * 16; the wave that reads a (request, KV head)'s
 * new position writes the new K and V rows there first (bf16 rows, fp8
 * codes, or bf16 rows quantised into fp8 pools with the pools' dequant
 * scales, exactly as the append does), and the merge pass then advances
 * seq_lens as the append does (flag 1 where the position is outside the
 * table or the pool).  One difference, for a position the append would
 * refuse because its block-table entry lies outside the pool: the append
 * leaves the request's attention over its old tokens, while here the
 * attention reads the new position, finds the entry outside the pool, and
 * writes that request's rows as NaN (flags 1 and 4).  The page that takes a
 * request's new row must not be read by any other request of the same call
 * (shared prefix pages are full, so this holds for them): the write and the
 * other request's read are not ordered within the launch.  Built for the
 * default steps only (opts pages_per_step 0, 1 or 2 and pipeline_depth 0 or
 * 2 over bf16 pools; pages_per_step 0 or 4 and pipeline_depth 0 or 1 over
 * fp8 pools) and without wave_times; other options return
 * BELLMAN_ERR_UNSUPPORTED before anything is written.  Same workspace and
 * graph-capture properties as bellman_decode_attention_opts. */
int bellman_decode_step(const bellman_tensor_t *k_new, const bellman_tensor_t *v_new,
                        const bellman_tensor_t *q, bellman_tensor_t *k_pages,
                        bellman_tensor_t *v_pages, const bellman_tensor_t *block_table,
                        bellman_tensor_t *seq_lens, float scale, bellman_tensor_t *out,
                        const bellman_attn_opts_t *opts, void *stream);

/* ----------------------------------------------------------- prompt path --
 * Before a request decodes, its prompt is prefilled (the step that sets the
 * time to first token, Sec. 3 "Our key proposal"; Sec. 4 "Setup and trace"):
 * the prompt's keys and values are written into its pages and every prompt
 * token attends causally over the cache.  Both calls take a batch of
 * requests whose new tokens are concatenated: q_start int32 [B + 1] (device,
 * contiguous) with q_start[0] = 0 gives request b the token rows
 * q_start[b] .. q_start[b+1]-1 (n_b = q_start[b+1] - q_start[b] >= 0).
 * Requests may already hold cached tokens (chunked prefill).
 */

/* Write n_b new tokens per request at positions seq_lens[b] .. seq_lens[b] +
 * n_b - 1 (page block_table[b][pos / 16], slot pos % 16), then set
 * seq_lens[b] += n_b.
 *   k_new, v_new  [T, H_kv, D] in the pools' element type, innermost
 *                 contiguous, rows 16-byte aligned; T = q_start[B].
 *   k_pages, v_pages, block_table: as for bellman_kv_append; the pages of
 *                 every new position must already be assigned.
 *   seq_lens      int32 [B] contiguous (read, then advanced).
 * Byte-exact copies; nothing else is written.  A token outside its
 * request's table or the pool is skipped and flagged (flag 1), and that
 * request's length is left unchanged when its last position does not fit.
 * Once the workspace has grown to the call's size, the call enqueues only
 * kernels on `stream` (graph-capturable). */
int bellman_kv_write(const bellman_tensor_t *k_new, const bellman_tensor_t *v_new,
                     bellman_tensor_t *k_pages, bellman_tensor_t *v_pages,
                     const bellman_tensor_t *block_table, bellman_tensor_t *seq_lens,
                     const bellman_tensor_t *q_start, void *stream);

/* Causal prompt attention over the paged cache: request b's query rows are
 * its last n_b of L_b = seq_lens[b] cached tokens, and the row of token
 * q_start[b] + i, at position p = L_b - n_b + i, gets
 *   out[., h, :] = sum_{t <= p} softmax_t(scale * <q[., h, :], k_t>) * v_t
 * (query head h reads KV head h / G).
 *   q            bf16 [T, H_q, D], innermost contiguous, rows 16-byte aligned.
 *   k_pages, v_pages  pools as for bellman_decode_attention, bf16 or fp8
 *                (fp8: each tensor's dequant_scale [B, H_kv] is required,
 *                and key k_t, value v_t of request b, KV head g read as
 *                k_scale[b][g] * code, v_scale[b][g] * code); D in {64,
 *                128}; H_q a multiple of H_kv.
 *   block_table  int32 [B, maxP]; seq_lens int32 [B] (after the write).
 *   out          bf16 [T, H_q, D] (written, rounded to nearest even); rows of
 *                a malformed request (n_b > L_b, rows past T, L_b past the
 *                table: flag 2) are not written; a q_start that decreases, starts below
 *                0 or ends past T writes no row at all (flag 2).
 * Each workgroup takes 128 query rows of one request and one query head;
 * QK^T runs on the bf16 matrix cores and PV on the fp16 ones, in one pass
 * with P rounded to fp16 (11 significant bits; P rounded to bf16 once would
 * spend the bf16 error budget).  Over bf16 pools the values the call reads
 * are first copied into the workspace as fp16, each (request, KV head) at
 * the power of two 2^e that brings its largest magnitude M into
 * [2^14, 2^15): every value of at least M 2^-28 converts exactly, none
 * overflows, and the output is scaled back by 2^-e.  Over fp8 pools the
 * codes are staged in LDS as bytes and widened exactly at the operand load
 * (K to bf16, V to fp16); the K scale folds into the softmax scale and the
 * V scale into the final normalisation.  Scratch in the per-device
 * workspace: 2 (B + 1) + B H_kv integers, and over bf16 pools B maxP
 * (4 + 4 H_kv + 32 D H_kv) bytes more for the value copy and its
 * bookkeeping (maxP = the block table's width).  Like bellman_kv_write, once
 * the workspace has grown to the call's size the call enqueues only kernels
 * (graph-capturable). */
int bellman_prefill_attention(const bellman_tensor_t *q, const bellman_tensor_t *k_pages,
                              const bellman_tensor_t *v_pages, const bellman_tensor_t *block_table,
                              const bellman_tensor_t *seq_lens, const bellman_tensor_t *q_start,
                              float scale, bellman_tensor_t *out, void *stream);

typedef struct bellman_prefill_opts {
    void *event_begin;    /* optional hipEvent_t recorded right before the attention
                             kernel (after the planning and value-copy kernels) */
    void *event_end;      /* optional hipEvent_t recorded right after it */
} bellman_prefill_opts_t;

/* bellman_prefill_attention with options (NULL = defaults). */
int bellman_prefill_attention_opts(const bellman_tensor_t *q, const bellman_tensor_t *k_pages,
                                   const bellman_tensor_t *v_pages, const bellman_tensor_t *block_table,
                                   const bellman_tensor_t *seq_lens, const bellman_tensor_t *q_start,
                                   float scale, bellman_tensor_t *out,
                                   const bellman_prefill_opts_t *opts, void *stream);

/* ------------------------------------------------ output-length control --
 * The paper's linear congestion controller (Sec. 3: "Our key proposal",
 * "Placeholder for congestion control", "Default unbounded run", "beLLMan in
 * action").  Host only; no HIP call.  Each second the scheduler's average TBT
 * is pushed; the controller keeps the moving average MA of the last `window`
 * samples and sets the reduction rate
 *     r = 0                                        if MA <= t1
 *     r = clamp(r_min + (r_max - r_min)(MA - t1)/(t2 - t1), r_min, r_max)
 *                                                  if MA >  t1
 * (r = r_max on trigger when t2 <= t1).  A queued request with predicted
 * unbounded length L is asked for N = max(1, floor(L (1 - r) + 0.5)), and
 * N = L when r = 0 or L = 0.  Arithmetic is binary64.  A controller object
 * is not thread-safe.
 */
typedef struct bellman_controller bellman_controller_t;

/* t1, t2: trigger and full-reduction thresholds (same unit as the TBT
 * samples; the paper uses the median and 75th percentile of an unbounded
 * run); window >= 1 samples (paper: 5 one-second samples); 0 <= r_min <=
 * r_max < 1 (paper: 0.05 and 0.20).  Returns NULL on invalid arguments. */
bellman_controller_t *bellman_controller_create(double t1, double t2, int32_t window,
                                                double r_min, double r_max);
void bellman_controller_destroy(bellman_controller_t *ctl);
/* Current reduction rate r, or a negative status for a NULL controller. */
double bellman_controller_rate(const bellman_controller_t *ctl);

typedef struct bellman_load_signal {
    bellman_controller_t *controller;  /* controller to read (and update) */
    int32_t has_sample;                /* 1: push tbt_avg first (once per second) */
    double tbt_avg;                    /* the last second's average TBT */
    int32_t predicted_len;             /* predicted unbounded output length L >= 0 */
} bellman_load_signal_t;

/* Optionally push one TBT sample, then return the length cap N for a request
 * whose predicted unbounded length is predicted_len (see above), or a
 * negative status (NULL signal or controller, negative length, non-finite
 * sample). */
int32_t bellman_length_cap(const bellman_load_signal_t *load_signal);

/* Thresholds from an unbounded run's per-second TBTs: *t1 = median, *t2 =
 * 75th percentile, by linear interpolation between order statistics
 * (fractional rank p/100 * (n - 1)).  Host arrays; n >= 1. */
int bellman_calibrate_thresholds(const double *tbt, int64_t n, double *t1, double *t2);

/* ------------------------------------------------- controller variants --
 * The controllers the paper's future-work section names (Sec. 5, "Toward
 * novel LLM congestion control") and per-class policies ("Nuanced fairness
 * issues").  The paper gives their goals, not algorithms; these are this
 * library's readings.  A variant observes one tick at a time
 * (bellman_controller_observe): whether TBT samples arrived, their mean
 * tbt (same unit as t1, t2), the tokens they decoded and the tick length.
 *
 * MPC (BELLMAN_CTL_MPC): on a tick with samples, once `window` samples exist
 *   a least-squares line through the last `window` gives slope s (per tick)
 *   and value v at the newest (before that s = 0, v = the newest sample); the
 *   floor b is the least of the last floor_window samples.  For a candidate
 *   rc, h ticks ahead:  u_h = max(v + s h, b);  f_h = 1 - exp(-h / tau)
 *   (the share of decode work from requests capped at rc);
 *   y_h = b + (u_h - b) ((1 - f_h) + f_h (1 - rc) / (1 - r)), and
 *   J = sum_{h=1..horizon} w_lat (max(0, y_h - t1) / (t2 - t1))^2
 *       + horizon (w_quality - w_energy) rc + w_delta ((rc - r) / r_max)^2.
 *   Candidates 0, r_min, r_min + step, ... (below r_max), r_max; the first
 *   with the least J becomes r.  Needs t2 > t1.
 * BBR-style (BELLMAN_CTL_BBR): x = tokens / tick_s each tick; BtlBw = max x of
 *   the last bw_window ticks; RTprop = min TBT of the last rt_window ticks
 *   with samples.  On a tick with samples: if TBT > RTprop (1 + margin) and
 *   x >= (1 - margin) BtlBw, r_base += bbr_step (at most r_max); else if
 *   TBT <= RTprop (1 + margin / 2), r_base -= bbr_step (at least 0).  Applied
 *   r = clamp(r_base + o, 0, r_max) with o = -probe on the first tick of each
 *   `cycle`-tick cycle, +probe on the second, 0 otherwise.
 * PCC (BELLMAN_CTL_PCC): rounds of two monitor intervals of `interval` ticks
 *   at center + epsilon and center - epsilon (clamped to [0, r_max]), up
 *   first in even rounds and down first in odd ones.  An interval's utility
 *   U = -pcc_w_lat max(0, mean TBT - t1) / (t2 - t1) - pcc_w_quality r / r_max
 *   (no latency term without samples); after a round
 *   center = clamp(center + gain (U_a - U_b) / (r_a - r_b), 0, r_max)
 *   (no step when the two rates coincide).  r is the running interval's rate.
 *   Needs t2 > t1.
 * Linear (BELLMAN_CTL_LINEAR): the controller above; a tick pushes its mean
 *   TBT when it has samples.
 * Arithmetic is binary64 in the order stated, without fused multiply-adds.
 */
typedef enum bellman_ctl_kind {
    BELLMAN_CTL_LINEAR = 1,
    BELLMAN_CTL_MPC = 2,
    BELLMAN_CTL_BBR = 3,
    BELLMAN_CTL_PCC = 4
} bellman_ctl_kind_t;

typedef struct bellman_ctl_params {
    int32_t kind;                 /* bellman_ctl_kind_t */
    int32_t window;               /* linear: MA samples; MPC: trend-fit samples (>= 1) */
    double t1, t2;                /* TBT thresholds (linear, MPC, PCC) */
    double r_min, r_max;          /* 0 <= r_min <= r_max < 1 */
    int32_t horizon;              /* MPC: ticks predicted (>= 1) */
    int32_t floor_window;         /* MPC: samples behind the TBT floor (>= 1) */
    double tau;                   /* MPC: ticks for a new rate to reach the load (> 0) */
    double w_lat, w_quality, w_energy, w_delta;   /* MPC cost weights (>= 0) */
    double step;                  /* MPC: candidate spacing (> 0) */
    int32_t bw_window, rt_window; /* BBR: ticks behind BtlBw and RTprop (>= 1) */
    int32_t cycle;                /* BBR: probe / drain cycle, ticks (>= 1) */
    int32_t reserved0;            /* 0 */
    double margin;                /* BBR: queueing margin over RTprop, in [0, 1) */
    double bbr_step, probe;       /* BBR: r_base step per tick, probe offset (>= 0) */
    int32_t interval;             /* PCC: ticks per monitor interval (>= 1) */
    int32_t reserved1;            /* 0 */
    double epsilon, gain;         /* PCC: rate offset of an experiment, gradient step (>= 0) */
    double pcc_w_lat, pcc_w_quality;  /* PCC utility weights (>= 0) */
} bellman_ctl_params_t;

/* Fill *p with the defaults of `kind` and thresholds t1, t2: window 5,
 * r in [0.05, 0.20]; MPC horizon 10, floor_window 60, tau 20, weights
 * 1 / 0.25 / 0.1 / 0.2, step 0.01; BBR windows 10 and 30, cycle 8, margin
 * 0.25, step 0.02, probe 0.02; PCC interval 10, epsilon 0.02, gain 0.02,
 * weights 1 / 0.5.  Returns 0 or BELLMAN_ERR_INVALID_ARG. */
int bellman_ctl_params_default(int32_t kind, double t1, double t2, bellman_ctl_params_t *p);

/* A controller of any kind (destroy with bellman_controller_destroy), or
 * NULL on invalid parameters. */
bellman_controller_t *bellman_controller_create_ex(const bellman_ctl_params_t *p);

typedef struct bellman_ctl_obs {
    int32_t has_sample;           /* 1: TBT samples arrived in the tick */
    int32_t reserved;             /* 0 */
    double tbt_avg;               /* their mean (finite when has_sample) */
    double tokens;                /* tokens they decoded (>= 0) */
    double tick_s;                /* tick length in seconds (> 0) */
} bellman_ctl_obs_t;

/* Feed one tick; returns the new rate r (>= 0) or a negative status (NULL
 * arguments, non-finite sample, negative tokens, tick_s <= 0).
 * bellman_length_cap's sample is a tick with no token count. */
double bellman_controller_observe(bellman_controller_t *ctl, const bellman_ctl_obs_t *obs);

typedef struct bellman_class_policy {
    double weight;                /* the class applies min(weight r, r_max); 0 exempts it */
    int32_t bypass_len;           /* predicted lengths at or below this are not reduced */
    int32_t reserved;             /* 0 */
} bellman_class_policy_t;

/* Length cap for a request of a class: N = L when L <= bypass_len, else
 * N = max(1, floor(L (1 - rc) + 0.5)) with rc = min(weight r, r_max)
 * (N = L when rc = 0 or L = 0).  Negative status on NULL arguments, L < 0
 * or a negative or non-finite weight. */
int32_t bellman_length_cap_class(const bellman_controller_t *ctl, int32_t predicted_len,
                                 const bellman_class_policy_t *policy);

/* ------------------------------------------- closed-loop serving model --
 * A discrete-event model of the paper's evaluation (Sec. 4, "Setup and
 * trace", "Default unbounded run", "beLLMan in action"): requests arrive
 * (caller-supplied times and sizes), wait in a FIFO queue, are admitted into a
 * continuously batched server with paged KV memory, chunked prefill and
 * preemption by recomputation (the behaviour of the vLLM scheduler the paper
 * serves with), decode one token per iteration until they reach their target
 * length, and the controller above sees the per-second average time between
 * tokens (TBT) and caps the targets of newly queued requests.  Host
 * arithmetic in integer nanoseconds; each iteration, in this order:
 *  1. Ticks (k * tick_ns) and arrivals up to the current time, in time order,
 *     a tick first on ties.  A tick averages the TBT samples of the tokens
 *     decoded in ((k-1) tick_ns, k tick_ns] and gives the controller that
 *     tick (the linear controller takes only ticks with samples).  An
 *     arrival is queued with target N = bellman_length_cap_class(L) under
 *     the current rate and its class's policy (N = L without a controller).
 *  2. First-come first-served admission while fewer than max_running run: the
 *     queue head must prefill P = prompt + generated tokens (generated > 0
 *     after a preemption) and is admitted if ceil(P / 16) pages can be taken
 *     leaving watermark_pages free.
 *  3. With nothing running, time jumps to the next arrival.
 *  4. In running order, a decoding request whose next KV position
 *     (prompt + generated - 1) lies past its pages takes one more page; with
 *     none free, the most recently admitted running requests are preempted
 *     (pages returned, prefill progress dropped, back at the queue head,
 *     earlier-admitted first) until one is, or the request itself was.
 *  5. In running order, prefilling requests take up to the remaining
 *     prefill_chunk_tokens of this iteration (no limit when 0).
 *  6. Duration = fixed_ns + attention time + prefill time: the model takes
 *     (attn_ps_per_token * KV + prefill_ps_per_token * chunk) / 1000 with KV
 *     the decoding requests' summed prompt + generated tokens; live mode
 *     replaces the attention term by the measured time of the real
 *     bellman_kv_append + bellman_decode_attention on the decoding requests
 *     times live_layers (and adds prefill_ps_per_token * chunk / 1000).
 *  7. Decoding requests gain a token and one TBT sample each (the duration);
 *     a request that completed its prefill gains a token (the first one fixes
 *     its TTFT) and starts decoding; one that reaches N finishes and frees
 *     its pages.  Running order is kept.
 */
typedef enum bellman_sim_controller_kind {
    BELLMAN_SIM_NO_CONTROL = 0,   /* targets = predicted lengths */
    BELLMAN_SIM_LINEAR = 1,       /* the paper's linear controller (t1, t2, window, r_min, r_max) */
    BELLMAN_SIM_MPC = 2,          /* controller variants (see above); each tick is an observation */
    BELLMAN_SIM_BBR = 3,          /* with the tick's TBT samples, their mean, the tokens they */
    BELLMAN_SIM_PCC = 4           /* decoded and tick_ns / 1e9 seconds */
} bellman_sim_controller_kind_t;

typedef struct bellman_sim_config {
    int32_t max_running;          /* >= 1 requests in the running batch (prefilling or decoding) */
    int32_t controller;           /* bellman_sim_controller_kind_t */
    int64_t kv_capacity_pages;    /* KV budget in 16-token pages */
    int64_t watermark_pages;      /* pages admission leaves free (>= 0) */
    int64_t fixed_ns;             /* per-iteration time of everything but attention and prefill */
    int64_t attn_ps_per_token;    /* model mode: attention picoseconds per attended KV token */
    int64_t prefill_ps_per_token; /* picoseconds per prefilled token */
    int64_t tick_ns;              /* controller period (paper: 1 s) */
    double t1, t2;                /* controller thresholds, nanoseconds of TBT */
    int32_t window;               /* controller moving-average length (paper: 5) */
    int32_t prefill_chunk_tokens; /* prefill tokens per iteration, 0 = unlimited */
    double r_min, r_max;          /* controller rate range (paper: 0.05, 0.20) */
    int32_t live;                 /* 0: model; 1: time the real kernels on the current device */
    int32_t live_layers;          /* live: model layers one measured attention layer stands for */
    int32_t live_q_heads;         /* live: per-GPU query heads of the measured layer */
    int32_t live_kv_heads;        /* live: per-GPU KV heads (bf16 pools, 16-token pages) */
    int32_t live_head_dim;        /* live: 64 or 128 */
    int32_t reserved;             /* 0 */
    void *stream;                 /* live: hipStream_t for the kernels (NULL = null stream) */
    const bellman_ctl_params_t *ctl_params;  /* controller parameters, kind = controller; NULL:
                                                the defaults with t1, t2, window, r_min, r_max above */
    const int32_t *req_class;     /* per-request class in [0, n_classes), or NULL (all class 0) */
    const bellman_class_policy_t *classes;   /* n_classes policies, or NULL (weight 1, no bypass) */
    int32_t n_classes;            /* >= 1 when req_class or classes is given */
    int32_t reserved2;            /* 0 */
} bellman_sim_config_t;

typedef struct bellman_sim_request {
    int64_t admit_ns;             /* first admission (prefill start) */
    int64_t first_ns;             /* first token */
    int64_t finish_ns;            /* last token */
    int32_t target;               /* N, tokens */
    int32_t preemptions;          /* times the request was preempted */
    double r_at_queue;            /* controller rate when the request arrived */
} bellman_sim_request_t;

typedef struct bellman_sim_tick {
    int64_t t_ns;                 /* tick time */
    int64_t tokens;               /* TBT samples in the tick's second */
    int64_t tbt_sum_ns;           /* their sum */
    double r;                     /* controller rate after the tick */
    int32_t queued;               /* queue length when the tick was taken */
    int32_t running;              /* running requests when the tick was taken */
} bellman_sim_tick_t;

typedef struct bellman_sim_iteration {
    int64_t end_ns;               /* iteration end */
    int64_t dt_ns;                /* its duration */
    int32_t decoding;             /* requests that decoded a token (TBT samples) */
    int32_t chunk;                /* prefill tokens processed */
    int32_t running;              /* running requests at the start of step 4 */
    int32_t queued;               /* queue length at the start of step 4 */
} bellman_sim_iteration_t;

typedef struct bellman_sim_stats {
    int64_t iterations;
    int64_t ticks;                /* ticks taken (only the first max_ticks are stored) */
    int64_t end_ns;               /* time the last request finished */
    int64_t preemptions;          /* total preemptions */
    double live_gpu_ms;           /* live: summed measured append + attention time */
    int64_t live_kv_bytes;        /* live: K/V bytes the measured attention launches read */
} bellman_sim_stats_t;

/* Run the model over n requests (host arrays: arrival_ns non-decreasing and
 * >= 0, prompt >= 1 and length >= 1 tokens, ceil((prompt + length) / 16) +
 * watermark_pages <= kv_capacity_pages).  Writes requests[n], the first
 * max_ticks ticks, the first max_iterations iteration records (iterations may
 * be NULL when max_iterations is 0) and *stats (host memory, caller-owned).  Live mode
 * allocates its own device buffers (KV pools of kv_capacity_pages pages,
 * block table, lengths, query and new-token rows), synchronises the stream
 * once per iteration to read the kernel time, and frees them before
 * returning.  Returns 0 or a negative status (bad configuration or arrays,
 * HIP failure, device error flags raised by the live kernels). */
int bellman_sim_run(const bellman_sim_config_t *cfg, int64_t n, const int64_t *arrival_ns,
                    const int32_t *prompt, const int32_t *length,
                    bellman_sim_request_t *requests, bellman_sim_tick_t *ticks,
                    int64_t max_ticks, bellman_sim_iteration_t *iterations,
                    int64_t max_iterations, bellman_sim_stats_t *stats);

/* ----------------------------------------------------------------- misc -- */

/* Text of the last error raised on the calling thread ("" if none). */
const char *bellman_last_error(void);

/* Make sure the current device's workspace holds at least `bytes`
 * (hipMalloc outside any timed region or graph capture; a smaller block it
 * replaces stays allocated until bellman_shutdown). */
int bellman_reserve_workspace(int64_t bytes);

/* Synchronise `stream`, copy the current device's error word to *flags and
 * clear it.  Bits: 1 = an append slot outside the block table or pool,
 * 2 = an attention length above maxP*16 (clamped) or a malformed prompt
 * range, 4 = a block-table entry
 * outside the pool (page skipped). */
int bellman_device_errors(void *stream, int32_t *flags);

/*
 * Diagnostic: the page-pattern ceiling.  Reads every tile of a device pool
 * of pool_bytes once, n = pool_bytes / tile_bytes tiles (n a power of two,
 * tile_bytes 2048, 4096 or 8192: an fp8 or bf16 KV page of one head at
 * head_dim 128, or two), in a fixed scrambled order (a bijection of the
 * tile indices built from odd multiplications and xor-shifts) that spreads
 * each wave's consecutive tiles, and the tiles all waves read at one time,
 * over the pool, as a batch's random pages are.  The loads are the decode kernel's (16 bytes a
 * lane, non-temporal), with no arithmetic but an XOR of every 32-bit word
 * into *sink, which the caller clears beforehand (the result is the XOR of
 * the whole pool).  max_waves caps the waves (0 = every resident wave).  The
 * bytes read over the kernel's time are the rate the attention kernel's page
 * stream can reach on this device.  pool 16-byte aligned, sink 4-byte
 * aligned; enqueues one kernel on `stream`.
 */
int bellman_probe_gather(const void *pool, int64_t pool_bytes, int32_t tile_bytes, int32_t max_waves,
                         uint32_t *sink, void *stream);

/* Synchronise every device that holds a workspace and free its blocks
 * (current and retired).  No call may be in flight, and graphs captured
 * with library calls must not be replayed afterwards. */
void bellman_shutdown(void);

/* Library version as "major.minor.patch". */
const char *bellman_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BELLMAN_H */
