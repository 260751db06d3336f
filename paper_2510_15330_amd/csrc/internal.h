// Internal declarations shared by the host ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/bellman.h"

namespace bellman {

constexpr int kPage = 16;           // tokens per KV page
constexpr int kWaveSize = 64;       // CDNA wavefront
constexpr int kAttnBlock = 256;     // threads per attention workgroup (4 independent waves)

// Device error word bits (also documented in bellman.h).
constexpr int kErrAppendSlot = 1;
constexpr int kErrLength = 2;
constexpr int kErrPage = 4;

constexpr int kMaxDevices = 64;

// A workspace (the library's growable one, or the fixed scratch array)
// starts with a 256-byte header; the per-call regions follow.  Nothing in it
// has to start at any value.
constexpr int kMaxWaves = 16384;
constexpr size_t kWsHeader = 256;

// Bytes of the fixed per-device scratch array of the no-allocation decode
// entry point (device_state.hip).
constexpr size_t kScratchBytes = (size_t)BELLMAN_FIXED_SCRATCH_BYTES;

struct AppendArgs {
    const void* k_new;   // [B, H_kv, D]
    const void* v_new;
    int64_t new_sb, new_sh;        // strides (elements) of k_new/v_new rows
    int64_t vnew_sb, vnew_sh;
    void* k_pages;       // [NP, H_kv, D/x, 16, x]
    void* v_pages;       // [NP, H_kv, D, 16]
    const int32_t* block_table;
    int64_t bt_stride;
    int32_t* seq_lens;
    int32_t* err;
    int64_t num_pages;
    const float* k_scale;  // quantising append only: fp32 [B, H_kv]
    const float* v_scale;
    int B, H_kv, D, max_pages, elem_bytes;
    int quant;             // 1: bf16 rows quantised into fp8 pools
};

struct AttnArgs {
    const uint16_t* q;   // bf16 [B, H_q, D]
    int64_t q_sb, q_sh;
    const void* k_pages;
    const void* v_pages;
    const float* k_scale;   // fp8 only, [B, H_kv]
    const float* v_scale;
    const int32_t* block_table;
    int64_t bt_stride;
    const int32_t* seq_lens;
    uint16_t* out;       // bf16 [B, H_q, D]
    int64_t o_sb, o_sh;
    int64_t num_pages;
    float scale_log2;    // softmax scale * log2(e)
    int B, H_q, H_kv, G, D, max_pages;
    int waves;           // waves sharing the flattened step stream (the grid's waves)
    int pp;              // pages per step of the launched attention kernel
    int skew;            // share weights 256 + skew (even-XCD workgroups) / 256 - skew on long shares; 0..255
                         // (work_split.h)
    int32_t* err;        // the device's error word
    // workspace
    int4* cuts;          // [waves]: (request, KV head, last wave, units) of the (request, head) in
                         // which wave w's range ends if it began inside the range and runs past
                         // it, else request -1; written by the attention kernel for the merge
    float2* part_ml;     // [2 * waves * G]: (running max in log2 units, sum) of each wave's two
                         // partial pieces (the request cut at its range's start, and at its end)
    float* part_o;       // [2 * waves * G * D]
    int64_t* wave_times; // optional [3 * waves] per-wave timing records (traced kernel), else null
    // decode step (the append fused into this call), else k_new null: the
    // attention reads length seq_lens[b] + 1 where 0 <= seq_lens[b] < maxP 16,
    // the wave that reads a (request, head)'s new position first writes the
    // new row there, and the merge pass advances the lengths
    const void* k_new;   // [B, H_kv, D] rows in the pools' element type, or bf16 into fp8 pools
    const void* v_new;
    int64_t new_sb, new_sh, vnew_sb, vnew_sh;   // strides (elements)
    int quant;           // 1: bf16 rows quantised into fp8 pools
    int32_t* lens_rw;    // seq_lens, advanced by the merge pass
};

// Prompt KV write (prefill.hip).
struct WriteArgs {
    const void* k_new;   // [T, H_kv, D] pool element type
    const void* v_new;
    int64_t k_st, k_sh, v_st, v_sh;   // row strides (elements)
    void* k_pages;
    void* v_pages;
    const int32_t* block_table;
    int64_t bt_stride;
    int32_t* seq_lens;
    const int32_t* q_start;  // [B + 1]
    int32_t* err;
    int64_t num_pages;
    int B, T, H_kv, D, max_pages, elem_bytes;
};

// Prompt (prefill) attention over the paged cache (prefill.hip).
constexpr int kPrefillRows = 128;   // query rows per workgroup (4 waves x 32)
struct PrefillArgs {
    const uint16_t* q;   // bf16 [T, H_q, D]
    int64_t q_st, q_sh;
    const void* k_pages;
    const void* v_pages;
    const int32_t* block_table;
    int64_t bt_stride;
    const int32_t* seq_lens;   // [B]: cached tokens, the last n_b are the queries
    const int32_t* q_start;    // [B + 1]
    uint16_t* out;       // bf16 [T, H_q, D]
    int64_t o_st, o_sh;
    int64_t num_pages;
    float scale_log2;
    int B, T, H_q, H_kv, G, D, max_pages;
    int32_t* err;
    int32_t* tile_start;   // workspace [B + 1]: first query tile of each request
    int fp8;               // pools of e4m3fn codes with the dequantisation scales below
    const float* k_scale;  // fp8 only, fp32 [B, H_kv]
    const float* v_scale;
    // bf16 pools: the fp16 copy of the values the attention reads (workspace)
    int32_t* page_off;     // [B + 1]: first copied page of each request
    int32_t* page_req;     // [B * maxP]: the request of each copied page
    float* tmax;           // [copied pages, H_kv]: the largest |v| of each (page, head) tile
    uint32_t* vmax;        // [B, H_kv]: float bits of the largest |v| of each (request, KV head)
    uint16_t* vcopy;       // [sum of copied pages, H_kv, D, 16] fp16
    int vgrid;             // workgroups of the copy passes (4 waves each)
};

// Launchers (kernels.hip).  They only enqueue; errors come back through
// hipGetLastError in the caller.
void launch_kv_append(const AppendArgs& a, hipStream_t s);
void launch_attention(const AttnArgs& a, int pages_per_step, int depth, bool fp8, int grid, hipStream_t s);
// Whether the attention kernel variant has a traced twin (wave_times).
bool attention_traced(int pages_per_step, int depth, bool fp8, int D);
// Whether the attention kernel variant has a decode-step twin (k_new set).
bool attention_step_built(int pages_per_step, int depth, bool fp8);
// Resident workgroups per CU of the attention kernel variant (occupancy).
int attention_blocks_per_cu(int pages_per_step, int depth, bool fp8, int D);
void launch_merge(const AttnArgs& a, hipStream_t s);
// Prefill launchers (prefill.hip).
void launch_kv_write(const WriteArgs& a, int32_t* page_start, hipStream_t s);
// The prompt attention's planning (and, over bf16 pools, the fp16 value
// copy), then the attention kernel itself.
void launch_prefill_prep(const PrefillArgs& a, hipStream_t s);
void launch_prefill_attn(const PrefillArgs& a, hipStream_t s);

// Page-pattern gather probe (probe.hip): n tiles of tile_bytes, n a power of
// two; nonzero if tile_bytes is not a built size.
int launch_gather_probe(const void* pool, int64_t n, int tile_bytes, int waves, uint32_t* sink, hipStream_t s);
int gather_probe_blocks_per_cu(int tile_bytes);

// Addresses of the current device's error word and fixed scratch array
// (device_state.hip); dev must be the current device.  0 or a negative
// bellman status.
int device_error_word(int dev, int32_t** p);
int device_scratch(int dev, char** p);

// Record the calling thread's last-error text (bellman_last_error) and
// return `code`; shared by the host-side parts of the library.
int set_error(int code, const char* fmt, ...);

}  // namespace bellman
