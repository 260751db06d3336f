// Closed-loop serving model: Poisson-fed continuous batching with beLLMan's
// output-length controller in the loop (arXiv 2510.15330, Sec. 4 "Setup and
// trace", "Default unbounded run", "beLLMan in action"; Sec. 3 "Our key
// proposal").  The steps and their order are documented with
// bellman_sim_run in bellman.h.  In live mode every iteration runs the
// library's own append and decode-attention kernels on the running batch
// (rows of the batch are the running requests, pages come from a free list)
// and uses their measured time.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <deque>
#include <initializer_list>
#include <map>
#include <utility>
#include <vector>

#include "../../include/bellman.h"
#include "internal.h"

using bellman::set_error;

namespace {

constexpr int64_t kPage = BELLMAN_PAGE_TOKENS;

int64_t ceil_pages(int64_t tokens) { return (tokens + kPage - 1) / kPage; }

// Device side of live mode: KV pools of the page budget, a batch of up to
// max_running rows (block table, lengths, query and new-token rows).
struct LiveGpu {
    hipStream_t s = nullptr;
    int Hq = 0, Hkv = 0, D = 0, M = 0;
    int64_t maxP = 0, NP = 0;
    void *kp = nullptr, *vp = nullptr, *bt = nullptr, *sl = nullptr;
    void *q = nullptr, *kn = nullptr, *vn = nullptr, *out = nullptr;
    int32_t *bt_h = nullptr, *sl_h = nullptr;  // pinned staging
    hipEvent_t e0 = nullptr, e1 = nullptr;
    std::vector<char> dirty;                   // rows whose block-table row must be uploaded

    ~LiveGpu() { release(); }

    void release() {
        if (s || kp) (void)hipStreamSynchronize(s);
        for (void* p : {kp, vp, bt, sl, q, kn, vn, out})
            if (p) (void)hipFree(p);
        kp = vp = bt = sl = q = kn = vn = out = nullptr;
        if (bt_h) (void)hipHostFree(bt_h);
        if (sl_h) (void)hipHostFree(sl_h);
        bt_h = sl_h = nullptr;
        if (e0) (void)hipEventDestroy(e0);
        if (e1) (void)hipEventDestroy(e1);
        e0 = e1 = nullptr;
    }

    int init(const bellman_sim_config_t* c, int64_t max_pages) {
        s = (hipStream_t)c->stream;
        Hq = c->live_q_heads;
        Hkv = c->live_kv_heads;
        D = c->live_head_dim;
        M = c->max_running;
        maxP = max_pages;
        NP = c->kv_capacity_pages;
        const size_t pool = (size_t)NP * Hkv * kPage * D * 2;
        const size_t rows_q = (size_t)M * Hq * D * 2, rows_kv = (size_t)M * Hkv * D * 2;
        hipError_t e;
#define SIM_HIP(call)                                                                          \
    do {                                                                                       \
        e = (call);                                                                            \
        if (e != hipSuccess) return set_error(BELLMAN_ERR_HIP, "sim: %s: %s", #call, hipGetErrorString(e)); \
    } while (0)
        SIM_HIP(hipMalloc(&kp, pool));
        SIM_HIP(hipMalloc(&vp, pool));
        SIM_HIP(hipMalloc(&bt, (size_t)M * maxP * 4));
        SIM_HIP(hipMalloc(&sl, (size_t)M * 4));
        SIM_HIP(hipMalloc(&q, rows_q));
        SIM_HIP(hipMalloc(&out, rows_q));
        SIM_HIP(hipMalloc(&kn, rows_kv));
        SIM_HIP(hipMalloc(&vn, rows_kv));
        SIM_HIP(hipHostMalloc((void**)&bt_h, (size_t)M * maxP * 4, hipHostMallocDefault));
        SIM_HIP(hipHostMalloc((void**)&sl_h, (size_t)M * 4, hipHostMallocDefault));
        SIM_HIP(hipEventCreate(&e0));
        SIM_HIP(hipEventCreate(&e1));
        SIM_HIP(hipMemsetAsync(kp, 0, pool, s));
        SIM_HIP(hipMemsetAsync(vp, 0, pool, s));
        // query and new-token rows: fixed bf16 values in [-1, 1) from a
        // xorshift stream (their values do not change the time)
        std::vector<uint16_t> h(std::max(rows_q, rows_kv) / 2);
        uint32_t x = 0x9e3779b9u;
        for (auto& v : h) {
            x ^= x << 13;
            x ^= x >> 17;
            x ^= x << 5;
            const float f = (float)(x >> 8) * (2.0f / 16777216.0f) - 1.0f;
            uint32_t u;
            memcpy(&u, &f, 4);
            v = (uint16_t)(u >> 16);
        }
        SIM_HIP(hipMemcpyAsync(q, h.data(), rows_q, hipMemcpyHostToDevice, s));
        SIM_HIP(hipMemcpyAsync(kn, h.data(), rows_kv, hipMemcpyHostToDevice, s));
        SIM_HIP(hipMemcpyAsync(vn, h.data(), rows_kv, hipMemcpyHostToDevice, s));
        SIM_HIP(hipStreamSynchronize(s));
        // One untimed step over a full batch (every row on page 0, length 0)
        // loads the kernels and grows the library's workspace before the
        // model's clock starts.
        for (int64_t i = 0; i < (int64_t)M * maxP; ++i) bt_h[i] = (i % maxP) == 0 ? 0 : -1;
        for (int r = 0; r < M; ++r) sl_h[r] = 0;
        dirty.assign((size_t)M, 1);
        double ms = 0.0;
        const int rc = step(M, &ms);
        if (rc) return rc;
        for (int64_t i = 0; i < (int64_t)M * maxP; ++i) bt_h[i] = -1;
        dirty.assign((size_t)M, 1);
        return 0;
    }

    // Upload the lengths of rows [0, B) and the changed block-table rows,
    // then time one append + decode attention over those rows.
    int step(int B, double* ms) {
        hipError_t e;
        SIM_HIP(hipMemcpyAsync(sl, sl_h, (size_t)B * 4, hipMemcpyHostToDevice, s));
        for (int r = 0; r < M; ++r)
            if (dirty[(size_t)r]) {
                SIM_HIP(hipMemcpyAsync((int32_t*)bt + (int64_t)r * maxP, bt_h + (int64_t)r * maxP, (size_t)maxP * 4,
                                       hipMemcpyHostToDevice, s));
                dirty[(size_t)r] = 0;
            }
        bellman_tensor_t kpt{}, vpt{}, btt{}, slt{}, qt{}, knt{}, vnt{}, ot{};
        auto set = [](bellman_tensor_t& t, void* p, int32_t dt, std::initializer_list<int64_t> shape) {
            t.data = p;
            t.dtype = dt;
            t.ndim = (int32_t)shape.size();
            int i = 0;
            for (int64_t v : shape) t.shape[i++] = v;
            int64_t st = 1;
            for (int k = t.ndim - 1; k >= 0; --k) {
                t.stride[k] = st;
                st *= t.shape[k];
            }
        };
        set(kpt, kp, BELLMAN_BF16, {NP, Hkv, D / 8, kPage, 8});
        set(vpt, vp, BELLMAN_BF16, {NP, Hkv, D, kPage});
        set(btt, bt, BELLMAN_INT32, {B, maxP});
        set(slt, sl, BELLMAN_INT32, {B});
        set(qt, q, BELLMAN_BF16, {B, Hq, D});
        set(ot, out, BELLMAN_BF16, {B, Hq, D});
        set(knt, kn, BELLMAN_BF16, {B, Hkv, D});
        set(vnt, vn, BELLMAN_BF16, {B, Hkv, D});
        SIM_HIP(hipEventRecord(e0, s));
        int rc = bellman_kv_append(&knt, &vnt, &kpt, &vpt, &btt, &slt, s);
        if (rc) return rc;
        rc = bellman_decode_attention(&qt, &kpt, &vpt, &btt, &slt, 1.0f / sqrtf((float)D), &ot, s);
        if (rc) return rc;
        SIM_HIP(hipEventRecord(e1, s));
        SIM_HIP(hipEventSynchronize(e1));
        float t = 0.f;
        SIM_HIP(hipEventElapsedTime(&t, e0, e1));
        *ms = t;
        return 0;
    }
#undef SIM_HIP
};

int check_config(const bellman_sim_config_t* c) {
    if (!c) return set_error(BELLMAN_ERR_INVALID_ARG, "sim: null config");
    if (c->max_running < 1) return set_error(BELLMAN_ERR_INVALID_ARG, "sim: max_running must be >= 1");
    if (c->kv_capacity_pages < 1 || c->watermark_pages < 0 || c->watermark_pages >= c->kv_capacity_pages)
        return set_error(BELLMAN_ERR_INVALID_ARG, "sim: page budget %lld with watermark %lld",
                         (long long)c->kv_capacity_pages, (long long)c->watermark_pages);
    if (c->fixed_ns < 0 || c->attn_ps_per_token < 0 || c->prefill_ps_per_token < 0 || c->prefill_chunk_tokens < 0)
        return set_error(BELLMAN_ERR_INVALID_ARG, "sim: negative time coefficient or chunk");
    if (c->tick_ns < 1) return set_error(BELLMAN_ERR_INVALID_ARG, "sim: tick_ns must be >= 1");
    if (c->controller < BELLMAN_SIM_NO_CONTROL || c->controller > BELLMAN_SIM_PCC)
        return set_error(BELLMAN_ERR_INVALID_ARG, "sim: unknown controller kind %d", c->controller);
    if (c->ctl_params && c->ctl_params->kind != c->controller)
        return set_error(BELLMAN_ERR_INVALID_ARG, "sim: controller parameters of kind %d for controller %d",
                         c->ctl_params->kind, c->controller);
    if ((c->req_class || c->classes) && c->n_classes < 1)
        return set_error(BELLMAN_ERR_INVALID_ARG, "sim: classes given with n_classes %d", c->n_classes);
    for (int32_t k = 0; c->classes && k < c->n_classes; ++k)
        if (!(c->classes[k].weight >= 0.0) || !isfinite(c->classes[k].weight))
            return set_error(BELLMAN_ERR_INVALID_ARG, "sim: class %d weight %g", k, c->classes[k].weight);
    if (c->live) {
        if (c->live_layers < 1) return set_error(BELLMAN_ERR_INVALID_ARG, "sim: live_layers must be >= 1");
        if (c->live_head_dim != 64 && c->live_head_dim != 128)
            return set_error(BELLMAN_ERR_UNSUPPORTED, "sim: live_head_dim must be 64 or 128");
        if (c->live_kv_heads < 1 || c->live_q_heads < c->live_kv_heads || c->live_q_heads % c->live_kv_heads ||
            c->live_q_heads / c->live_kv_heads > 16)
            return set_error(BELLMAN_ERR_UNSUPPORTED, "sim: live heads %d/%d", c->live_q_heads, c->live_kv_heads);
        if (c->max_running > 8192) return set_error(BELLMAN_ERR_UNSUPPORTED, "sim: live max_running above 8192");
        if (c->kv_capacity_pages > ((int64_t)1 << 31) - 1)
            return set_error(BELLMAN_ERR_UNSUPPORTED, "sim: live page budget above 2^31 pages");
    }
    return 0;
}

enum State : int8_t { kNotArrived = 0, kQueued, kPrefill, kDecode, kDone };

}  // namespace

extern "C" int bellman_sim_run(const bellman_sim_config_t* cfg, int64_t n, const int64_t* arrival_ns,
                               const int32_t* prompt, const int32_t* length, bellman_sim_request_t* requests,
                               bellman_sim_tick_t* ticks, int64_t max_ticks, bellman_sim_iteration_t* iterations,
                               int64_t max_iterations, bellman_sim_stats_t* stats) {
    int rc = check_config(cfg);
    if (rc) return rc;
    if (n < 0 || !stats || (n > 0 && (!arrival_ns || !prompt || !length || !requests)) || max_ticks < 0 ||
        (max_ticks > 0 && !ticks) || max_iterations < 0 || (max_iterations > 0 && !iterations))
        return set_error(BELLMAN_ERR_INVALID_ARG, "sim: bad array arguments");
    int64_t max_pages = 1;
    for (int64_t j = 0; j < n; ++j) {
        if (arrival_ns[j] < 0 || (j > 0 && arrival_ns[j] < arrival_ns[j - 1]))
            return set_error(BELLMAN_ERR_INVALID_ARG, "sim: arrivals must be non-negative and non-decreasing (request %lld)",
                             (long long)j);
        if (prompt[j] < 1 || length[j] < 1)
            return set_error(BELLMAN_ERR_INVALID_ARG, "sim: request %lld has prompt %d, length %d", (long long)j,
                             prompt[j], length[j]);
        const int64_t need = ceil_pages((int64_t)prompt[j] + length[j]);
        if (need + cfg->watermark_pages > cfg->kv_capacity_pages)
            return set_error(BELLMAN_ERR_INVALID_ARG, "sim: request %lld needs %lld pages, budget %lld - %lld",
                             (long long)j, (long long)need, (long long)cfg->kv_capacity_pages,
                             (long long)cfg->watermark_pages);
        max_pages = std::max(max_pages, need);
        if (cfg->req_class && (cfg->req_class[j] < 0 || cfg->req_class[j] >= cfg->n_classes))
            return set_error(BELLMAN_ERR_INVALID_ARG, "sim: request %lld has class %d of %d", (long long)j,
                             cfg->req_class[j], cfg->n_classes);
    }
    memset(stats, 0, sizeof *stats);

    bellman_controller_t* ctl = nullptr;
    if (cfg->controller != BELLMAN_SIM_NO_CONTROL) {
        bellman_ctl_params_t p;
        if (cfg->ctl_params) {
            p = *cfg->ctl_params;
        } else {
            bellman_ctl_params_default(cfg->controller, cfg->t1, cfg->t2, &p);
            p.window = cfg->window;
            p.r_min = cfg->r_min;
            p.r_max = cfg->r_max;
        }
        ctl = bellman_controller_create_ex(&p);
        if (!ctl) return set_error(BELLMAN_ERR_INVALID_ARG, "sim: invalid controller parameters");
    }
    const bellman_class_policy_t default_class{1.0, 0, 0};
    const double tick_s = (double)cfg->tick_ns / 1e9;
    struct CtlGuard {
        bellman_controller_t* c;
        ~CtlGuard() {
            if (c) bellman_controller_destroy(c);
        }
    } guard{ctl};
    auto rate = [&]() { return ctl ? bellman_controller_rate(ctl) : 0.0; };

    LiveGpu gpu;
    if (cfg->live && (rc = gpu.init(cfg, max_pages))) return rc;

    const size_t N = (size_t)n;
    std::vector<int8_t> state(N, kNotArrived);
    std::vector<int32_t> target(N, 0), gen(N, 0), row_of(N, -1);
    std::vector<int64_t> todo(N, 0), filled(N, 0);
    std::vector<std::vector<int32_t>> pages_of(N);  // pages held, in KV order
    std::vector<int32_t> req_of((size_t)cfg->max_running, -1);
    std::vector<int32_t> free_pages((size_t)cfg->kv_capacity_pages);
    for (int64_t p = 0; p < cfg->kv_capacity_pages; ++p) free_pages[(size_t)p] = (int32_t)(cfg->kv_capacity_pages - 1 - p);
    for (int64_t j = 0; j < n; ++j) requests[j] = bellman_sim_request_t{-1, -1, -1, 0, 0, 0.0};

    std::deque<int64_t> queue;
    std::vector<int64_t> running, still, back;
    std::vector<char> completing(N, 0);
    std::map<int64_t, std::pair<int64_t, int64_t>> windows;  // tick index -> (TBT sum, samples)
    int64_t now = 0, next_tick = cfg->tick_ns, i = 0, done = 0;
    int rows = 0;  // live: rows [0, rows) of the device batch hold the decoding requests

    auto take_page = [&](int64_t j) {
        const int32_t p = free_pages.back();
        free_pages.pop_back();
        pages_of[(size_t)j].push_back(p);
        if (cfg->live && row_of[(size_t)j] >= 0) {
            const int r = row_of[(size_t)j];
            gpu.bt_h[(int64_t)r * gpu.maxP + (int64_t)pages_of[(size_t)j].size() - 1] = p;
            gpu.dirty[(size_t)r] = 1;
        }
    };
    auto drop_row = [&](int64_t j) {  // live: the last row takes the freed row's place
        if (!cfg->live || row_of[(size_t)j] < 0) return;
        const int r = row_of[(size_t)j], last = rows - 1;
        if (r != last) {
            const int32_t m = req_of[(size_t)last];
            memcpy(gpu.bt_h + (int64_t)r * gpu.maxP, gpu.bt_h + (int64_t)last * gpu.maxP, (size_t)gpu.maxP * 4);
            gpu.dirty[(size_t)r] = 1;
            req_of[(size_t)r] = m;
            row_of[(size_t)m] = r;
        }
        req_of[(size_t)last] = -1;
        row_of[(size_t)j] = -1;
        --rows;
    };
    auto add_row = [&](int64_t j) {
        if (!cfg->live) return;
        const int r = rows++;
        row_of[(size_t)j] = r;
        req_of[(size_t)r] = (int32_t)j;
        int32_t* row = gpu.bt_h + (int64_t)r * gpu.maxP;
        const auto& pg = pages_of[(size_t)j];
        for (int64_t k = 0; k < gpu.maxP; ++k) row[k] = k < (int64_t)pg.size() ? pg[(size_t)k] : -1;
        gpu.dirty[(size_t)r] = 1;
    };
    auto release_pages = [&](int64_t j) {
        for (int32_t p : pages_of[(size_t)j]) free_pages.push_back(p);
        pages_of[(size_t)j].clear();
    };

    while (done < n) {
        // 1. ticks and arrivals up to now, in time order (a tick first on ties)
        for (;;) {
            const bool more = i < n;
            if (next_tick <= now && (!more || next_tick <= arrival_ns[i])) {
                auto it = windows.find(next_tick / cfg->tick_ns);
                int64_t s = 0, c = 0;
                if (it != windows.end()) {
                    s = it->second.first;
                    c = it->second.second;
                    windows.erase(it);
                }
                if (ctl) {
                    const bellman_ctl_obs_t obs{c > 0 ? 1 : 0, 0, c > 0 ? (double)s / (double)c : 0.0, (double)c, tick_s};
                    if (bellman_controller_observe(ctl, &obs) < 0.0)
                        return set_error(BELLMAN_ERR_INVALID_ARG, "sim: controller rejected a tick");
                }
                if (stats->ticks < max_ticks)
                    ticks[stats->ticks] = bellman_sim_tick_t{next_tick, c, s, rate(), (int32_t)queue.size(), (int32_t)running.size()};
                ++stats->ticks;
                next_tick += cfg->tick_ns;
                continue;
            }
            if (more && arrival_ns[i] <= now) {
                int32_t Nt = length[i];
                if (ctl) {
                    const int32_t k = cfg->req_class ? cfg->req_class[i] : 0;
                    Nt = bellman_length_cap_class(ctl, length[i], cfg->classes ? &cfg->classes[k] : &default_class);
                    if (Nt < 0) return set_error(BELLMAN_ERR_INVALID_ARG, "sim: length cap failed");
                }
                target[(size_t)i] = Nt;
                requests[i].target = Nt;
                requests[i].r_at_queue = rate();
                state[(size_t)i] = kQueued;
                queue.push_back(i);
                ++i;
                continue;
            }
            break;
        }
        // 2. first-come first-served admission
        while (!queue.empty() && (int64_t)running.size() < cfg->max_running) {
            const int64_t j = queue.front();
            const int64_t P = (int64_t)prompt[j] + gen[(size_t)j];
            const int64_t need = ceil_pages(P);
            if ((int64_t)free_pages.size() - need < cfg->watermark_pages) break;
            queue.pop_front();
            for (int64_t k = 0; k < need; ++k) take_page(j);
            todo[(size_t)j] = P;
            filled[(size_t)j] = 0;
            state[(size_t)j] = kPrefill;
            running.push_back(j);
            if (requests[j].admit_ns < 0) requests[j].admit_ns = now;
        }
        // 3. idle: jump to the next arrival
        if (running.empty()) {
            now = arrival_ns[i];
            continue;
        }
        const int32_t run0 = (int32_t)running.size(), queued0 = (int32_t)queue.size();
        // 4. pages for the decodes; preempt the latest admitted when none is free
        for (size_t k = 0; k < running.size();) {
            const int64_t j = running[k];
            if (state[(size_t)j] == kDecode &&
                ((int64_t)prompt[j] + gen[(size_t)j] - 1) / kPage >= (int64_t)pages_of[(size_t)j].size()) {
                bool self = false;
                back.clear();
                while (free_pages.empty()) {
                    const int64_t v = running.back();
                    running.pop_back();
                    drop_row(v);
                    release_pages(v);
                    state[(size_t)v] = kQueued;
                    ++requests[v].preemptions;
                    ++stats->preemptions;
                    back.push_back(v);
                    if (v == j) {
                        self = true;
                        break;
                    }
                }
                for (int64_t v : back) queue.push_front(v);
                if (self) continue;  // j is gone and was the last running request
                take_page(j);
            }
            ++k;
        }
        // 5. prefill chunks
        int64_t budget = cfg->prefill_chunk_tokens > 0 ? cfg->prefill_chunk_tokens : INT64_MAX;
        int64_t chunk = 0;
        for (int64_t j : running) {
            if (state[(size_t)j] != kPrefill) continue;
            const int64_t t = std::min(todo[(size_t)j] - filled[(size_t)j], budget);
            filled[(size_t)j] += t;
            budget -= t;
            chunk += t;
            if (filled[(size_t)j] == todo[(size_t)j]) completing[(size_t)j] = 1;
            if (budget == 0) break;
        }
        // 6. iteration time
        int64_t kv = 0, decoding = 0;
        for (int64_t j : running)
            if (state[(size_t)j] == kDecode) {
                kv += (int64_t)prompt[j] + gen[(size_t)j];
                ++decoding;
            }
        int64_t dt;
        if (cfg->live) {
            int64_t attn_ns = 0;
            if (rows > 0) {
                for (int r = 0; r < rows; ++r) {
                    const int32_t j = req_of[(size_t)r];
                    gpu.sl_h[r] = prompt[j] + gen[(size_t)j] - 1;  // KV length before this step's append
                }
                double ms = 0.0;
                if ((rc = gpu.step(rows, &ms))) return rc;
                stats->live_gpu_ms += ms;
                stats->live_kv_bytes += kv * cfg->live_kv_heads * cfg->live_head_dim * 2 * 2;
                attn_ns = llround(ms * 1e6) * cfg->live_layers;
            }
            dt = cfg->fixed_ns + attn_ns + cfg->prefill_ps_per_token * chunk / 1000;
        } else {
            dt = cfg->fixed_ns + (cfg->attn_ps_per_token * kv + cfg->prefill_ps_per_token * chunk) / 1000;
        }
        const int64_t end = now + dt;
        // 7. tokens and finishes
        if (decoding > 0) {
            auto& w = windows[(end + cfg->tick_ns - 1) / cfg->tick_ns];
            w.first += dt * decoding;
            w.second += decoding;
        }
        still.clear();
        for (int64_t j : running) {
            const size_t u = (size_t)j;
            if (state[u] == kDecode) {
                ++gen[u];
            } else if (completing[u]) {
                completing[u] = 0;
                ++gen[u];
                if (requests[j].first_ns < 0) requests[j].first_ns = end;
                state[u] = kDecode;
                add_row(j);
            }
            if (state[u] == kDecode && gen[u] >= target[u]) {
                requests[j].finish_ns = end;
                drop_row(j);
                release_pages(j);
                state[u] = kDone;
                ++done;
            } else {
                still.push_back(j);
            }
        }
        if (stats->iterations < max_iterations)
            iterations[stats->iterations] =
                bellman_sim_iteration_t{end, dt, (int32_t)decoding, (int32_t)chunk, run0, queued0};
        running.swap(still);
        now = end;
        ++stats->iterations;
    }
    stats->end_ns = now;
    if (cfg->live) {
        int32_t flags = 0;
        if ((rc = bellman_device_errors(gpu.s, &flags))) return rc;
        if (flags) return set_error(BELLMAN_ERR_HIP, "sim: device error flags 0x%x after the live run", flags);
    }
    return 0;
}
