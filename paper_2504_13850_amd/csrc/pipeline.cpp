// The server's concurrent structure run against emulated devices: the
// Receiver and the Compute Engine of Sec. 5.1 as two host threads sharing the
// Task Scheduler's pool (Alg. 2 put(), Alg. 3 get()), the activation flow
// control of Sec. 3.4.1, devices leaving and rejoining (Sec. 3.4.2) under the
// dropout and bandwidth variation of Sec. 6.4, and the Compute Engine of
// Alg. 4 training on one stream while its aggregations run on another.
//
// Receiver thread: device k runs local iterations (Alg. 1) of
// iter_seconds[k] x (the interval's slow-down factor) wall-clock seconds
// each.  After an iteration it puts its next activation batch if its Sender
// Status is on (else it goes on without sending), and after every H
// iterations it puts its model and waits for the server's reply (Alg. 1,
// receive of the global model) before its next iteration.  At the start of
// every interval each device is away for that interval with probability
// p_drop and, if present, draws its slow-down factor from U[1, slow_max].
//
// Compute Engine thread: get() from the Task Scheduler; pending models are
// aggregated (or skipped past the maximum delay), all of them in fused
// launches on the pool's stream, and each device is told the global version it
// now holds; an activation batch is
// trained on with fo_server_step on the model's stream, at most max_inflight
// steps ahead of the GPU; with nothing queued the engine first waits for its
// GPU work, then sleeps until a device puts something, and that sleep is the
// server's idle time.
#include <hip/hip_runtime.h>

#include <chrono>
#include <cmath>
#include <condition_variable>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "common.h"
#include "model.h"
#include "pool.h"

using fo::set_error;

namespace {

using Clock = std::chrono::steady_clock;

double secs(Clock::time_point a, Clock::time_point b) { return std::chrono::duration<double>(b - a).count(); }

// splitmix64 (Steele, Lea and Flood, 2014): a counter-based draw per
// (seed, interval, device, purpose), independent of thread timing.
uint64_t splitmix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}
double draw(uint64_t seed, int64_t interval, int32_t k, int32_t purpose) {
    const uint64_t h = splitmix64(splitmix64(splitmix64(seed) ^ (uint64_t)interval) ^ ((uint64_t)k << 2 | purpose));
    return (double)(h >> 11) * (1.0 / 9007199254740992.0);  // 53 bits -> [0, 1)
}

struct Shared {
    std::mutex mu;
    std::condition_variable cv;
    bool stop = false;
    int64_t work_epoch = 0;            // bumped after every put
    std::vector<int64_t> version;      // global version each device holds (t_k)
    std::vector<uint8_t> awaiting;     // device waits for the reply to its model
    std::vector<uint8_t> replied;      // reply arrived, not yet seen by the Receiver
    fo_status err = FO_OK;
    std::string msg;

    void fail(fo_status st, const char* who) {
        std::lock_guard<std::mutex> lk(mu);
        if (err == FO_OK) {
            err = st;
            msg = std::string(who) + ": " + fo_last_error();
        }
        stop = true;
        cv.notify_all();
    }
};

struct Geometry {
    int64_t slot_bytes;
    int32_t batch, with_lengths;
};

void receiver(fo_queues* q, const fo_pipeline_config& c, const Geometry& g, int64_t n_global, int32_t K,
              Clock::time_point start, Clock::time_point end, Shared& sh, fo_pipeline_stats& st) {
    std::vector<double> next(K, 0.0), scale(K, 1.0);
    std::vector<int64_t> iters(K, 0), sent(K, 0), rounds(K, 0);
    std::vector<uint8_t> present(K, 1);
    int64_t interval = -1;
    const char* bx = (const char*)c.bank_x;
    for (;;) {
        const double now = secs(start, Clock::now());
        if (Clock::now() >= end) break;
        {
            std::lock_guard<std::mutex> lk(sh.mu);
            if (sh.stop) break;
            for (int32_t k = 0; k < K; ++k)
                if (sh.replied[k]) {  // the global model arrived: the next iteration starts now
                    sh.replied[k] = 0;
                    next[k] = now + c.iter_seconds[k] * scale[k];
                }
        }
        const int64_t iv = (int64_t)std::floor(now / c.interval_seconds);
        if (iv != interval) {  // dropout and bandwidth draws of the new interval
            const bool first = interval < 0;
            interval = iv;
            for (int32_t k = 0; k < K; ++k) {
                const bool away = draw(c.seed, iv, k, 0) < c.p_drop;
                scale[k] = 1.0 + (c.slow_max - 1.0) * draw(c.seed, iv, k, 1);
                if (first && !away) next[k] = now + c.iter_seconds[k] * scale[k];
                if (away == !present[k]) continue;
                fo_status s = fo_queues_set_device_active(q, k, away ? 0 : 1);
                if (s != FO_OK) return sh.fail(s, "fo_pipeline_run (device leave/rejoin)");
                present[k] = away ? 0 : 1;
                if (away) {
                    if (!first) st.leaves++;
                } else {
                    st.rejoins++;
                    next[k] = now + c.iter_seconds[k] * scale[k];
                }
            }
        }
        // the earliest iteration to finish among present devices not waiting for a reply
        int32_t kmin = -1;
        {
            std::lock_guard<std::mutex> lk(sh.mu);
            for (int32_t k = 0; k < K; ++k)
                if (present[k] && !sh.awaiting[k] && (kmin < 0 || next[k] < next[kmin])) kmin = k;
        }
        const double wake = std::min(kmin >= 0 ? next[kmin] : 1e300, (interval + 1) * c.interval_seconds);
        if (wake > now) {
            std::unique_lock<std::mutex> lk(sh.mu);
            const auto until = start + std::chrono::duration_cast<Clock::duration>(std::chrono::duration<double>(wake));
            sh.cv.wait_until(lk, std::min(until, end), [&] {
                if (sh.stop) return true;
                for (int32_t k = 0; k < K; ++k)
                    if (sh.replied[k]) return true;
                return false;
            });
            continue;
        }
        if (kmin < 0) continue;
        // device kmin finished a local iteration
        const int32_t k = kmin;
        iters[k]++;
        st.device_iterations++;
        const int64_t e = (k + sent[k]) % c.bank_n;
        fo_status s = fo_queues_push(q, k, bx + e * g.slot_bytes, c.bank_labels + e * g.batch,
                                     g.with_lengths ? c.bank_lengths + e * g.batch : nullptr, 0);
        if (s == FO_OK) {
            sent[k]++;
            st.sent++;
        } else if (s == FO_FULL) {
            st.not_sent++;  // Sender off: the device goes on without sending
        } else {
            return sh.fail(s, "fo_pipeline_run (activation put)");
        }
        bool model = iters[k] % c.H == 0;
        if (model) {
            int64_t tk;
            {
                std::lock_guard<std::mutex> lk(sh.mu);
                tk = sh.version[k];
                sh.awaiting[k] = 1;  // set before the put, so the reply cannot come first
            }
            const float* local = c.local_bank + (int64_t)((k + rounds[k]) % c.n_local) * n_global;
            s = fo_queues_push_model(q, k, local, n_global, tk);
            if (s != FO_OK) return sh.fail(s, "fo_pipeline_run (model put)");
            rounds[k]++;
            st.models_sent++;
        }
        {
            std::lock_guard<std::mutex> lk(sh.mu);
            sh.work_epoch++;
        }
        sh.cv.notify_all();
        if (!model) {
            next[k] += c.iter_seconds[k] * scale[k];
            if (next[k] < now) next[k] = now;  // a Receiver that fell behind does not replay the backlog
        }
    }
    std::lock_guard<std::mutex> lk(sh.mu);
    sh.stop = true;
    sh.cv.notify_all();
}

void engine(fo_queues* q, fo_model* m, fo_vec* global, const fo_pipeline_config& c, Clock::time_point end,
            Shared& sh, fo_pipeline_stats& st, std::vector<hipEvent_t>& ring) {
    size_t head = 0, inflight = 0;  // ring[head] is the oldest step still in flight
    hipEvent_t last = nullptr;
    std::vector<int32_t> drained;
    try {
        drained.reserve(4096);
    } catch (...) {
        set_error("out of host memory");
        return sh.fail(FO_ENOMEM, "fo_pipeline_run");
    }
    for (;;) {
        int64_t seen;
        {
            std::lock_guard<std::mutex> lk(sh.mu);
            if (sh.stop) break;
            seen = sh.work_epoch;
        }
        if (Clock::now() >= end) break;
        const int32_t k = fo_pick_device(q);
        if (k == -2) {  // models first (Alg. 3), every pending one in fused launches
            int32_t applied = 0, skipped = 0;
            int64_t version = 0;
            drained.clear();
            fo_status r = fo::pool_drain_models(q, global, c.alpha, &applied, &skipped, &drained, &version);
            if (r != FO_OK) return sh.fail(r, "fo_pipeline_run (aggregation)");
            st.aggregations += applied;
            st.skipped += skipped;
            {
                std::lock_guard<std::mutex> lk(sh.mu);
                for (int32_t kk : drained) {  // each device now holds the current global model
                    sh.version[kk] = version;
                    sh.awaiting[kk] = 0;
                    sh.replied[kk] = 1;
                }
            }
            sh.cv.notify_all();
            continue;
        }
        if (k >= 0) {
            fo_acts acts;
            const int32_t* labels = nullptr;
            fo_status r = fo_queues_in_service(q, &acts, &labels, nullptr, nullptr);
            if (r == FO_OK) r = fo_server_step(m, &acts, labels, k);
            fo_status r2 = fo_queues_release(q);
            if (r != FO_OK) return sh.fail(r, "fo_pipeline_run (training step)");
            if (r2 != FO_OK) return sh.fail(r2, "fo_pipeline_run (release)");
            if (inflight == ring.size()) {  // bound the run-ahead: wait for the oldest step
                if (hipEventSynchronize(ring[head]) != hipSuccess) {
                    set_error("hipEventSynchronize failed");
                    return sh.fail(FO_EHIP, "fo_pipeline_run (run-ahead wait)");
                }
                head = (head + 1) % ring.size();
                inflight--;
            }
            const size_t slot = (head + inflight) % ring.size();
            if (hipEventRecord(ring[slot], m->stream) != hipSuccess) {
                set_error("hipEventRecord failed");
                return sh.fail(FO_EHIP, "fo_pipeline_run (step event)");
            }
            last = ring[slot];
            inflight++;
            st.steps++;
            st.samples += acts.batch;
            continue;
        }
        if (k != -1) return sh.fail(FO_ESTATE, "fo_pipeline_run (pick)");
        // nothing queued: finish the GPU work first, then sleep until a put
        if (last && hipEventSynchronize(last) != hipSuccess) {
            set_error("hipEventSynchronize failed");
            return sh.fail(FO_EHIP, "fo_pipeline_run (drain)");
        }
        head = 0;
        inflight = 0;
        const auto t0 = Clock::now();
        {
            std::unique_lock<std::mutex> lk(sh.mu);
            sh.cv.wait_until(lk, end, [&] { return sh.stop || sh.work_epoch != seen; });
        }
        st.idle_seconds += secs(t0, Clock::now());
    }
    std::lock_guard<std::mutex> lk(sh.mu);
    sh.stop = true;
    sh.cv.notify_all();
}

}  // namespace

extern "C" fo_status fo_pipeline_run(fo_queues* q, fo_model* m, fo_vec* global, const fo_pipeline_config* cfg,
                                     fo_pipeline_stats* out) {
    FO_CHECK(q && m && global && cfg && out, "fo_pipeline_run: NULL argument");
    const fo_pipeline_config& c = *cfg;
    fo_queue_stats qs;
    fo_status st0 = fo_queues_stats(q, &qs);
    if (st0 != FO_OK) return st0;
    const int32_t K = qs.K;
    Geometry g;
    fo::pool_geometry(q, &g.slot_bytes, &g.batch, &g.with_lengths);
    FO_CHECK(m->cid != 6, "fo_pipeline_run: config 6 is a device-side model");
    FO_CHECK(c.seconds > 0 && std::isfinite(c.seconds), "fo_pipeline_run: seconds=%g", c.seconds);
    FO_CHECK(c.iter_seconds != nullptr, "fo_pipeline_run: NULL iter_seconds");
    for (int32_t k = 0; k < K; ++k)
        FO_CHECK(c.iter_seconds[k] > 0 && std::isfinite(c.iter_seconds[k]), "fo_pipeline_run: iter_seconds[%d]=%g",
                 k, c.iter_seconds[k]);
    FO_CHECK(c.H >= 1, "fo_pipeline_run: H=%d", c.H);
    FO_CHECK(c.p_drop >= 0 && c.p_drop < 1, "fo_pipeline_run: p_drop=%g outside [0,1)", c.p_drop);
    FO_CHECK(c.interval_seconds > 0, "fo_pipeline_run: interval_seconds=%g", c.interval_seconds);
    FO_CHECK(c.slow_max >= 1 && std::isfinite(c.slow_max), "fo_pipeline_run: slow_max=%g", c.slow_max);
    FO_CHECK(g.slot_bytes > 0, "fo_pipeline_run: the pool holds no activation slots");
    FO_CHECK(c.bank_n >= 1 && c.bank_x && c.bank_labels && (!g.with_lengths || c.bank_lengths),
             "fo_pipeline_run: empty or incomplete activation bank");
    FO_CHECK(((uintptr_t)c.bank_x & 15) == 0, "fo_pipeline_run: bank_x not 16-byte aligned");
    FO_CHECK(g.batch <= m->max_batch, "fo_pipeline_run: pool batch %d exceeds the model's max_batch %d", g.batch,
             m->max_batch);
    FO_CHECK(c.n_local >= 1 && c.local_bank, "fo_pipeline_run: empty model bank");
    FO_CHECK(global->n >= 0 && (global->n == 0 || ((uintptr_t)c.local_bank % 16 == 0 &&
                                                   (global->n * 4) % 16 == 0)),
             "fo_pipeline_run: model vectors must keep 16-byte alignment (n %% 4 == 0)");
    FO_CHECK(c.alpha >= 0 && c.alpha <= 1, "fo_pipeline_run: alpha=%g outside [0,1]", (double)c.alpha);
    FO_CHECK(c.max_inflight >= 1 && c.max_inflight <= 64, "fo_pipeline_run: max_inflight=%d outside [1,64]",
             c.max_inflight);
    FO_CHECK(qs.in_service == 0, "fo_pipeline_run: release the batch in service first");

    *out = fo_pipeline_stats{};
    std::vector<hipEvent_t> ring(c.max_inflight, nullptr);
    for (auto& e : ring)
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
            for (auto& f : ring)
                if (f) (void)hipEventDestroy(f);
            set_error("fo_pipeline_run: hipEventCreate failed");
            return FO_EHIP;
        }
    Shared sh;
    fo_pipeline_stats rs{}, es{};
    fo_status result = FO_OK;
    const auto start = Clock::now();
    const auto end = start + std::chrono::duration_cast<Clock::duration>(std::chrono::duration<double>(c.seconds));
    try {
        sh.version.assign(K, qs.version);
        sh.awaiting.assign(K, 0);
        sh.replied.assign(K, 0);
        std::thread te(engine, q, m, global, std::cref(c), end, std::ref(sh), std::ref(es), std::ref(ring));
        std::thread tr(receiver, q, std::cref(c), std::cref(g), global->n, K, start, end, std::ref(sh),
                       std::ref(rs));
        tr.join();
        te.join();
    } catch (...) {
        set_error("fo_pipeline_run: could not start the Receiver and Compute Engine threads");
        result = FO_ENOMEM;
    }
    // the run ends when the last step and aggregation have finished on the GPU
    hipError_t e1 = hipStreamSynchronize(m->stream);
    hipError_t e2 = hipStreamSynchronize(fo::pool_stream(q));
    const auto stop = Clock::now();
    for (auto& e : ring) (void)hipEventDestroy(e);
    if (result != FO_OK) return result;
    if (sh.err != FO_OK) {
        set_error("%s", sh.msg.c_str());
        return sh.err;
    }
    if (e1 != hipSuccess || e2 != hipSuccess) {
        set_error("fo_pipeline_run: %s", hipGetErrorString(e1 != hipSuccess ? e1 : e2));
        return FO_EHIP;
    }
    *out = es;
    out->sent = rs.sent;
    out->not_sent = rs.not_sent;
    out->models_sent = rs.models_sent;
    out->leaves = rs.leaves;
    out->rejoins = rs.rejoins;
    out->device_iterations = rs.device_iterations;
    out->wall_seconds = secs(start, stop);
    return FO_OK;
}
