// Task Scheduler and activation-queue pool (Alg. 2 put(), Alg. 3 get(),
// activation flow control of Sec. 3.4.1, versions of Alg. 4).
//
// All state is host-side and O(K); the only device work is the copy of an
// admitted batch into its preallocated slot and the aggregation kernels,
// both ordered on the pool's stream.
//
// Every entry point takes the pool's own lock, so that the Receiver side
// (pushes of activations and models) and the Compute Engine side (picks,
// releases, aggregations) may run on different host threads.
//
// Live pools are kept in a registry so that a training step whose batch lies
// in a pool slot can be checked against that pool's last pick, and so that a
// step enqueued on a stream other than the pool's is ordered before the
// slot's next reuse (an event recorded after the step, waited for by the
// pool's stream before its next copy into that slot).
#include <algorithm>
#include <atomic>
#include <deque>
#include <mutex>
#include <unordered_map>
#include <vector>

#include "kernels.h"
#include "pool.h"

namespace fo {
std::atomic<int64_t> g_max_delay{-1};
}

struct fo_queues {
    int32_t K = 0;
    int64_t slot_bytes = 0;
    int32_t batch = 0;
    int32_t with_lengths = 0;
    int64_t n_slots = 0, omega = 0;
    hipStream_t stream = nullptr;
    char* slab = nullptr;
    int32_t* labels = nullptr;
    int32_t* lengths = nullptr;

    mutable std::mutex mu;
    int32_t policy = FO_SCHED_COUNTER;

    struct Item { int64_t seq, slot, order; };  // order: admission index over all devices
    std::vector<std::deque<Item>> q;
    std::vector<int64_t> c, next_seq;
    std::vector<uint8_t> sender_on;
    std::vector<uint8_t> active;  // 0 while a device has left
    std::vector<int64_t> free_stack;

    bool busy = false;  // a batch is in service
    int32_t svc_k = -1;
    Item svc{-1, -1, -1};

    struct ModelMsg { int32_t k; const float* local; int64_t n; int64_t t_k; };
    std::deque<ModelMsg> qm;

    int64_t t = 0, queued = 0, admitted = 0, refused = 0, picks = 0, peak = 0, turn_ons = 0;

    // Optional record of every state transition, four int64 per event
    // (type, device, a, b), reserved up front so recording never allocates.
    int64_t log_cap = 0;
    std::vector<int64_t> log;
    void log_ev(int64_t type, int64_t k, int64_t a, int64_t b) {
        if ((int64_t)log.size() < 4 * log_cap) {
            log.push_back(type);
            log.push_back(k);
            log.push_back(a);
            log.push_back(b);
        }
    }

    // Slot reuse across streams: svc_ev is recorded after a step that read the
    // batch in service from another stream; on release it guards that slot,
    // and the next push into the slot makes the pool's stream wait for it.
    hipEvent_t svc_ev = nullptr;
    hipEvent_t ready_ev = nullptr;  // the other direction: the step waits for the copies into its slot
    std::unordered_map<int64_t, hipEvent_t> guard;
    std::vector<hipEvent_t> ev_free;

    bool in_slab(const void* p) const {
        const char* c = (const char*)p;
        return slab && c >= slab && c < slab + slot_bytes * n_slots;
    }
    bool in_labels(const void* p) const {
        const int32_t* c = (const int32_t*)p;
        return labels && c >= labels && c < labels + (int64_t)batch * n_slots;
    }

    // after an enqueue to or dequeue from Q_k: below the cap, an off Sender of a
    // present device gets a 'turn-on' signal
    void turn_on_check(int32_t k) {
        if (active[k] && !sender_on[k] && queued < omega) {
            sender_on[k] = 1;
            turn_ons++;
        }
    }
};

using fo::set_error;

namespace {
std::mutex g_pools_mu;
std::vector<fo_queues*> g_pools;  // every pool between create and destroy
}  // namespace

extern "C" fo_status fo_queues_create(int32_t K, int64_t slot_bytes, int32_t batch, int32_t with_lengths,
                                      int64_t n_slots, void* hip_stream, fo_queues** out) {
    FO_CHECK(out != nullptr, "fo_queues_create: out is NULL");
    *out = nullptr;
    FO_CHECK(K >= 1, "fo_queues_create: K=%d must be >= 1", K);
    FO_CHECK(n_slots > K, "fo_queues_create: n_slots=%lld must exceed K=%d", (long long)n_slots, K);
    FO_CHECK(batch >= 1, "fo_queues_create: batch=%d must be >= 1", batch);
    FO_CHECK(slot_bytes >= 0 && slot_bytes % 16 == 0, "fo_queues_create: slot_bytes=%lld must be a multiple of 16",
             (long long)slot_bytes);
    fo_queues* q = new (std::nothrow) fo_queues();
    if (!q) return FO_ENOMEM;
    q->K = K;
    q->slot_bytes = slot_bytes;
    q->batch = batch;
    q->with_lengths = with_lengths ? 1 : 0;
    q->n_slots = n_slots;
    q->omega = n_slots - K;
    q->stream = (hipStream_t)hip_stream;
    try {  // host bookkeeping: O(K + n_slots); never let an exception cross the C ABI
        q->q.resize(K);
        q->c.assign(K, 0);
        q->next_seq.assign(K, 0);
        q->sender_on.assign(K, 1);
        q->active.assign(K, 1);
        q->free_stack.reserve(n_slots);
        for (int64_t s = n_slots - 1; s >= 0; --s) q->free_stack.push_back(s);
    } catch (...) {
        set_error("fo_queues_create: host bookkeeping for %lld slots does not fit", (long long)n_slots);
        delete q;
        return FO_ENOMEM;
    }
    if (slot_bytes > 0) {
        hipError_t e = hipMalloc((void**)&q->slab, (size_t)slot_bytes * (size_t)n_slots);
        if (e == hipSuccess) e = hipMalloc((void**)&q->labels, sizeof(int32_t) * (size_t)batch * (size_t)n_slots);
        if (e == hipSuccess && q->with_lengths)
            e = hipMalloc((void**)&q->lengths, sizeof(int32_t) * (size_t)batch * (size_t)n_slots);
        if (e != hipSuccess) {
            set_error("fo_queues_create: device pool of %lld slots x %lld bytes: %s", (long long)n_slots,
                      (long long)slot_bytes, hipGetErrorString(e));
            fo_queues_destroy(q);
            return e == hipErrorOutOfMemory ? FO_ENOMEM : FO_EHIP;
        }
    }
    try {
        std::lock_guard<std::mutex> lk(g_pools_mu);
        g_pools.push_back(q);
    } catch (...) {
        set_error("fo_queues_create: out of host memory");
        fo_queues_destroy(q);
        return FO_ENOMEM;
    }
    *out = q;
    return FO_OK;
}

extern "C" void fo_queues_destroy(fo_queues* q) {
    if (!q) return;
    {
        std::lock_guard<std::mutex> lk(g_pools_mu);
        for (size_t i = 0; i < g_pools.size(); ++i)
            if (g_pools[i] == q) {
                g_pools.erase(g_pools.begin() + i);
                break;
            }
    }
    if (q->slab || q->svc_ev || !q->guard.empty()) (void)hipStreamSynchronize(q->stream);
    if (q->svc_ev) {
        (void)hipEventSynchronize(q->svc_ev);
        (void)hipEventDestroy(q->svc_ev);
    }
    for (auto& kv : q->guard) {
        (void)hipEventSynchronize(kv.second);
        (void)hipEventDestroy(kv.second);
    }
    for (hipEvent_t e : q->ev_free) (void)hipEventDestroy(e);
    if (q->ready_ev) (void)hipEventDestroy(q->ready_ev);
    if (q->slab) (void)hipFree(q->slab);
    if (q->labels) (void)hipFree(q->labels);
    if (q->lengths) (void)hipFree(q->lengths);
    delete q;
}

namespace fo {

fo_status pool_step_begin(const fo_acts* acts, const int32_t* labels, int32_t device_id, hipStream_t step_stream,
                          fo_queues** owner) {
    *owner = nullptr;
    std::lock_guard<std::mutex> lk(g_pools_mu);
    for (fo_queues* q : g_pools) {
        const bool x_in = q->in_slab(acts->x), lab_in = q->in_labels(labels);
        if (!x_in && !lab_in) continue;
        std::lock_guard<std::mutex> ql(q->mu);
        FO_CHECK(q->busy, "fo_server_step: the batch lies in a pool slot that is not in service");
        const char* x_svc = q->slab + q->svc.slot * q->slot_bytes;
        const int32_t* lab_svc = q->labels + q->svc.slot * q->batch;
        FO_CHECK(acts->x == x_svc, "fo_server_step: the activations lie in pool slot memory other than the "
                 "batch in service (slot %lld)", (long long)q->svc.slot);
        FO_CHECK(labels == lab_svc, "fo_server_step: the labels are not those of the batch in service (slot %lld)",
                 (long long)q->svc.slot);
        FO_CHECK(!q->lengths || acts->lengths == q->lengths + q->svc.slot * q->batch,
                 "fo_server_step: the lengths are not those of the batch in service (slot %lld)",
                 (long long)q->svc.slot);
        FO_CHECK(device_id == q->svc_k, "fo_server_step: device_id=%d, but the batch in service came from "
                 "device %d (the last pick)", device_id, q->svc_k);
        if (step_stream != q->stream) {  // the step reads the slot after the copies into it
            if (!q->ready_ev) FO_HIP(hipEventCreateWithFlags(&q->ready_ev, hipEventDisableTiming));
            FO_HIP(hipEventRecord(q->ready_ev, q->stream));
            FO_HIP(hipStreamWaitEvent(step_stream, q->ready_ev, 0));
        }
        *owner = q;
        return FO_OK;
    }
    return FO_OK;
}

void pool_geometry(const fo_queues* q, int64_t* slot_bytes, int32_t* batch, int32_t* with_lengths) {
    *slot_bytes = q->slot_bytes;
    *batch = q->batch;
    *with_lengths = q->with_lengths;
}
hipStream_t pool_stream(const fo_queues* q) { return q->stream; }

fo_status pool_step_done(fo_queues* q, hipStream_t step_stream) {
    if (step_stream == q->stream) return FO_OK;  // stream order already keeps the reuse after the step
    std::lock_guard<std::mutex> lk(q->mu);
    if (!q->svc_ev) {
        if (!q->ev_free.empty()) {
            q->svc_ev = q->ev_free.back();
            q->ev_free.pop_back();
        } else {
            FO_HIP(hipEventCreateWithFlags(&q->svc_ev, hipEventDisableTiming));
        }
    }
    FO_HIP(hipEventRecord(q->svc_ev, step_stream));
    return FO_OK;
}

}  // namespace fo

namespace {

// put() bookkeeping of one activation batch from device k (Alg. 2, Sec. 3.4.1):
// FO_FULL when the Sender Status is off (the batch never arrives), else the
// slot it goes to (*slot_out), with the pool's stream ordered after any step
// on another stream that last read that slot.
fo_status admit(fo_queues* q, int32_t k, int64_t* slot_out) {
    if (!q->sender_on[k]) {
        q->refused++;
        q->log_ev(FO_EV_PUSH, k, 0, -1);
        return FO_FULL;
    }
    if (q->free_stack.empty()) {  // cannot happen while omega = n_slots - K holds
        fo::set_error("fo_queues_push: pool exhausted (internal invariant broken)");
        return FO_ESTATE;
    }
    const int64_t slot = q->free_stack.back();
    auto g = q->guard.find(slot);
    if (g != q->guard.end()) {  // a step on another stream read this slot: copy after it
        FO_HIP(hipStreamWaitEvent(q->stream, g->second, 0));
        q->ev_free.push_back(g->second);
        q->guard.erase(g);
    }
    try {
        q->q[k].push_back({q->next_seq[k], slot, q->admitted});
    } catch (...) {
        set_error("fo_queues_push: out of host memory");
        return FO_ENOMEM;
    }
    q->next_seq[k]++;
    q->free_stack.pop_back();
    q->queued++;
    q->admitted++;
    if (q->queued > q->peak) q->peak = q->queued;
    q->sender_on[k] = 0;   // deactivated until the server turns it on
    q->log_ev(FO_EV_PUSH, k, 1, q->next_seq[k] - 1);
    q->turn_on_check(k);   // enqueue: below the cap -> 'turn-on'
    *slot_out = slot;
    return FO_OK;
}

}  // namespace

extern "C" fo_status fo_queues_push(fo_queues* q, int32_t k, const void* x_src, const int32_t* labels_src,
                                    const int32_t* lengths_src, int32_t src_on_host) {
    FO_CHECK(q != nullptr, "fo_queues_push: NULL handle");
    std::lock_guard<std::mutex> lk(q->mu);
    FO_CHECK(k >= 0 && k < q->K, "fo_queues_push: device %d out of range [0,%d)", k, q->K);
    if (q->slab) {
        FO_CHECK(x_src != nullptr && labels_src != nullptr, "fo_queues_push: NULL source");
        FO_CHECK(!q->with_lengths || lengths_src != nullptr, "fo_queues_push: this pool needs lengths");
    }
    int64_t slot = -1;
    fo_status st = admit(q, k, &slot);
    if (st != FO_OK || !q->slab) return st;
    char* xd = q->slab + slot * q->slot_bytes;
    int32_t* ld = q->labels + slot * q->batch;
    int32_t* nd = q->with_lengths ? q->lengths + slot * q->batch : nullptr;
    if (!src_on_host && ((uintptr_t)x_src & 15) == 0)  // device sources: one launch for the three parts
        return fo::launch_pool_put(x_src, xd, q->slot_bytes, labels_src, ld, nd ? lengths_src : nullptr, nd, q->batch,
                                   q->stream);
    hipMemcpyKind kind = src_on_host ? hipMemcpyHostToDevice : hipMemcpyDeviceToDevice;
    FO_HIP(hipMemcpyAsync(xd, x_src, (size_t)q->slot_bytes, kind, q->stream));
    FO_HIP(hipMemcpyAsync(ld, labels_src, sizeof(int32_t) * q->batch, kind, q->stream));
    if (nd) FO_HIP(hipMemcpyAsync(nd, lengths_src, sizeof(int32_t) * q->batch, kind, q->stream));
    return FO_OK;
}

extern "C" fo_status fo_queues_push_batch(fo_queues* q, int32_t n, const int32_t* k, const void* const* x_src,
                                          const int32_t* const* labels_src, const int32_t* const* lengths_src,
                                          int32_t* status_out) {
    FO_CHECK(q != nullptr, "fo_queues_push_batch: NULL handle");
    std::lock_guard<std::mutex> lk(q->mu);
    FO_CHECK(n >= 0 && (n == 0 || k != nullptr), "fo_queues_push_batch: n=%d", n);
    for (int32_t i = 0; i < n; ++i) {  // every argument checked before any state changes
        FO_CHECK(k[i] >= 0 && k[i] < q->K, "fo_queues_push_batch: entry %d: device %d out of range [0,%d)", i, k[i],
                 q->K);
        if (q->slab) {
            FO_CHECK(x_src && labels_src && x_src[i] && labels_src[i], "fo_queues_push_batch: entry %d: NULL source",
                     i);
            FO_CHECK(((uintptr_t)x_src[i] & 15) == 0, "fo_queues_push_batch: entry %d: activations not 16-byte aligned",
                     i);
            FO_CHECK(!q->with_lengths || (lengths_src && lengths_src[i]),
                     "fo_queues_push_batch: entry %d: this pool needs lengths", i);
        }
    }
    fo::PutTable t;
    t.count = 0;
    auto flush = [&]() -> fo_status {
        if (t.count == 0) return FO_OK;
        fo_status st = fo::launch_pool_put_gather(t, q->slot_bytes, q->batch, q->stream);
        t.count = 0;
        return st;
    };
    for (int32_t i = 0; i < n; ++i) {
        int64_t slot = -1;
        fo_status st = admit(q, k[i], &slot);
        if (status_out) status_out[i] = st == FO_FULL ? FO_FULL : FO_OK;
        if (st == FO_FULL) continue;
        if (st != FO_OK) return st;
        if (!q->slab) continue;
        const int e = t.count++;
        t.xs[e] = (const uint4*)x_src[i];
        t.xd[e] = (uint4*)(q->slab + slot * q->slot_bytes);
        t.ls[e] = labels_src[i];
        t.ld[e] = q->labels + slot * q->batch;
        t.ns[e] = q->with_lengths ? lengths_src[i] : nullptr;
        t.nd[e] = q->with_lengths ? q->lengths + slot * q->batch : nullptr;
        if (t.count == fo::kPutMaxBatches) {
            st = flush();
            if (st != FO_OK) return st;
        }
    }
    return flush();
}

extern "C" fo_status fo_queues_push_model(fo_queues* q, int32_t k, const float* local, int64_t n, int64_t t_k) {
    FO_CHECK(q != nullptr, "fo_queues_push_model: NULL handle");
    std::lock_guard<std::mutex> lk(q->mu);
    FO_CHECK(k >= 0 && k < q->K, "fo_queues_push_model: device %d out of range [0,%d)", k, q->K);
    FO_CHECK(n >= 0 && (n == 0 || local != nullptr), "fo_queues_push_model: bad vector");
    FO_CHECK(t_k >= 0, "fo_queues_push_model: negative version");
    try {
        q->qm.push_back({k, local, n, t_k});
        q->log_ev(FO_EV_MODEL, k, t_k, 0);
    } catch (...) {
        set_error("fo_queues_push_model: out of host memory");
        return FO_ENOMEM;
    }
    return FO_OK;
}

extern "C" fo_status fo_queues_push_model_batch(fo_queues* q, int32_t n, const int32_t* k, const float* const* local,
                                                int64_t len, const int64_t* t_k) {
    FO_CHECK(q != nullptr, "fo_queues_push_model_batch: NULL handle");
    std::lock_guard<std::mutex> lk(q->mu);
    FO_CHECK(n >= 0 && (n == 0 || (k != nullptr && t_k != nullptr)), "fo_queues_push_model_batch: n=%d", n);
    FO_CHECK(len >= 0 && (len == 0 || n == 0 || local != nullptr), "fo_queues_push_model_batch: bad vectors");
    for (int32_t i = 0; i < n; ++i) {
        FO_CHECK(k[i] >= 0 && k[i] < q->K, "fo_queues_push_model_batch: entry %d: device %d out of range", i, k[i]);
        FO_CHECK(t_k[i] >= 0, "fo_queues_push_model_batch: entry %d: negative version", i);
        FO_CHECK(len == 0 || local[i] != nullptr, "fo_queues_push_model_batch: entry %d: NULL vector", i);
    }
    try {
        for (int32_t i = 0; i < n; ++i) {
            q->qm.push_back({k[i], len ? local[i] : nullptr, len, t_k[i]});
            q->log_ev(FO_EV_MODEL, k[i], t_k[i], 0);
        }
    } catch (...) {
        set_error("fo_queues_push_model_batch: out of host memory");
        return FO_ENOMEM;
    }
    return FO_OK;
}

extern "C" int32_t fo_pick_device(fo_queues* q) {
    if (!q) {
        fo::set_error("fo_pick_device: NULL handle");
        return -3;
    }
    std::lock_guard<std::mutex> lk(q->mu);
    if (!q->qm.empty()) return -2;  // Alg. 3: models are served first
    if (q->busy) {
        fo::set_error("fo_pick_device: release the batch in service first");
        return -3;
    }
    int32_t best = -1;
    for (int32_t k = 0; k < q->K; ++k) {
        if (q->q[k].empty()) continue;
        if (best < 0 ||
            (q->policy == FO_SCHED_COUNTER ? q->c[k] < q->c[best]
                                           : q->q[k].front().order < q->q[best].front().order))
            best = k;
    }
    if (best < 0) return -1;
    q->svc = q->q[best].front();
    q->q[best].pop_front();
    q->svc_k = best;
    q->busy = true;
    q->queued--;
    q->c[best]++;
    q->picks++;
    q->log_ev(FO_EV_PICK, best, q->svc.seq, q->svc.slot);
    q->turn_on_check(best);  // dequeue: below the cap -> 'turn-on'
    return best;
}

extern "C" fo_status fo_queues_in_service(fo_queues* q, fo_acts* acts_out, const int32_t** labels_out,
                                          int64_t* seq_out, int64_t* slot_out) {
    FO_CHECK(q != nullptr, "fo_queues_in_service: NULL handle");
    std::lock_guard<std::mutex> lk(q->mu);
    if (!q->busy) {
        fo::set_error("fo_queues_in_service: no batch in service");
        return FO_ESTATE;
    }
    if (acts_out) {
        acts_out->x = q->slab ? q->slab + q->svc.slot * q->slot_bytes : nullptr;
        acts_out->lengths = q->lengths ? q->lengths + q->svc.slot * q->batch : nullptr;
        acts_out->batch = q->batch;
    }
    if (labels_out) *labels_out = q->labels ? q->labels + q->svc.slot * q->batch : nullptr;
    if (seq_out) *seq_out = q->svc.seq;
    if (slot_out) *slot_out = q->svc.slot;
    return FO_OK;
}

extern "C" fo_status fo_queues_release(fo_queues* q) {
    FO_CHECK(q != nullptr, "fo_queues_release: NULL handle");
    std::lock_guard<std::mutex> lk(q->mu);
    if (!q->busy) {
        fo::set_error("fo_queues_release: no batch in service");
        return FO_ESTATE;
    }
    if (q->svc_ev) {
        try {
            q->guard.emplace(q->svc.slot, q->svc_ev);
        } catch (...) {  // cannot keep the guard: order the pool's stream after the step now
            FO_HIP(hipStreamWaitEvent(q->stream, q->svc_ev, 0));
            q->ev_free.push_back(q->svc_ev);
        }
        q->svc_ev = nullptr;
    }
    q->free_stack.push_back(q->svc.slot);
    q->log_ev(FO_EV_RELEASE, q->svc_k, q->svc.seq, q->svc.slot);
    q->busy = false;
    q->svc_k = -1;
    return FO_OK;
}

static fo_status check_global(const fo_vec* global, const char* who) {
    FO_CHECK(global != nullptr, "%s: NULL global", who);
    FO_CHECK(global->n >= 0, "%s: negative length", who);
    FO_CHECK(global->n == 0 || ((uintptr_t)global->ptr % 16 == 0), "%s: global not 16-byte aligned", who);
    return FO_OK;
}

extern "C" fo_status fo_aggregate_pending(fo_queues* q, fo_vec* global, float alpha, int32_t* k_out,
                                          int64_t* staleness_out) {
    FO_CHECK(q != nullptr, "fo_aggregate_pending: NULL handle");
    std::lock_guard<std::mutex> lk(q->mu);
    fo_status st = check_global(global, "fo_aggregate_pending");
    if (st != FO_OK) return st;
    FO_CHECK(alpha >= 0.f && alpha <= 1.f, "fo_aggregate_pending: alpha=%g outside [0,1]", (double)alpha);
    if (q->qm.empty()) return FO_EMPTY;
    fo_queues::ModelMsg m = q->qm.front();
    FO_CHECK(m.n == global->n, "fo_aggregate_pending: model length %lld != global %lld", (long long)m.n,
             (long long)global->n);
    FO_CHECK(m.n == 0 || (uintptr_t)m.local % 16 == 0, "fo_aggregate_pending: local not 16-byte aligned");
    const int64_t s = q->t - m.t_k;
    // a failed check leaves the message at the head of the FIFO
    FO_CHECK(s >= 0, "fo_aggregate_pending: model version %lld is newer than the global %lld", (long long)m.t_k,
             (long long)q->t);
    if (k_out) *k_out = m.k;
    if (staleness_out) *staleness_out = s;
    int64_t D = fo::g_max_delay.load();
    if (D >= 0 && s > D) {
        q->qm.pop_front();
        q->log_ev(FO_EV_AGG, m.k, 0, s);
        return FO_SKIPPED;
    }
    float w = alpha / (float)(s + 1);
    st = fo::launch_agg_lerp(global->ptr, m.local, global->n, w, q->stream);
    if (st != FO_OK) return st;  // not applied: the message stays queued and t is unchanged
    q->qm.pop_front();
    q->t++;
    q->log_ev(FO_EV_AGG, m.k, 1, s);
    return FO_OK;
}

namespace {

// The fused drain of every pending model message, under the pool's lock;
// devices (if given) receives the device of every message drained, in order.
fo_status drain_models(fo_queues* q, fo_vec* global, float alpha, int32_t* applied_out, int32_t* skipped_out,
                       std::vector<int32_t>* devices) {
    fo_status st = check_global(global, "fo_aggregate_pending_all");
    if (st != FO_OK) return st;
    FO_CHECK(alpha >= 0.f && alpha <= 1.f, "fo_aggregate_pending_all: alpha=%g outside [0,1]", (double)alpha);
    int64_t D = fo::g_max_delay.load();
    {   // validate the whole FIFO before launching anything
        int64_t t_sim = q->t;
        for (const auto& m : q->qm) {
            FO_CHECK(m.n == global->n, "fo_aggregate_pending_all: model length %lld != global %lld",
                     (long long)m.n, (long long)global->n);
            FO_CHECK(m.n == 0 || (uintptr_t)m.local % 16 == 0,
                     "fo_aggregate_pending_all: local not 16-byte aligned");
            int64_t s = t_sim - m.t_k;
            FO_CHECK(s >= 0, "fo_aggregate_pending_all: model version %lld is newer than the global %lld",
                     (long long)m.t_k, (long long)t_sim);
            if (!(D >= 0 && s > D)) t_sim++;
        }
    }
    // Each launch takes up to kAggMaxFused applied messages (and the stale ones
    // between them).  The FIFO and t advance only past messages whose launch was
    // enqueued, so a failing launch leaves them consistent with what the global
    // model received.
    int32_t applied = 0, skipped = 0;
    if (applied_out) *applied_out = 0;
    if (skipped_out) *skipped_out = 0;
    while (!q->qm.empty()) {
        fo::AggTable tab;
        tab.count = 0;
        size_t used = 0;
        int64_t t_next = q->t;
        int32_t skipped_here = 0;
        while (used < q->qm.size() && tab.count < fo::kAggMaxFused) {
            const fo_queues::ModelMsg& m = q->qm[used];
            const int64_t s = t_next - m.t_k;
            ++used;
            if (D >= 0 && s > D) {
                skipped_here++;
                continue;
            }
            tab.local[tab.count] = m.local;
            tab.w[tab.count] = alpha / (float)(s + 1);
            tab.count++;
            t_next++;
        }
        if (devices) {  // room for this group's devices before anything is launched
            try {
                devices->reserve(devices->size() + used);
            } catch (...) {
                set_error("fo_aggregate_pending_all: out of host memory");
                return FO_ENOMEM;
            }
        }
        if (tab.count > 0) {
            st = fo::launch_agg_lerp_multi(global->ptr, tab, global->n, q->stream);
            if (st != FO_OK) return st;
        }
        {
            int64_t tl = q->t;
            for (size_t i = 0; i < used; ++i) {
                const int64_t s = tl - q->qm[i].t_k;
                const bool skip = D >= 0 && s > D;
                q->log_ev(FO_EV_AGG, q->qm[i].k, skip ? 0 : 1, s);
                if (!skip) tl++;
            }
        }
        if (devices)
            for (size_t i = 0; i < used; ++i) devices->push_back(q->qm[i].k);
        q->qm.erase(q->qm.begin(), q->qm.begin() + used);
        q->t = t_next;
        applied += tab.count;
        skipped += skipped_here;
        if (applied_out) *applied_out = applied;
        if (skipped_out) *skipped_out = skipped;
    }
    return FO_OK;
}

}  // namespace

extern "C" fo_status fo_aggregate_pending_all(fo_queues* q, fo_vec* global, float alpha, int32_t* applied_out,
                                              int32_t* skipped_out) {
    FO_CHECK(q != nullptr, "fo_aggregate_pending_all: NULL handle");
    std::lock_guard<std::mutex> lk(q->mu);
    return drain_models(q, global, alpha, applied_out, skipped_out, nullptr);
}

namespace fo {
fo_status pool_drain_models(fo_queues* q, fo_vec* global, float alpha, int32_t* applied, int32_t* skipped,
                            std::vector<int32_t>* devices, int64_t* version) {
    std::lock_guard<std::mutex> lk(q->mu);
    fo_status st = drain_models(q, global, alpha, applied, skipped, devices);
    *version = q->t;
    return st;
}
}  // namespace fo

extern "C" fo_status fo_queues_stats(const fo_queues* q, fo_queue_stats* out) {
    FO_CHECK(q != nullptr && out != nullptr, "fo_queues_stats: NULL argument");
    std::lock_guard<std::mutex> lk(q->mu);
    out->K = q->K;
    out->n_slots = q->n_slots;
    out->omega = q->omega;
    out->queued = q->queued;
    out->in_service = q->busy ? 1 : 0;
    out->models_pending = (int64_t)q->qm.size();
    out->admitted = q->admitted;
    out->refused = q->refused;
    out->picks = q->picks;
    out->peak_queued = q->peak;
    out->version = q->t;
    out->turn_on_signals = q->turn_ons;
    int32_t present = 0;
    for (int32_t k = 0; k < q->K; ++k) present += q->active[k] ? 1 : 0;
    out->active_devices = present;
    out->policy = q->policy;
    return FO_OK;
}

extern "C" fo_status fo_queues_counters(const fo_queues* q, int64_t* c_out, int32_t K) {
    FO_CHECK(q != nullptr && c_out != nullptr, "fo_queues_counters: NULL argument");
    std::lock_guard<std::mutex> lk(q->mu);
    FO_CHECK(K >= 0 && K <= q->K, "fo_queues_counters: K=%d out of range", K);
    for (int32_t k = 0; k < K; ++k) c_out[k] = q->c[k];
    return FO_OK;
}

extern "C" int32_t fo_queues_add_device(fo_queues* q) {
    if (!q) {
        fo::set_error("fo_queues_add_device: NULL handle");
        return -1;
    }
    std::lock_guard<std::mutex> lk(q->mu);
    if (q->n_slots - (q->K + 1) < 1) {
        fo::set_error("fo_queues_add_device: pool of %lld slots cannot take another device", (long long)q->n_slots);
        return -1;
    }
    try {
        q->q.emplace_back();
        q->c.push_back(0);
        q->next_seq.push_back(0);
        q->sender_on.push_back(1);
        q->active.push_back(1);
    } catch (...) {
        fo::set_error("fo_queues_add_device: out of host memory");
        return -1;
    }
    q->K++;
    q->omega = q->n_slots - q->K;
    q->log_ev(FO_EV_JOIN, q->K - 1, 1, 0);
    return q->K - 1;
}

extern "C" fo_status fo_queues_set_policy(fo_queues* q, int32_t policy) {
    FO_CHECK(q != nullptr, "fo_queues_set_policy: NULL handle");
    FO_CHECK(policy == FO_SCHED_COUNTER || policy == FO_SCHED_FIFO, "fo_queues_set_policy: unknown policy %d",
             policy);
    std::lock_guard<std::mutex> lk(q->mu);
    q->policy = policy;
    return FO_OK;
}

extern "C" fo_status fo_queues_set_device_active(fo_queues* q, int32_t k, int32_t active) {
    FO_CHECK(q != nullptr, "fo_queues_set_device_active: NULL handle");
    std::lock_guard<std::mutex> lk(q->mu);
    FO_CHECK(k >= 0 && k < q->K, "fo_queues_set_device_active: device %d out of range [0,%d)", k, q->K);
    const uint8_t a = active ? 1 : 0;
    if (q->active[k] == a) return FO_OK;
    q->active[k] = a;
    q->sender_on[k] = a;  // leaving: off and kept off; rejoining: on, as for a new device
    q->log_ev(a ? FO_EV_JOIN : FO_EV_LEAVE, k, 0, 0);
    return FO_OK;
}

extern "C" int32_t fo_queues_sender_status(fo_queues* q, int32_t k) {
    if (!q) {
        fo::set_error("fo_queues_sender_status: NULL handle");
        return -1;
    }
    std::lock_guard<std::mutex> lk(q->mu);
    if (k < 0 || k >= q->K) {
        fo::set_error("fo_queues_sender_status: device %d out of range [0,%d)", k, q->K);
        return -1;
    }
    return q->sender_on[k];
}

extern "C" fo_status fo_queues_log_enable(fo_queues* q, int64_t max_events) {
    FO_CHECK(q != nullptr, "fo_queues_log_enable: NULL handle");
    FO_CHECK(max_events >= 0, "fo_queues_log_enable: max_events=%lld", (long long)max_events);
    std::lock_guard<std::mutex> lk(q->mu);
    std::vector<int64_t> fresh;
    try {
        fresh.reserve((size_t)(4 * max_events));
    } catch (...) {
        set_error("fo_queues_log_enable: %lld events do not fit in host memory", (long long)max_events);
        return FO_ENOMEM;
    }
    q->log.swap(fresh);
    q->log_cap = max_events;
    return FO_OK;
}

extern "C" fo_status fo_queues_log_read(fo_queues* q, int64_t* out, int64_t max_events, int64_t* n_out) {
    FO_CHECK(q != nullptr && n_out != nullptr, "fo_queues_log_read: NULL argument");
    FO_CHECK(max_events >= 0 && (max_events == 0 || out != nullptr), "fo_queues_log_read: bad buffer");
    std::lock_guard<std::mutex> lk(q->mu);
    const int64_t n = std::min<int64_t>((int64_t)q->log.size() / 4, max_events);
    for (int64_t i = 0; i < 4 * n; ++i) out[i] = q->log[i];
    *n_out = (int64_t)q->log.size() / 4;
    return FO_OK;
}

extern "C" fo_status fo_set_max_delay(int64_t max_delay) {
    fo::g_max_delay.store(max_delay < 0 ? -1 : max_delay);
    return FO_OK;
}
