// Task Scheduler and activation-queue pool (Alg. 2 put(), Alg. 3 get(),
// activation flow control of Sec. 3.4.1, versions of Alg. 4).
//
// All state is host-side and O(K); the only device work is the copy of an
// admitted batch into its preallocated slot and the aggregation kernels,
// both ordered on the pool's stream.
#include <atomic>
#include <deque>
#include <vector>

#include "kernels.h"

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

    struct Item { int64_t seq, slot; };
    std::vector<std::deque<Item>> q;
    std::vector<int64_t> c, next_seq;
    std::vector<uint8_t> sender_on;
    std::vector<int64_t> free_stack;

    bool busy = false;  // a batch is in service
    int32_t svc_k = -1;
    Item svc{-1, -1};

    struct ModelMsg { int32_t k; const float* local; int64_t n; int64_t t_k; };
    std::deque<ModelMsg> qm;

    int64_t t = 0, queued = 0, admitted = 0, refused = 0, picks = 0, peak = 0;

    void turn_on_check(int32_t k) {
        if (queued < omega) sender_on[k] = 1;
    }
};

using fo::set_error;

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
    *out = q;
    return FO_OK;
}

extern "C" void fo_queues_destroy(fo_queues* q) {
    if (!q) return;
    if (q->slab) (void)hipFree(q->slab);
    if (q->labels) (void)hipFree(q->labels);
    if (q->lengths) (void)hipFree(q->lengths);
    delete q;
}

extern "C" fo_status fo_queues_push(fo_queues* q, int32_t k, const void* x_src, const int32_t* labels_src,
                                    const int32_t* lengths_src, int32_t src_on_host) {
    FO_CHECK(q != nullptr, "fo_queues_push: NULL handle");
    FO_CHECK(k >= 0 && k < q->K, "fo_queues_push: device %d out of range [0,%d)", k, q->K);
    if (q->slab) {
        FO_CHECK(x_src != nullptr && labels_src != nullptr, "fo_queues_push: NULL source");
        FO_CHECK(!q->with_lengths || lengths_src != nullptr, "fo_queues_push: this pool needs lengths");
    }
    // Alg. 2 / Sec. 3.4.1: a batch sent while the Sender Status is off never arrives.
    if (!q->sender_on[k]) {
        q->refused++;
        return FO_FULL;
    }
    if (q->free_stack.empty()) {  // cannot happen while omega = n_slots - K holds
        fo::set_error("fo_queues_push: pool exhausted (internal invariant broken)");
        return FO_ESTATE;
    }
    int64_t slot = q->free_stack.back();
    if (q->slab) {
        hipMemcpyKind kind = src_on_host ? hipMemcpyHostToDevice : hipMemcpyDeviceToDevice;
        FO_HIP(hipMemcpyAsync(q->slab + slot * q->slot_bytes, x_src, (size_t)q->slot_bytes, kind, q->stream));
        FO_HIP(hipMemcpyAsync(q->labels + slot * q->batch, labels_src, sizeof(int32_t) * q->batch, kind,
                              q->stream));
        if (q->with_lengths)
            FO_HIP(hipMemcpyAsync(q->lengths + slot * q->batch, lengths_src, sizeof(int32_t) * q->batch, kind,
                                  q->stream));
    }
    try {
        q->q[k].push_back({q->next_seq[k], slot});
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
    q->turn_on_check(k);   // enqueue: below the cap -> 'turn-on'
    return FO_OK;
}

extern "C" fo_status fo_queues_push_model(fo_queues* q, int32_t k, const float* local, int64_t n, int64_t t_k) {
    FO_CHECK(q != nullptr, "fo_queues_push_model: NULL handle");
    FO_CHECK(k >= 0 && k < q->K, "fo_queues_push_model: device %d out of range [0,%d)", k, q->K);
    FO_CHECK(n >= 0 && (n == 0 || local != nullptr), "fo_queues_push_model: bad vector");
    FO_CHECK(t_k >= 0, "fo_queues_push_model: negative version");
    try {
        q->qm.push_back({k, local, n, t_k});
    } catch (...) {
        set_error("fo_queues_push_model: out of host memory");
        return FO_ENOMEM;
    }
    return FO_OK;
}

extern "C" int32_t fo_pick_device(fo_queues* q) {
    if (!q) {
        fo::set_error("fo_pick_device: NULL handle");
        return -3;
    }
    if (!q->qm.empty()) return -2;  // Alg. 3: models are served first
    if (q->busy) {
        fo::set_error("fo_pick_device: release the batch in service first");
        return -3;
    }
    int32_t best = -1;
    for (int32_t k = 0; k < q->K; ++k)
        if (!q->q[k].empty() && (best < 0 || q->c[k] < q->c[best])) best = k;
    if (best < 0) return -1;
    q->svc = q->q[best].front();
    q->q[best].pop_front();
    q->svc_k = best;
    q->busy = true;
    q->queued--;
    q->c[best]++;
    q->picks++;
    q->turn_on_check(best);  // dequeue: below the cap -> 'turn-on'
    return best;
}

extern "C" fo_status fo_queues_in_service(fo_queues* q, fo_acts* acts_out, const int32_t** labels_out,
                                          int64_t* seq_out, int64_t* slot_out) {
    FO_CHECK(q != nullptr, "fo_queues_in_service: NULL handle");
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
    if (!q->busy) {
        fo::set_error("fo_queues_release: no batch in service");
        return FO_ESTATE;
    }
    q->free_stack.push_back(q->svc.slot);
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
    fo_status st = check_global(global, "fo_aggregate_pending");
    if (st != FO_OK) return st;
    FO_CHECK(alpha >= 0.f && alpha <= 1.f, "fo_aggregate_pending: alpha=%g outside [0,1]", (double)alpha);
    if (q->qm.empty()) return FO_EMPTY;
    fo_queues::ModelMsg m = q->qm.front();
    FO_CHECK(m.n == global->n, "fo_aggregate_pending: model length %lld != global %lld", (long long)m.n,
             (long long)global->n);
    FO_CHECK(m.n == 0 || (uintptr_t)m.local % 16 == 0, "fo_aggregate_pending: local not 16-byte aligned");
    q->qm.pop_front();
    int64_t s = q->t - m.t_k;
    if (k_out) *k_out = m.k;
    if (staleness_out) *staleness_out = s;
    int64_t D = fo::g_max_delay.load();
    if (s < 0) {
        fo::set_error("fo_aggregate_pending: model version %lld is newer than the global %lld", (long long)m.t_k,
                      (long long)q->t);
        return FO_EINVAL;
    }
    if (D >= 0 && s > D) return FO_SKIPPED;
    float w = alpha / (float)(s + 1);
    st = fo::launch_agg_lerp(global->ptr, m.local, global->n, w, q->stream);
    if (st != FO_OK) return st;
    q->t++;
    return FO_OK;
}

extern "C" fo_status fo_aggregate_pending_all(fo_queues* q, fo_vec* global, float alpha, int32_t* applied_out,
                                              int32_t* skipped_out) {
    FO_CHECK(q != nullptr, "fo_aggregate_pending_all: NULL handle");
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
    int32_t applied = 0, skipped = 0;
    fo::AggTable tab;
    tab.count = 0;
    while (!q->qm.empty()) {
        fo_queues::ModelMsg m = q->qm.front();
        q->qm.pop_front();
        int64_t s = q->t - m.t_k;
        if (D >= 0 && s > D) {
            skipped++;
            continue;
        }
        tab.local[tab.count] = m.local;
        tab.w[tab.count] = alpha / (float)(s + 1);
        tab.count++;
        q->t++;
        applied++;
        if (tab.count == fo::kAggMaxFused) {
            st = fo::launch_agg_lerp_multi(global->ptr, tab, global->n, q->stream);
            if (st != FO_OK) return st;
            tab.count = 0;
        }
    }
    if (tab.count > 0) {
        st = fo::launch_agg_lerp_multi(global->ptr, tab, global->n, q->stream);
        if (st != FO_OK) return st;
    }
    if (applied_out) *applied_out = applied;
    if (skipped_out) *skipped_out = skipped;
    return FO_OK;
}

extern "C" fo_status fo_queues_stats(const fo_queues* q, fo_queue_stats* out) {
    FO_CHECK(q != nullptr && out != nullptr, "fo_queues_stats: NULL argument");
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
    return FO_OK;
}

extern "C" fo_status fo_queues_counters(const fo_queues* q, int64_t* c_out, int32_t K) {
    FO_CHECK(q != nullptr && c_out != nullptr, "fo_queues_counters: NULL argument");
    FO_CHECK(K >= 0 && K <= q->K, "fo_queues_counters: K=%d out of range", K);
    for (int32_t k = 0; k < K; ++k) c_out[k] = q->c[k];
    return FO_OK;
}

extern "C" int32_t fo_queues_add_device(fo_queues* q) {
    if (!q) {
        fo::set_error("fo_queues_add_device: NULL handle");
        return -1;
    }
    if (q->n_slots - (q->K + 1) < 1) {
        fo::set_error("fo_queues_add_device: pool of %lld slots cannot take another device", (long long)q->n_slots);
        return -1;
    }
    try {
        q->q.emplace_back();
        q->c.push_back(0);
        q->next_seq.push_back(0);
        q->sender_on.push_back(1);
    } catch (...) {
        fo::set_error("fo_queues_add_device: out of host memory");
        return -1;
    }
    q->K++;
    q->omega = q->n_slots - q->K;
    return q->K - 1;
}

extern "C" fo_status fo_set_max_delay(int64_t max_delay) {
    fo::g_max_delay.store(max_delay < 0 ? -1 : max_delay);
    return FO_OK;
}
