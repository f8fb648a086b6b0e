// Kernel timing instrumentation: HIP events around the launches a thread
// issues while profiling is on.  Device-side sizes (packed token counts,
// sequence offsets) are copied by the recorded kernel itself into the
// record's snapshot slot, so the FLOP count of every launch is the one of its
// own batch and no extra work enters the timed stream.
#include <algorithm>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "prof.h"

namespace fo {
namespace {

constexpr int kSnapInts = kProfSnapInts;

struct Rec {
    std::string name;
    ProfInfo info;
    hipEvent_t a = nullptr, b = nullptr;
    bool closed = false;
};

struct Profiler {
    int cap = 0;
    std::vector<Rec> recs;
    std::vector<hipEvent_t> events;  // 2 per record, created up front
    int* snap = nullptr;             // device: cap * kSnapInts
    ~Profiler() { release(); }
    void release() {
        for (hipEvent_t e : events) (void)hipEventDestroy(e);
        events.clear();
        if (snap) (void)hipFree(snap);
        snap = nullptr;
        recs.clear();
        cap = 0;
    }
};

thread_local Profiler* tl_prof = nullptr;

}  // namespace

int prof_begin(hipStream_t s, const char* name, const ProfInfo& info) {
    Profiler* p = tl_prof;
    if (!p || (int)p->recs.size() >= p->cap) return -1;
    const int h = (int)p->recs.size();
    Rec r;
    r.name = name;
    r.info = info;
    r.a = p->events[2 * h];
    r.b = p->events[2 * h + 1];
    (void)hipEventRecord(r.a, s);
    p->recs.push_back(r);
    return h;
}

int prof_begin_ext(const char* name, const ProfInfo& info, hipEvent_t* a, hipEvent_t* b) {
    *a = *b = nullptr;
    Profiler* p = tl_prof;
    if (!p || (int)p->recs.size() >= p->cap) return -1;
    const int h = (int)p->recs.size();
    Rec r;
    r.name = name;
    r.info = info;
    r.a = *a = p->events[2 * h];
    r.b = *b = p->events[2 * h + 1];
    p->recs.push_back(r);
    return h;
}

void prof_end_ext(int h) {
    Profiler* p = tl_prof;
    if (!p || h < 0 || h >= (int)p->recs.size()) return;
    p->recs[h].closed = true;
}

bool prof_active() { return tl_prof != nullptr; }

int* prof_snap(int h) {
    Profiler* p = tl_prof;
    if (!p || h < 0 || h >= (int)p->recs.size()) return nullptr;
    return p->snap + (size_t)h * kSnapInts;
}

void prof_end(int h, hipStream_t s) {
    Profiler* p = tl_prof;
    if (!p || h < 0 || h >= (int)p->recs.size()) return;
    (void)hipEventRecord(p->recs[h].b, s);
    p->recs[h].closed = true;
}

}  // namespace fo

using namespace fo;

extern "C" fo_status fo_profile_enable(int32_t max_launches) {
    FO_CHECK(max_launches >= 0, "fo_profile_enable: max_launches=%d < 0", max_launches);
    if (tl_prof) {
        delete tl_prof;
        tl_prof = nullptr;
    }
    if (max_launches == 0) return FO_OK;
    Profiler* p = new (std::nothrow) Profiler();
    if (!p) return FO_ENOMEM;
    p->cap = max_launches;
    try {
        p->events.resize(2 * (size_t)max_launches, nullptr);
        p->recs.reserve(max_launches);
    } catch (...) {
        delete p;
        set_error("fo_profile_enable: out of host memory");
        return FO_ENOMEM;
    }
    for (auto& e : p->events) {
        if (hipEventCreate(&e) != hipSuccess) {
            e = nullptr;
            delete p;
            set_error("fo_profile_enable: hipEventCreate failed");
            return FO_EHIP;
        }
    }
    if (hipMalloc((void**)&p->snap, sizeof(int) * kSnapInts * (size_t)max_launches) != hipSuccess) {
        delete p;
        set_error("fo_profile_enable: hipMalloc failed");
        return FO_ENOMEM;
    }
    tl_prof = p;
    return FO_OK;
}

extern "C" int32_t fo_profile_read(fo_kernel_stat* out, int32_t max) {
    Profiler* p = tl_prof;
    if (!p) return 0;
    const int n = (int)p->recs.size();
    std::vector<int> snap((size_t)n * kSnapInts, 0);
    if (n > 0) {
        for (const Rec& r : p->recs)
            if (r.closed && hipEventSynchronize(r.b) != hipSuccess) {
                set_error("fo_profile_read: event synchronisation failed");
                return FO_EHIP;
            }
        if (hipMemcpy(snap.data(), p->snap, sizeof(int) * snap.size(), hipMemcpyDeviceToHost) != hipSuccess) {
            set_error("fo_profile_read: snapshot copy failed");
            return FO_EHIP;
        }
    }
    struct Acc { int64_t launches = 0; double ms = 0, flops = 0, mfma = 0; };
    std::map<std::string, Acc> agg;
    std::vector<std::string> order;
    for (int h = 0; h < n; ++h) {
        const Rec& r = p->recs[h];
        if (!r.closed) continue;
        float ms = 0.f;
        (void)hipEventElapsedTime(&ms, r.a, r.b);
        const int* sn = snap.data() + (size_t)h * kSnapInts;
        double flops = 0, mfma = 0;
        const ProfInfo& f = r.info;
        if (f.kind == PROF_GEMM && f.ngroup > 0) {  // grouped launch: (M, K) per member
            for (int i = 0; i < f.ngroup && i < 4; ++i) flops += 2.0 * sn[2 * i] * f.gN[i] * sn[2 * i + 1];
            mfma = flops;
        } else if (f.kind == PROF_GEMM) {
            double M = sn[0], K = sn[1];  // effective sizes written by the kernel
            flops = 2.0 * M * f.N * K;
            mfma = flops * f.nseg;
        } else if ((f.kind == PROF_ATTN_FWD || f.kind == PROF_ATTN_BWD) && f.B + 1 <= kSnapInts) {
            double sq = 0;  // sum over sequences of len^2
            for (int b = 0; b < f.B; ++b) {
                double len = sn[b + 1] - sn[b];
                sq += len * len;
            }
            // forward: S = Q K^T and O = P V, 2 len^2 dh MACs per head -> 4 d len^2 FLOPs;
            // backward: dP, dV, dQ, dK -> 8 d len^2 FLOPs
            flops = (f.kind == PROF_ATTN_FWD ? 4.0 : 8.0) * f.d * sq;
        }
        if (!agg.count(r.name)) order.push_back(r.name);
        Acc& a = agg[r.name];
        a.launches++;
        a.ms += ms;
        a.flops += flops;
        a.mfma += mfma;
    }
    int i = 0;
    for (const std::string& nm : order) {
        if (out && i < max) {
            fo_kernel_stat& st = out[i];
            std::memset(&st, 0, sizeof(st));
            std::strncpy(st.name, nm.c_str(), sizeof(st.name) - 1);
            const Acc& a = agg[nm];
            st.launches = a.launches;
            st.ms = a.ms;
            st.flops = a.flops;
            st.mfma_flops = a.mfma;
        }
        ++i;
    }
    p->recs.clear();
    return i;
}
