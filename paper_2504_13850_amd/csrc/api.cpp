// C ABI entry points: errors, configuration queries, model lifetime, the
// training step dispatch and the stand-alone aggregation call.
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>

#include "model.h"
#include "pool.h"
#include "prof.h"

namespace fo {

static thread_local char tl_error[512] = "";
static thread_local hipStream_t tl_agg_stream = nullptr;
extern std::atomic<int64_t> g_max_delay;

void set_error(const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(tl_error, sizeof(tl_error), fmt, ap);
    va_end(ap);
}

// Parameter counts and classes per configuration (derived from the layer
// lists in the model executors).
int64_t cnn32_param_count();
int64_t cnn16_param_count(int32_t cid);
int64_t bert_param_count();
int64_t device_param_count();
int64_t tfsmall_param_count(int32_t cid);
int64_t vgg5_param_count();
int64_t mbv3_param_count();

}  // namespace fo

using namespace fo;

extern "C" const char* fo_last_error(void) { return tl_error; }

extern "C" int64_t fo_config_param_count(int32_t cid) {
    switch (cid) {
        case 1: return cnn32_param_count();
        case 2: case 3: case 5: return cnn16_param_count(cid);
        case 4: return bert_param_count();
        case 6: return device_param_count();
        case 7: case 8: return tfsmall_param_count(cid);
        case 9: return vgg5_param_count();
        case 10: return mbv3_param_count();
        default: return -1;
    }
}

extern "C" int32_t fo_config_num_classes(int32_t cid) {
    switch (cid) {
        case 1: case 2: case 5: case 6: case 9: return 10;
        case 3: return 100;
        case 4: case 7: case 8: return 2;
        case 10: return 200;
        default: return -1;
    }
}

static const Family* family_of(int32_t cid) {
    switch (cid) {
        case 1: return family_cnn32();
        case 2: case 3: case 5: return family_cnn16();
        case 4: return family_bert();
        case 6: return family_device();
        case 7: return family_tfsmall7();
        case 8: return family_tfsmall8();
        case 9: return family_vgg5();
        case 10: return family_mbv3();
        default: return nullptr;
    }
}

extern "C" fo_status fo_model_create(int32_t cid, int32_t max_batch, const float* host_init, int64_t n_params,
                                     void* hip_stream, fo_model** out) {
    FO_CHECK(out != nullptr, "fo_model_create: out is NULL");
    *out = nullptr;
    const Family* fam = family_of(cid);
    FO_CHECK(fam != nullptr, "fo_model_create: unknown config %d", cid);
    FO_CHECK(max_batch >= 1 && max_batch <= 4096, "fo_model_create: max_batch=%d out of range [1,4096]", max_batch);
    FO_CHECK(host_init != nullptr, "fo_model_create: host_init is NULL");
    int64_t np = fo_config_param_count(cid);
    FO_CHECK(n_params == np, "fo_model_create: n_params=%lld, config %d has %lld", (long long)n_params, cid,
             (long long)np);
    fo_model* m = new (std::nothrow) fo_model();
    if (!m) return FO_ENOMEM;
    m->cid = cid;
    m->max_batch = max_batch;
    m->classes = fo_config_num_classes(cid);
    m->stream = (hipStream_t)hip_stream;
    m->n_params = np;
    m->momentum = cid == 3 ? 0.9f : 0.f;
    m->fam = fam;
    const bool bf16 = cid != 1 && cid < 7;  // the fp32 configs (1, 7-10) keep no bf16 shadows
    size_t bytes = 0;
    auto add = [&](size_t b) { bytes += (b + 255) & ~size_t(255); };
    add(sizeof(float) * np);                          // params
    add(sizeof(float) * np);                          // grads
    if (m->momentum != 0.f) add(sizeof(float) * np);  // momentum
    if (bf16) add(sizeof(bf16_t) * np);               // shadow (high part)
    if (bf16) add(sizeof(bf16_t) * np);               // shadow (low part)
    add(sizeof(float) * (size_t)max_batch * m->classes);
    add(sizeof(float) * 64);
    add(sizeof(StepIn));                              // the step's batch pointers
    bytes += fam->workspace_bytes(m) + 4096;
    hipError_t e = hipMalloc((void**)&m->mem, bytes);
    if (e != hipSuccess) {
        set_error("fo_model_create: hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
        delete m;
        return e == hipErrorOutOfMemory ? FO_ENOMEM : FO_EHIP;
    }
    m->arena.base = m->mem;
    m->arena.size = bytes;
    m->params = m->arena.take<float>(np);
    m->grads = m->arena.take<float>(np);
    if (m->momentum != 0.f) m->mom = m->arena.take<float>(np);
    if (bf16) m->w16 = m->arena.take<bf16_t>(np);
    if (bf16) m->w16lo = m->arena.take<bf16_t>(np);
    m->logits = m->arena.take<float>((size_t)max_batch * m->classes);
    m->loss = m->arena.take<float>(64);
    m->dev_in = m->arena.take<StepIn>(1);
    fo_status st = FO_OK;
    e = hipMemcpyAsync(m->params, host_init, sizeof(float) * np, hipMemcpyHostToDevice, m->stream);
    if (e == hipSuccess) e = hipMemsetAsync(m->grads, 0, sizeof(float) * np, m->stream);
    if (e == hipSuccess) e = hipMemsetAsync(m->loss, 0, sizeof(float) * 64, m->stream);
    if (e == hipSuccess && m->mom) e = hipMemsetAsync(m->mom, 0, sizeof(float) * np, m->stream);
    if (e != hipSuccess) {
        set_error("fo_model_create: upload: %s", hipGetErrorString(e));
        st = FO_EHIP;
    }
    if (st == FO_OK && m->w16) st = launch_cast_bf16(m->params, m->w16, m->w16lo, np, m->stream);
    if (st == FO_OK) st = fam->init(m);
    if (st == FO_OK) {
        e = hipStreamSynchronize(m->stream);
        if (e != hipSuccess) {
            set_error("fo_model_create: %s", hipGetErrorString(e));
            st = FO_EHIP;
        }
    }
    if (st != FO_OK) {
        fo_model_destroy(m);
        return st;
    }
    *out = m;
    return FO_OK;
}

extern "C" void fo_model_destroy(fo_model* m) {
    if (!m) return;
    if (m->mem) (void)hipStreamSynchronize(m->stream);
    for (auto& kv : m->graphs) {
        if (kv.second.exec) (void)hipGraphExecDestroy(kv.second.exec);
        if (kv.second.graph) (void)hipGraphDestroy(kv.second.graph);
    }
    m->graphs.clear();
    if (m->capture_stream) (void)hipStreamDestroy(m->capture_stream);
    if (m->fam && m->plan) m->fam->destroy(m);
    if (m->mem) (void)hipFree(m->mem);
    delete m;
}

// ------------------------------------------------------------------ graph replay of the step
// A step is a fixed sequence of launches for a given batch size (sizes that
// depend on the batch's contents, such as the packed token count, stay on the
// device), so it is captured once per batch size into a HIP graph and replayed:
// one launch instead of one per kernel.  The kernels read the batch through
// the model's StepIn record, which the step's first launch (latch_inputs)
// fills; that launch is the graph's only root, and before each replay its
// arguments are set to the new batch's pointers, so the batch is never copied.
// Capture runs on a private stream (the null stream cannot be captured) with
// the model's stream swapped for it; replays go to the model's stream.
static int g_graph_mode = 1;

__global__ void latch_inputs(StepIn* __restrict__ in, const void* x, const int32_t* labels, const int32_t* lengths,
                             void* out) {
    in->x = x;
    in->labels = labels;
    in->lengths = lengths;
    in->out = out;
}

static fo_status launch_latch(fo_model* m, const fo_acts* acts, const int32_t* labels, void* out, hipStream_t s) {
    hipLaunchKernelGGL(latch_inputs, dim3(1), dim3(1), 0, s, m->dev_in, acts->x, labels, acts->lengths, out);
    FO_LAUNCHED();
    return FO_OK;
}

// The step as launched directly: the latch, then the family's kernels.
static fo_status step_direct(fo_model* m, const fo_acts* acts, const int32_t* labels, void* out) {
    fo_status st = launch_latch(m, acts, labels, out, m->stream);
    return st != FO_OK ? st : m->fam->step(m, acts, labels);
}

static fo_status capture_step(fo_model* m, const fo_acts* acts, const int32_t* labels, void* outp,
                              fo_model::Captured* out) {
    if (!m->capture_stream && hipStreamCreateWithFlags(&m->capture_stream, hipStreamNonBlocking) != hipSuccess) {
        m->capture_stream = nullptr;
        set_error("fo_server_step: hipStreamCreateWithFlags failed");
        return FO_EHIP;
    }
    hipStream_t user = m->stream;
    hipError_t e = hipStreamBeginCapture(m->capture_stream, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) {
        set_error("fo_server_step: hipStreamBeginCapture: %s", hipGetErrorString(e));
        return FO_EHIP;
    }
    m->stream = m->capture_stream;
    const fo_status st = step_direct(m, acts, labels, outp);
    m->stream = user;
    hipGraph_t g = nullptr;
    e = hipStreamEndCapture(m->capture_stream, &g);
    if (st != FO_OK || e != hipSuccess) {
        if (g) (void)hipGraphDestroy(g);
        if (st != FO_OK) return st;
        set_error("fo_server_step: hipStreamEndCapture: %s", hipGetErrorString(e));
        return FO_EHIP;
    }
    // the latch is the graph's only root: every other launch follows it in stream order
    size_t nroot = 0;
    e = hipGraphGetRootNodes(g, nullptr, &nroot);
    hipGraphNode_t root = nullptr;
    hipGraphNodeType type = hipGraphNodeTypeEmpty;
    if (e == hipSuccess && nroot == 1) e = hipGraphGetRootNodes(g, &root, &nroot);
    if (e == hipSuccess && nroot == 1) e = hipGraphNodeGetType(root, &type);
    if (e != hipSuccess || nroot != 1 || type != hipGraphNodeTypeKernel) {
        (void)hipGraphDestroy(g);
        set_error("fo_server_step: the captured step does not start with its input latch (%zu roots)", nroot);
        return FO_EHIP;
    }
    hipGraphExec_t ex = nullptr;
    e = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    if (e != hipSuccess) {
        (void)hipGraphDestroy(g);
        set_error("fo_server_step: hipGraphInstantiate: %s", hipGetErrorString(e));
        return FO_EHIP;
    }
    out->graph = g;
    out->exec = ex;
    out->latch = root;
    return FO_OK;
}

static fo_status step_graph(fo_model* m, const fo_acts* acts, const int32_t* labels, void* outp) {
    const int B = acts->batch;
    auto it = m->graphs.find(B);
    if (it == m->graphs.end()) {
        fo_model::Captured c;
        fo_status st = capture_step(m, acts, labels, outp, &c);
        if (st != FO_OK) return st;
        try {
            it = m->graphs.emplace(B, c).first;
        } catch (...) {
            (void)hipGraphExecDestroy(c.exec);
            (void)hipGraphDestroy(c.graph);
            set_error("fo_server_step: out of host memory");
            return FO_ENOMEM;
        }
    }
    // this batch's pointers into the latch launch
    StepIn* in = m->dev_in;
    const void* x = acts->x;
    const int32_t* lab = labels;
    const int32_t* len = acts->lengths;
    void* args[] = {&in, &x, &lab, &len, &outp};
    hipKernelNodeParams p = {};
    p.func = reinterpret_cast<void*>(&latch_inputs);
    p.gridDim = dim3(1);
    p.blockDim = dim3(1);
    p.sharedMemBytes = 0;
    p.kernelParams = args;
    p.extra = nullptr;
    hipError_t e = hipGraphExecKernelNodeSetParams(it->second.exec, it->second.latch, &p);
    if (e == hipSuccess) e = hipGraphLaunch(it->second.exec, m->stream);
    if (e != hipSuccess) {
        set_error("fo_server_step: graph replay: %s", hipGetErrorString(e));
        return FO_EHIP;
    }
    return FO_OK;
}

extern "C" fo_status fo_set_graph_mode(int32_t enable) {
    g_graph_mode = enable != 0;
    return FO_OK;
}

extern "C" fo_status fo_server_step(fo_model* m, const fo_acts* acts, const int32_t* labels, int32_t device_id) {
    FO_CHECK(m != nullptr, "fo_server_step: NULL model");
    FO_CHECK(m->cid != 6, "fo_server_step: config 6 is a device-side model (fo_device_step)");
    FO_CHECK(acts != nullptr && acts->x != nullptr, "fo_server_step: NULL activations");
    FO_CHECK(labels != nullptr, "fo_server_step: NULL labels");
    FO_CHECK(acts->batch >= 1 && acts->batch <= m->max_batch, "fo_server_step: batch=%d outside [1,%d]",
             acts->batch, m->max_batch);
    FO_CHECK(device_id >= 0, "fo_server_step: device_id=%d must be >= 0", device_id);
    FO_CHECK((m->cid != 4 && m->cid != 7 && m->cid != 8) || acts->lengths != nullptr,
             "fo_server_step: config %d needs sequence lengths", m->cid);
    FO_CHECK(((uintptr_t)acts->x % 16) == 0, "fo_server_step: activations not 16-byte aligned");
    // A batch taken from a pool must be the one its last pick put in service.
    fo_queues* owner = nullptr;
    fo_status st = pool_step_begin(acts, labels, device_id, m->stream, &owner);
    if (st != FO_OK) return st;
    // Kernel profiling records every launch with its own events: run eagerly then.
    st = (g_graph_mode && !prof_active()) ? step_graph(m, acts, labels, nullptr) : step_direct(m, acts, labels, nullptr);
    if (st != FO_OK) return st;
    if (owner) {
        st = pool_step_done(owner, m->stream);
        if (st != FO_OK) return st;
    }
    m->last_batch = acts->batch;
    m->steps_total++;
    if ((size_t)device_id >= m->steps_per_device.size()) m->steps_per_device.resize(device_id + 1, 0);
    m->steps_per_device[device_id]++;
    return FO_OK;
}

extern "C" fo_status fo_device_step(fo_model* m, const float* x, const int32_t* labels, int32_t batch,
                                    uint16_t* acts_out) {
    FO_CHECK(m != nullptr, "fo_device_step: NULL model");
    FO_CHECK(m->cid == 6, "fo_device_step: config %d is a server-side model (fo_server_step)", m->cid);
    FO_CHECK(x != nullptr && labels != nullptr && acts_out != nullptr, "fo_device_step: NULL pointer");
    FO_CHECK(batch >= 1 && batch <= m->max_batch, "fo_device_step: batch=%d outside [1,%d]", batch, m->max_batch);
    FO_CHECK(((uintptr_t)x % 16) == 0 && ((uintptr_t)acts_out % 16) == 0,
             "fo_device_step: input and output must be 16-byte aligned");
    fo_acts acts;
    acts.x = x;
    acts.lengths = nullptr;
    acts.batch = batch;
    fo_status st = (g_graph_mode && !prof_active()) ? step_graph(m, &acts, labels, acts_out)
                                                    : step_direct(m, &acts, labels, acts_out);
    if (st != FO_OK) return st;
    m->last_batch = batch;
    m->steps_total++;
    return FO_OK;
}

extern "C" int64_t fo_model_steps(const fo_model* m, int32_t device_id) {
    if (!m) return -1;
    if (device_id < 0) return m->steps_total;
    return (size_t)device_id < m->steps_per_device.size() ? m->steps_per_device[device_id] : 0;
}

extern "C" int64_t fo_model_buffer_size(const fo_model* m, int32_t which) {
    if (!m) return -1;
    switch (which) {
        case FO_BUF_PARAMS: case FO_BUF_GRADS: return m->n_params;
        case FO_BUF_LOGITS: return (int64_t)m->last_batch * m->classes;
        case FO_BUF_LOSS: return 1;
        case FO_BUF_MOMENTUM: return m->mom ? m->n_params : -1;
        default: return -1;
    }
}

static float* buffer_ptr(fo_model* m, int32_t which) {
    switch (which) {
        case FO_BUF_PARAMS: return m->params;
        case FO_BUF_GRADS: return m->grads;
        case FO_BUF_LOGITS: return m->logits;
        case FO_BUF_LOSS: return m->loss;
        case FO_BUF_MOMENTUM: return m->mom;
        default: return nullptr;
    }
}

extern "C" fo_status fo_model_read(fo_model* m, int32_t which, float* host_out, int64_t n) {
    FO_CHECK(m != nullptr && host_out != nullptr, "fo_model_read: NULL argument");
    float* p = buffer_ptr(m, which);
    FO_CHECK(p != nullptr, "fo_model_read: model has no buffer %d", which);
    if ((which == FO_BUF_LOGITS || which == FO_BUF_LOSS) && m->steps_total == 0) {
        set_error("fo_model_read: no step has run yet");
        return FO_ESTATE;
    }
    FO_CHECK(n == fo_model_buffer_size(m, which), "fo_model_read: n=%lld, buffer holds %lld", (long long)n,
             (long long)fo_model_buffer_size(m, which));
    FO_HIP(hipMemcpyAsync(host_out, p, sizeof(float) * n, hipMemcpyDeviceToHost, m->stream));
    float flags[2] = {0.f, 0.f};  // labels / lengths out of range in the last step (clamped by the kernels)
    if (which == FO_BUF_LOSS || which == FO_BUF_LOGITS)
        FO_HIP(hipMemcpyAsync(flags, m->loss + 1, sizeof(flags), hipMemcpyDeviceToHost, m->stream));
    FO_HIP(hipStreamSynchronize(m->stream));
    if (flags[0] != 0.f || flags[1] != 0.f) {
        set_error("fo_model_read: the last step had %d label(s) outside [0,%d) and %d sequence length(s) outside "
                  "[1,L]; they were clamped, so its loss and logits are not those of the batch as sent",
                  (int)flags[0], m->classes, (int)flags[1]);
        return FO_EINVAL;
    }
    return FO_OK;
}

extern "C" fo_status fo_model_write(fo_model* m, int32_t which, const float* host_in, int64_t n) {
    FO_CHECK(m != nullptr && host_in != nullptr, "fo_model_write: NULL argument");
    FO_CHECK(which == FO_BUF_PARAMS || which == FO_BUF_MOMENTUM, "fo_model_write: only PARAMS and MOMENTUM");
    float* p = buffer_ptr(m, which);
    FO_CHECK(p != nullptr, "fo_model_write: model has no buffer %d", which);
    FO_CHECK(n == m->n_params, "fo_model_write: n=%lld, buffer holds %lld", (long long)n, (long long)m->n_params);
    FO_HIP(hipMemcpyAsync(p, host_in, sizeof(float) * n, hipMemcpyHostToDevice, m->stream));
    if (which == FO_BUF_PARAMS && m->w16) {
        fo_status st = launch_cast_bf16(m->params, m->w16, m->w16lo, m->n_params, m->stream);
        if (st != FO_OK) return st;
    }
    FO_HIP(hipStreamSynchronize(m->stream));
    return FO_OK;
}

extern "C" fo_status fo_set_stream(void* hip_stream) {
    tl_agg_stream = (hipStream_t)hip_stream;
    return FO_OK;
}

extern "C" fo_status fo_async_aggregate(fo_vec* global, const fo_vec* local, float alpha, int32_t staleness) {
    FO_CHECK(global != nullptr && local != nullptr, "fo_async_aggregate: NULL vector");
    FO_CHECK(global->n == local->n, "fo_async_aggregate: lengths differ (%lld vs %lld)", (long long)global->n,
             (long long)local->n);
    FO_CHECK(global->n >= 0, "fo_async_aggregate: negative length");
    FO_CHECK(global->n == 0 || (global->ptr != nullptr && local->ptr != nullptr), "fo_async_aggregate: NULL data");
    FO_CHECK(((uintptr_t)global->ptr % 16) == 0 && ((uintptr_t)local->ptr % 16) == 0,
             "fo_async_aggregate: vectors must be 16-byte aligned");
    FO_CHECK(alpha >= 0.f && alpha <= 1.f, "fo_async_aggregate: alpha=%g outside [0,1]", (double)alpha);
    FO_CHECK(staleness >= 0, "fo_async_aggregate: staleness=%d < 0", staleness);
    int64_t D = g_max_delay.load();
    if (D >= 0 && staleness > D) return FO_SKIPPED;
    float w = alpha / (float)(staleness + 1);
    return launch_agg_lerp(global->ptr, local->ptr, global->n, w, tl_agg_stream);
}
