// The server model object behind fo_model and the per-family executors.
#pragma once

#include <map>
#include <vector>

#include "kernels.h"

namespace fo {
struct Family;
}

struct fo_model {
    int32_t cid = 0;
    int32_t max_batch = 0;
    int32_t classes = 0;
    hipStream_t stream = nullptr;
    int64_t n_params = 0;
    float lr = 0.01f, momentum = 0.f;

    // flat buffers in the library layout (device)
    float* params = nullptr;   // fp32 master
    float* grads = nullptr;    // fp32 gradient of the last step
    float* mom = nullptr;      // momentum buffer (config 3)
    fo::bf16_t* w16 = nullptr;   // bf16(params) (bf16 configs)
    fo::bf16_t* w16lo = nullptr; // bf16(params - bf16(params)): low part for compensated products
    float* logits = nullptr;   // [max_batch][classes]
    float* loss = nullptr;     // scalar

    int32_t last_batch = 0;
    int64_t steps_total = 0;
    std::vector<int64_t> steps_per_device;

    // The batch pointers of the current step (device record read by the step's
    // kernels; filled by the step's first launch).
    fo::StepIn* dev_in = nullptr;
    // Graph replay of the step: one captured graph per batch size; its only root
    // is the launch that fills dev_in, whose arguments change per replay.
    struct Captured {
        hipGraph_t graph = nullptr;
        hipGraphExec_t exec = nullptr;
        hipGraphNode_t latch = nullptr;
    };
    hipStream_t capture_stream = nullptr;  // private (capture cannot run on the null stream)
    std::map<int32_t, Captured> graphs;    // one per batch size

    char* mem = nullptr;       // one allocation for everything above and the workspace
    fo::Arena arena;
    const fo::Family* fam = nullptr;
    void* plan = nullptr;      // family-specific state
};

namespace fo {

struct Family {
    // Bytes of one input sample at the boundary (activations of one batch row).
    int64_t sample_bytes;
    // Bytes of workspace (beyond params/grads/...) for batches up to max_batch.
    size_t (*workspace_bytes)(const fo_model* m);
    // Carve the plan out of m->arena; called once after the flat buffers exist.
    fo_status (*init)(fo_model* m);
    // Enqueue one training step on m->stream.
    fo_status (*step)(fo_model* m, const fo_acts* acts, const int32_t* labels);
    void (*destroy)(fo_model* m);
};

// Orders `to` after everything enqueued so far on `from` (a fork or a join of
// two streams of one model; inside a capture it becomes a graph edge).
inline fo_status order_after(hipStream_t to, hipStream_t from, hipEvent_t e) {
    FO_HIP(hipEventRecord(e, from));
    FO_HIP(hipStreamWaitEvent(to, e, 0));
    return FO_OK;
}

// Accessors (function-local statics keep the tables out of device code).
const Family* family_cnn32();   // config 1
const Family* family_cnn16();   // configs 2, 3, 5
const Family* family_bert();    // config 4
const Family* family_device();  // config 6 (device side of configs 2 and 5)
const Family* family_tfsmall7();  // config 7 (Transformer-6 after its embedding)
const Family* family_tfsmall8();  // config 8 (Transformer-12 after its embedding)
const Family* family_vgg5();      // config 9 (VGG-5 after its second pool)
const Family* family_mbv3();      // config 10 (MobileNetV3-Large after its seventh bottleneck)

}  // namespace fo
