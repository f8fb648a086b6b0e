// What the training step needs to know about the activation pools.
#pragma once

#include <vector>

#include "common.h"

namespace fo {

// If the batch (activations or labels) lies in a live pool's slot memory, it
// must be that pool's batch in service (activations, labels and lengths of
// its slot) and device_id must be the device of the last pick; *owner is
// then that pool (else NULL).  FO_EINVAL on a mismatch.  When step_stream is
// not the pool's stream, step_stream is made to wait for the work already
// queued on the pool's stream (the copies into the slot).
fo_status pool_step_begin(const fo_acts* acts, const int32_t* labels, int32_t device_id, hipStream_t step_stream,
                          fo_queues** owner);
// Called after a step on the pool's batch in service has been enqueued on
// step_stream: when that is not the pool's stream, an event recorded there
// makes the next copy into the slot wait for the step.
fo_status pool_step_done(fo_queues* q, hipStream_t step_stream);

// Slot size, batch and whether slots hold lengths; the pool's stream.
void pool_geometry(const fo_queues* q, int64_t* slot_bytes, int32_t* batch, int32_t* with_lengths);
hipStream_t pool_stream(const fo_queues* q);

// fo_aggregate_pending_all that also reports, atomically with the drain, the
// device of every message drained (in FIFO order) and the global version after it.
fo_status pool_drain_models(fo_queues* q, fo_vec* global, float alpha, int32_t* applied, int32_t* skipped,
                            std::vector<int32_t>* devices, int64_t* version);

}  // namespace fo
