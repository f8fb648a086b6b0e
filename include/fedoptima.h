/*
 * fedoptima.h -- C ABI of the FedOptima server hot path on MI355X (gfx950).
 *
 * FedOptima (Zhang, Wong, Varghese) splits a network between K devices and a
 * server.  Devices train the first layers against a local auxiliary loss and
 * upload the activations of their last layer; the server trains the remaining
 * layers (the server-side network M_s) centrally on activation batches chosen
 * by its Task Scheduler, and mixes device-side models that arrive into a
 * global one with a staleness-dependent weight.  This library implements the
 * server's part:
 *
 *   fo_server_step      one training iteration of M_s (Alg. 4, activation branch)
 *   fo_async_aggregate  staleness-weighted mixing of one arriving model (Alg. 4,
 *                       aggregation branch)
 *   fo_pick_device      the Task Scheduler's get() (Alg. 3)
 *
 * together with the activation-queue pool and flow control they need
 * (Alg. 2 put(), Sec. 3.4.1 and the memory bound of Eq. 3).
 *
 * Conventions for every entry point:
 *   - Plain pointers and sizes only.  "device" pointers are HIP device memory
 *     (any allocator), "host" pointers are ordinary host memory.
 *   - GPU work is asynchronous and ordered on the stream bound to the handle
 *     (a hipStream_t passed as void*; NULL is the legacy default stream).
 *     Caller-owned device buffers must stay valid until that work completes.
 *   - Every argument is checked on the host before anything is launched; a
 *     failing check launches nothing and returns a negative fo_status.  The
 *     message for the last failure of the calling thread is fo_last_error().
 *   - The library never allocates device memory inside fo_server_step /
 *     fo_async_aggregate / fo_pick_device; all device memory is allocated by
 *     the *_create calls.  In graph mode (fo_set_graph_mode) the first
 *     fo_server_step of a model at a new batch size creates a private capture
 *     stream and instantiates a HIP graph (host-side objects, freed by
 *     fo_model_destroy).
 */
#ifndef FEDOPTIMA_H
#define FEDOPTIMA_H

#include <stdint.h>

/* The library is built with hidden visibility; only the entry points below are exported. */
#define FO_API __attribute__((visibility("default")))

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FO_OK = 0,        /* done                                                 */
    FO_SKIPPED = 1,   /* aggregation dropped: staleness above the maximum delay */
    FO_EMPTY = 2,     /* nothing to serve                                     */
    FO_FULL = 3,      /* activation batch refused by flow control             */
    FO_EINVAL = -1,   /* bad argument                                         */
    FO_ENOMEM = -2,   /* device or host allocation failed                     */
    FO_EHIP = -3,     /* a HIP runtime call failed                            */
    FO_ESTATE = -4    /* call not valid in the current state                  */
} fo_status;

typedef struct fo_model fo_model;    /* opaque: server model, gradients, optimiser state, workspace */
typedef struct fo_queues fo_queues;  /* opaque: Task Scheduler state and the activation pool        */

/* A caller-owned flat fp32 vector in device memory, 16-byte aligned. */
typedef struct { float* ptr; int64_t n; } fo_vec;

/* One activation batch as sent by a device (device pointers).
 *   x        CNN configs: [batch][C][H][W] (NCHW) -- fp32 for config 1, bf16 bit
 *            patterns (uint16) for configs 2, 3, 5.  Transformer config 4:
 *            [batch][L][d] bf16 hidden states, row-major.
 *   lengths  config 4 only: int32[batch] valid-token counts in [1, L]; keys at
 *            positions >= length are masked.  NULL for the CNN configs.
 *   batch    1 <= batch <= the model's max_batch.                              */
typedef struct { const void* x; const int32_t* lengths; int32_t batch; } fo_acts;

/* ------------------------------------------------------------------ configs
 * Configuration ids 1..5 fix the server network and its precision:
 *   1  tiny CNN, fp32: conv3x3 32->64 + ReLU, maxpool2, conv3x3 64->64 + ReLU,
 *      global average pool, linear 64->10; plain SGD.
 *   2  VGG-16 after its first block (input [64,16,16]): 10 conv3x3 + ReLU with
 *      4 max pools, FC 512-512-10; bf16 GEMMs, fp32 master weights; plain SGD.
 *   3  ResNet-18 stages 2-4 (input [64,16,16]) with training-mode BatchNorm,
 *      global average pool, FC 512->100; bf16; SGD with momentum 0.9.
 *   4  BERT-base-shaped: 10 post-LN encoder layers (d=768, 12 heads, FFN 3072,
 *      exact GELU), tanh pooler on token 0, linear 768->2; bf16; plain SGD.
 *   5  same network as 2 (the 128-device pool-stress workload).
 *   6  the device side of configs 2 and 5 (Alg. 1): the device network
 *      (VGG-16's first block: conv3x3 3->64 + ReLU, conv3x3 64->64 + ReLU,
 *      2x2 max pool) and its auxiliary network (conv3x3 64->64 + ReLU, global
 *      average pool, linear 64->10, Sec. 3.2.2); trained with fo_device_step on
 *      fp32 [B][3][32][32] inputs; bf16 GEMMs, fp32 master weights; plain SGD.
 * Loss: mean softmax cross-entropy over the batch (the server loss f_s, Eq. 5).
 * Learning rate 0.01.  Parameter layout of the flat fp32 vector ("library
 * layout"): layers in network order; per layer weight then bias (or scale then
 * shift for norms); conv weights [Cout][kh][kw][Cin], linear weights [out][in],
 * attention input projection [3d][d] with query, key, value rows in that order. */

/* Number of parameters of a configuration (host only; -1 for a bad id). */
FO_API int64_t fo_config_param_count(int32_t config_id);
/* Number of classes (logits per sample) of a configuration (-1 for a bad id). */
FO_API int32_t fo_config_num_classes(int32_t config_id);

/* ------------------------------------------------------------------ model
 * Creates the server model of `config_id` for batches of up to `max_batch`
 * samples.  `host_init` (host, fp32, n_params = fo_config_param_count) is
 * copied to the device.  All device memory the step needs is allocated here.
 * `hip_stream` is the stream every later call on this model uses.
 * Errors: FO_EINVAL (bad id, size mismatch, max_batch < 1), FO_ENOMEM, FO_EHIP. */
FO_API fo_status fo_model_create(int32_t config_id, int32_t max_batch, const float* host_init,
                          int64_t n_params, void* hip_stream, fo_model** out);
FO_API void fo_model_destroy(fo_model* model);

/* One centralized training iteration of M_s on one activation batch
 * (Alg. 4, activation branch): forward of M_s, loss f_s, backward, then
 * theta_s <- theta_s - gamma_s * grad (with momentum for config 3).  The
 * activation gradient of the first server layer is never formed: devices do
 * not receive gradients from the server.  `labels` is a device int32[batch]
 * of class ids in [0, classes).  `device_id` (>= 0) names the device the batch
 * came from and is counted per device (fo_model_steps).  Asynchronous on the
 * model's stream; loss and logits of this step stay readable until the next
 * step.
 * Batches from a pool: when acts->x or labels lie in the slot memory of a live
 * fo_queues pool, they must be that pool's batch in service (its activations,
 * labels and lengths, from fo_queues_in_service) and device_id must be the
 * device its last fo_pick_device returned.  If the model's stream is not the
 * pool's, the step waits for the work queued on the pool's stream (the copies
 * into the slot), and the slot's next reuse waits for the step, so the two
 * streams need no other synchronisation.
 * Labels outside [0, classes) and lengths outside [1, L] cannot be checked on
 * the host without a synchronisation: the kernels clamp them (every access
 * stays in bounds) and count them, and the next fo_model_read of LOSS or
 * LOGITS returns FO_EINVAL.
 * Errors: FO_EINVAL (NULL pointers, batch out of range, lengths missing for
 * config 4, device_id < 0, a pool batch that is not the one in service or a
 * device_id other than its pick's), FO_EHIP. */
FO_API fo_status fo_server_step(fo_model* model, const fo_acts* acts, const int32_t* labels,
                         int32_t device_id);

/* One local training iteration of a device (Alg. 1) on a config 6 model:
 * forward of the device network on the mini-batch x (device, fp32 NCHW
 * [batch][3][32][32], 16-byte aligned), its output activations written to
 * acts_out (device, bf16 bit patterns NCHW [batch][64][16][16], 16-byte
 * aligned: the batch the device sends to the server, in the layout
 * fo_queues_push and fo_server_step take for configs 2 and 5), forward of the
 * auxiliary network on them, the local loss f_d (mean cross-entropy against
 * labels, device int32[batch] in [0, 10)), backward through both networks and
 * SGD on the device and auxiliary parameters (one flat vector in the library
 * layout: conv1, conv2, auxiliary conv, auxiliary linear).  Asynchronous on
 * the model's stream; loss and logits (of the auxiliary classifier) readable
 * with fo_model_read.  Graph replay as for fo_server_step.  Errors: FO_EINVAL
 * (not a config 6 model, NULL or unaligned pointers, batch out of range),
 * FO_EHIP. */
FO_API fo_status fo_device_step(fo_model* model, const float* x, const int32_t* labels, int32_t batch,
                                uint16_t* acts_out);

/* Process-wide switch for how fo_server_step issues its kernels (default 1).
 * Every step of a model at one batch size is the same sequence of launches
 * over the same buffers: the step's first launch stores the batch pointers
 * (activations, labels, lengths) in a model-owned device record that the
 * other kernels read.  With enable != 0 the launch sequence is captured once
 * per batch size into a HIP graph on a private stream and replayed on the
 * model's stream afterwards, with only that first launch's arguments changed
 * to the new batch's pointers (the batch is never copied).  Results are
 * bit-identical to enable == 0, which launches every kernel directly.  While
 * the calling thread profiles (fo_profile_enable) steps always launch
 * directly.  Steps already captured stay cached until fo_model_destroy.
 * Returns FO_OK. */
FO_API fo_status fo_set_graph_mode(int32_t enable);

/* Steps taken so far on batches from `device_id` (all devices if -1). */
FO_API int64_t fo_model_steps(const fo_model* model, int32_t device_id);

enum {
    FO_BUF_PARAMS = 0,    /* fp32 master parameters, library layout             */
    FO_BUF_GRADS = 1,     /* fp32 gradient of the last step, library layout     */
    FO_BUF_LOGITS = 2,    /* fp32 [batch][classes] logits of the last step      */
    FO_BUF_LOSS = 3,      /* fp32 scalar loss of the last step                  */
    FO_BUF_MOMENTUM = 4   /* fp32 momentum buffer (config 3 only)               */
};
/* Element count of a readable buffer (-1 if the model has none of that kind). */
FO_API int64_t fo_model_buffer_size(const fo_model* model, int32_t which);
/* Synchronous copies between a model buffer and host memory (host_out/host_in
 * hold n fp32 values; n must equal fo_model_buffer_size, except LOGITS where
 * n = batch * classes of the last step).  Used for parity checks and for
 * checkpoint / resume.  Errors: FO_EINVAL (also, after copying, for LOSS and
 * LOGITS of a step whose labels or lengths were out of range), FO_ESTATE (no
 * step yet), FO_EHIP. */
FO_API fo_status fo_model_read(fo_model* model, int32_t which, float* host_out, int64_t n);
FO_API fo_status fo_model_write(fo_model* model, int32_t which, const float* host_in, int64_t n);

/* ------------------------------------------------------------------ aggregation
 * Staleness-weighted mixing of one arriving device-side model (Alg. 4,
 * aggregation branch).  global (device, fp32, n) is updated in place with
 * local (device, fp32, same n):
 *     if staleness > D (see fo_set_max_delay): nothing changes, FO_SKIPPED;
 *     else w = alpha / (staleness + 1) and global <- global + w * (local - global).
 * With alpha = 1 the weight is the 1/(t - t_k + 1) of Alg. 4; alpha = 0 leaves
 * global unchanged bit for bit, as does local == global.  The device-side
 * model and its auxiliary model are mixed by the same rule, so callers pass
 * them as one flat vector.  Runs on the stream set by fo_set_stream for the
 * calling thread.  Errors: FO_EINVAL (NULL, n mismatch or < 0, pointers not
 * 16-byte aligned, alpha outside [0,1], staleness < 0), FO_EHIP. */
FO_API fo_status fo_async_aggregate(fo_vec* global, const fo_vec* local, float alpha, int32_t staleness);

/* Stream used by fo_async_aggregate on the calling thread (default NULL). */
FO_API fo_status fo_set_stream(void* hip_stream);
/* Maximum delay D of Alg. 4 for the whole library; D < 0 means no cutoff
 * (the default). */
FO_API fo_status fo_set_max_delay(int64_t max_delay);

/* ------------------------------------------------------------------ scheduler + pool
 * The Task Scheduler (Alg. 2 put(), Alg. 3 get()) over K per-device activation
 * queues Q_k and a model queue, with consumption counters c_k, the global
 * version t of Alg. 4, and the activation flow control of Sec. 3.4.1.
 *
 * Pool: n_slots fixed-size slots preallocated in device memory (slot_bytes of
 * activations, batch int32 labels and, if with_lengths, batch int32 lengths
 * each).  slot_bytes == 0 keeps only the host bookkeeping (no device memory;
 * pushes then carry no data).  Free slots form a stack handing out the lowest
 * ids first; a released slot is reused first.
 * Flow control: each device's Sender Status starts on.  A batch pushed while
 * it is off is refused (FO_FULL; the device dropped it at the source).  An
 * admitted batch switches it off; after every enqueue to or dequeue from Q_k
 * the status of device k switches back on if the number of queued batches is
 * below omega = n_slots - K.  Queued plus in-service batches therefore never
 * exceed n_slots, whatever K is (Eq. 3: memory = model + omega activation
 * batches, independent of the number of devices).
 * Threads: every pool entry point takes the pool's lock, so pushes (the
 * Receiver's side) and picks, releases and aggregations (the Compute
 * Engine's side) may come from different host threads; the order in which
 * the pool performed them is the order of its event record.
 * Errors: FO_EINVAL (K < 1, n_slots <= K, batch < 1), FO_ENOMEM, FO_EHIP. */
FO_API fo_status fo_queues_create(int32_t K, int64_t slot_bytes, int32_t batch, int32_t with_lengths,
                           int64_t n_slots, void* hip_stream, fo_queues** out);
/* Waits for the pool's stream (and for steps that read its slots from other
 * streams), then frees the pool. */
FO_API void fo_queues_destroy(fo_queues* q);

/* put() for an activation batch from device k (Alg. 2).  x_src holds
 * slot_bytes, labels_src batch int32, lengths_src batch int32 (if the pool has
 * lengths); src_on_host says whether the sources are host or device memory.
 * The copies into the slot are ordered on the pool's stream: from device
 * memory (activations 16-byte aligned) one kernel launch moves the
 * activations, labels and lengths; from host memory, or from unaligned device
 * activations, one copy each.  Returns FO_OK
 * (admitted), FO_FULL (refused by flow control; nothing copied) or an error
 * (FO_EINVAL: k out of range, NULL source for a pool with device memory). */
FO_API fo_status fo_queues_push(fo_queues* q, int32_t k, const void* x_src, const int32_t* labels_src,
                         const int32_t* lengths_src, int32_t src_on_host);

/* put() for n activation batches in arrival order: the same admissions,
 * refusals, slots and sequence numbers as n fo_queues_push calls.  k[i] is the
 * sending device; x_src[i], labels_src[i] and (if the pool has lengths)
 * lengths_src[i] are device pointers, the activations 16-byte aligned.
 * status_out[i] (host, may be NULL) receives FO_OK (admitted) or FO_FULL
 * (refused by flow control).  The copies of the admitted batches run on the
 * pool's stream, up to 32 batches per launch.  Every entry is checked before
 * anything changes (FO_EINVAL: device out of range, NULL or unaligned source);
 * after a failed launch (FO_EHIP) the batches admitted so far are queued but
 * may not have been copied. */
FO_API fo_status fo_queues_push_batch(fo_queues* q, int32_t n, const int32_t* k, const void* const* x_src,
                                      const int32_t* const* labels_src, const int32_t* const* lengths_src,
                                      int32_t* status_out);

/* put() for a model message from device k with local version t_k (Alg. 2):
 * appended to the model FIFO.  `local` (device fp32[n]) is not copied and must
 * stay valid until the message is aggregated. */
FO_API fo_status fo_queues_push_model(fo_queues* q, int32_t k, const float* local, int64_t n, int64_t t_k);
/* The same for n messages in arrival order (device k[i], vector local[i] of
 * len floats, version t_k[i]); every entry is checked before any is queued. */
FO_API fo_status fo_queues_push_model_batch(fo_queues* q, int32_t n, const int32_t* k, const float* const* local,
                                            int64_t len, const int64_t* t_k);

/* get() (Alg. 3).  Returns:
 *   -2  a model message is pending; serve it first (fo_aggregate_pending);
 *   -1  every activation queue is empty;
 *  k>=0 the non-empty queue with the smallest counter c_k (lowest k on ties);
 *       its oldest batch is popped and becomes the batch in service, and c_k
 *       is incremented.  The previous batch in service must have been released.
 *  -3  misuse (NULL handle, or a batch still in service); see fo_last_error. */
FO_API int32_t fo_pick_device(fo_queues* q);

/* The batch popped by the last pick: device pointers into its slot (valid
 * until fo_queues_release) plus its per-device sequence number and slot id. */
FO_API fo_status fo_queues_in_service(fo_queues* q, fo_acts* acts_out, const int32_t** labels_out,
                               int64_t* seq_out, int64_t* slot_out);
/* Returns the in-service slot to the free stack.  Call it after the
 * fo_server_step calls on that batch have been enqueued: later pushes reuse the
 * slot with copies ordered after them (by stream order when the model runs on
 * the pool's stream, else by an event the step recorded on the model's
 * stream). */
FO_API fo_status fo_queues_release(fo_queues* q);

/* Serves the oldest pending model message (Alg. 4, aggregation branch):
 * staleness s = t - t_k; if s > D it is dropped (FO_SKIPPED, t unchanged);
 * otherwise global is mixed with fo_async_aggregate's rule and t <- t + 1.
 * k_out / staleness_out (may be NULL) report the message.  FO_EMPTY if no
 * model is pending.  On an error (FO_EINVAL: length mismatch, misaligned
 * vector, t_k > t; FO_EHIP) the message stays at the head of the FIFO and t is
 * unchanged.  Runs on the pool's stream. */
FO_API fo_status fo_aggregate_pending(fo_queues* q, fo_vec* global, float alpha, int32_t* k_out,
                               int64_t* staleness_out);

/* Drains every pending model message in FIFO order, fusing the mixes: each
 * launch applies up to 64 messages to every element of global in registers
 * (global read and written once per 64 messages), in FIFO order, so the
 * result equals the same sequence of fo_aggregate_pending calls bit for bit.
 * Stale messages are dropped as above and do not advance t.  applied_out /
 * skipped_out may be NULL.  The whole FIFO is validated before anything is
 * launched; if a launch fails, the FIFO and t have advanced past exactly the
 * messages whose launches were enqueued (reported in applied_out /
 * skipped_out).  Runs on the pool's stream. */
FO_API fo_status fo_aggregate_pending_all(fo_queues* q, fo_vec* global, float alpha, int32_t* applied_out,
                                   int32_t* skipped_out);

typedef struct {
    int32_t K;
    int64_t n_slots, omega;
    int64_t queued, in_service, models_pending;
    int64_t admitted, refused, picks, peak_queued;
    int64_t version;            /* global version t */
    int64_t turn_on_signals;    /* off Senders switched on by the cap check (Sec. 3.4.1) */
    int32_t active_devices;     /* devices that have not left */
    int32_t policy;             /* FO_SCHED_COUNTER or FO_SCHED_FIFO */
} fo_queue_stats;
FO_API fo_status fo_queues_stats(const fo_queues* q, fo_queue_stats* out);
/* Copies the counters c_k of the first K devices into c_out. */
FO_API fo_status fo_queues_counters(const fo_queues* q, int64_t* c_out, int32_t K);
/* A device joining mid-run: a new empty queue with c_k = 0 and its Sender on.
 * Returns the new device index, or -1 on error. */
FO_API int32_t fo_queues_add_device(fo_queues* q);

/* Which activation batch get() serves (Alg. 3 and the scheduler ablation of
 * Sec. 6.5).  FO_SCHED_COUNTER (default): the oldest batch of the device with
 * the smallest consumption counter c_k among devices with a queued batch,
 * lowest index on ties.  FO_SCHED_FIFO: the batch admitted earliest over all
 * devices.  c_k is counted under both.  Models are always served first.
 * Errors: FO_EINVAL (unknown policy). */
enum { FO_SCHED_COUNTER = 0, FO_SCHED_FIFO = 1 };
FO_API fo_status fo_queues_set_policy(fo_queues* q, int32_t policy);

/* Device k leaves (active = 0) or rejoins (active = 1) training (Sec. 3.4.2;
 * the dropout of Sec. 6.4).  A device that has left has its Sender Status off
 * and kept off: every batch it would send is refused (FO_FULL) and no
 * 'turn-on' signal reaches it; the batches it sent before leaving stay queued
 * and are served as usual.  On rejoining its Sender starts on, as for a device
 * joining for the first time, and it keeps its counter c_k.  Setting the state
 * a device already has does nothing.  Errors: FO_EINVAL (k out of range). */
FO_API fo_status fo_queues_set_device_active(fo_queues* q, int32_t k, int32_t active);

/* The Sender Status of device k as the device sees it (Sec. 3.4.1): 1 if its
 * next batch would be admitted, 0 if it would be refused, -1 on error. */
FO_API int32_t fo_queues_sender_status(fo_queues* q, int32_t k);

/* Event record of the pool: every state transition in the order the pool
 * performed them, four int64 per event (type, device k, a, b):
 *   FO_EV_PUSH     a = 1 admitted (b = its sequence number) | 0 refused (b = -1)
 *   FO_EV_MODEL    a = t_k of the model message put (Alg. 2)
 *   FO_EV_PICK     a = sequence number, b = slot of the batch served (Alg. 3)
 *   FO_EV_RELEASE  a = sequence number, b = slot
 *   FO_EV_AGG      a = 1 applied | 0 skipped (staleness > D), b = staleness (Alg. 4)
 *   FO_EV_LEAVE    device k left
 *   FO_EV_JOIN     a = 1: new device (fo_queues_add_device) | 0: device k rejoined
 * fo_queues_log_enable reserves room for max_events (host memory, allocated
 * here, never during recording), clears the record and starts recording; events
 * beyond max_events are dropped.  fo_queues_log_read copies the first
 * min(max_events, recorded) events into out ([max_events][4]) and reports the
 * number recorded in *n_out.  Errors: FO_EINVAL, FO_ENOMEM. */
enum { FO_EV_PUSH = 1, FO_EV_MODEL = 2, FO_EV_PICK = 3, FO_EV_RELEASE = 4, FO_EV_AGG = 5, FO_EV_LEAVE = 6,
       FO_EV_JOIN = 7 };
FO_API fo_status fo_queues_log_enable(fo_queues* q, int64_t max_events);
FO_API fo_status fo_queues_log_read(fo_queues* q, int64_t* out, int64_t max_events, int64_t* n_out);

/* ------------------------------------------------------------------ concurrent pipeline
 * The server's concurrent structure (Sec. 5.1: Receiver, Task Scheduler and
 * Compute Engine threads) run for a fixed wall-clock time against K emulated
 * devices, with the flow control of Sec. 3.4.1, devices leaving and rejoining
 * (Sec. 3.4.2) and the dropout and bandwidth variation of Sec. 6.4.
 *
 * Receiver thread (the devices, Alg. 1): device k runs local iterations of
 * iter_seconds[k] x s seconds each, s the slow-down factor of the current
 * interval.  After each iteration it puts its next activation batch if its
 * Sender Status is on, else goes on without sending; after every H
 * iterations it also puts its model (tagged with the global version t_k it
 * holds) and waits for the server's reply before its next iteration.  At the
 * start of every interval of interval_seconds each device is away for that
 * interval with probability p_drop (fo_queues_set_device_active), and a
 * present device draws s from U[1, slow_max]; the draws come from splitmix64
 * of (seed, interval, device), so they do not depend on thread timing.
 * Compute Engine thread (the server, Alg. 3 and Alg. 4): pending models are
 * aggregated with weights alpha / (staleness + 1) (or skipped past the maximum
 * delay), all that are pending in fused launches on the pool's stream as
 * fo_aggregate_pending_all does, and each of their devices then holds the
 * current global version; otherwise the pick is trained on with fo_server_step on the model's
 * stream, at most max_inflight steps ahead of the GPU.  With nothing queued
 * the engine first waits for its steps to finish and then sleeps until a
 * device puts something: that sleep is the server's idle time.
 *
 * Activations the devices send: bank_n batches in device memory laid out like
 * the pool's slots; device k's n-th sent batch is entry (k + n) mod bank_n.
 * Device models: n_local vectors of global->n floats (n % 4 == 0, 16-byte
 * aligned) in device memory; device k's r-th model is entry (k + r) mod
 * n_local.  The run ends after `seconds` (whatever is still queued stays in
 * the pool) once the GPU work it enqueued has finished.  With the pool's
 * event record enabled, the record is the exact interleaving of the two
 * threads' pool operations.
 * Errors: FO_EINVAL (bad configuration, a device-side model, a batch in
 * service), FO_ENOMEM, FO_EHIP, or the first error either thread hit (its
 * message in fo_last_error). */
typedef struct {
    double seconds;              /* wall-clock length of the run, > 0 */
    const double* iter_seconds;  /* host [K]: seconds per local iteration of device k, > 0 */
    int32_t H;                   /* local iterations per round (a model put every H), >= 1 */
    double p_drop;               /* probability a device is away for an interval, in [0, 1) */
    double interval_seconds;     /* length of a dropout / bandwidth interval, > 0 */
    double slow_max;             /* slow-down factors drawn from U[1, slow_max], >= 1 */
    uint64_t seed;
    const void* bank_x;          /* device [bank_n][slot_bytes], 16-byte aligned */
    const int32_t* bank_labels;  /* device [bank_n][batch] */
    const int32_t* bank_lengths; /* device [bank_n][batch] if the pool has lengths, else NULL */
    int32_t bank_n;
    const float* local_bank;     /* device [n_local][global->n] */
    int32_t n_local;
    float alpha;                 /* aggregation weight of Alg. 4, in [0, 1] */
    int32_t max_inflight;        /* in [1, 64] */
} fo_pipeline_config;

typedef struct {
    double wall_seconds;         /* start to the end of the last GPU work */
    double idle_seconds;         /* Compute Engine idle: nothing queued, no step in flight */
    int64_t steps, samples;      /* training iterations (Alg. 4) and their samples */
    int64_t aggregations, skipped; /* models applied / skipped (staleness > D) */
    int64_t sent, not_sent;      /* activation batches sent / withheld (Sender off) */
    int64_t models_sent;
    int64_t leaves, rejoins;     /* dropout transitions after the first interval's draw */
    int64_t device_iterations;   /* local iterations completed by all devices */
} fo_pipeline_stats;

FO_API fo_status fo_pipeline_run(fo_queues* q, fo_model* m, fo_vec* global, const fo_pipeline_config* cfg,
                                 fo_pipeline_stats* out);

/* ------------------------------------------------------------------ pre-processor
 * The initialization stage's Pre-processor (Sec. 3.2.1; auxiliary network of
 * Sec. 3.2.2).  Host code, no GPU work.
 *
 * A network is a table of units the split may follow: a convolution (with its
 * normalisation and activation), a pooling layer, a fully connected layer, a
 * MobileNetV3 bottleneck block (expansion, depthwise, optional
 * squeeze-excitation, projection), an embedding, a transformer encoder layer.
 * Blocks are never cut: the paper splits only at sequential connections.
 * Per unit and sample, fwd_flops counts 2 per multiply-add of its
 * convolutions and matrix products (normalisation, activations, pooling and
 * softmax not counted) and out_elems its output values. */
enum { FO_UNIT_CONV = 1, FO_UNIT_POOL = 2, FO_UNIT_FC = 3, FO_UNIT_BNECK = 4, FO_UNIT_EMB = 6, FO_UNIT_ENC = 7 };
typedef struct {
    int32_t kind;               /* FO_UNIT_* */
    int32_t k, stride;          /* kernel side and stride (0, 1 for a global pool) */
    int32_t c_in, c_out;        /* channels, features, or model width */
    int32_t h_out, w_out;       /* output rows and columns; sequence units: length, 1 */
    int32_t expand;             /* bottleneck expansion width */
    int32_t heads, hidden;      /* encoder heads and FFN width */
    int32_t norm, se;           /* has normalisation; has squeeze-excitation */
    int64_t params;             /* trainable parameters */
    double fwd_flops;           /* forward FLOPs of one sample */
    double out_elems;           /* output values of one sample */
} fo_unit;

/* The unit tables of the paper's networks (Table 4) and of VGG-16:
 *   FO_NET_VGG5              conv3-32, pool, conv3-64, pool, conv3-64, pool, fc-128, fc-classes
 *                            (batch norm, no bias, per convolution); in_hw = image side, % 8 == 0
 *   FO_NET_MOBILENETV3_LARGE conv3-16 stride 2, the 15 bottlenecks, conv1-960, global pool,
 *                            fc-1280, fc-classes; in_hw = image side
 *   FO_NET_TRANSFORMER6/12   EMB-100, 6 encoders (d 100, 5 heads, FFN 100) or 12 (50 heads),
 *                            fc-classes; in_hw = sequence length (the embedding table, whose
 *                            size the paper does not give, counts no parameters)
 *   FO_NET_VGG16             thirteen conv3 (bias) with five pools, fc 512-512-classes;
 *                            in_hw = image side, % 32 == 0
 * Writes min(count, max_units) units to out and returns the count, or -1
 * (unknown network, bad sizes; message in fo_last_error). */
enum { FO_NET_VGG5 = 1, FO_NET_MOBILENETV3_LARGE = 2, FO_NET_TRANSFORMER6 = 3, FO_NET_TRANSFORMER12 = 4,
       FO_NET_VGG16 = 5 };
FO_API int32_t fo_net_units(int32_t net, int32_t classes, int32_t in_hw, fo_unit* out, int32_t max_units);

/* Split-point selection (Eq. 6-8): for every split l = 1..L (M_d = units
 * 1..l), cost(l) = max over devices k of max(sum_{i<=l} O_i / o_k, S_l / b_k),
 * with O_i = 3 x fwd_flops x batch (forward, input- and weight-gradient
 * products of one iteration) and S_l = out_elems x batch x bytes_per_value;
 * *split_out = the l of least cost (the smallest on ties).  flops_per_s[k]
 * (o_k) and bytes_per_s[k] (b_k) are device k's compute rate and bandwidth,
 * host arrays of K > 0 values.  cost_out (host [L], may be NULL) receives
 * every cost.  Errors: FO_EINVAL. */
FO_API fo_status fo_select_split(const fo_unit* units, int32_t L, int32_t batch, int32_t bytes_per_value,
                                 int32_t K, const double* flops_per_s, const double* bytes_per_s,
                                 double* cost_out, int32_t* split_out);

/* The default auxiliary network (Sec. 3.2.2) for the split after unit
 * `split` (1-based): one unit of the same kind as the last unit of M_d that
 * has parameters (pools skipped), as wide as M_d's output, stride 1, then the
 * classifier: global average pool and fc-classes after a convolution or a
 * bottleneck, fc-classes on the first token after an encoder, fc-classes
 * after a fully connected unit; after an embedding, the classifier alone.
 * Writes min(count, max_units) units and returns the count, or -1. */
FO_API int32_t fo_aux_network(const fo_unit* units, int32_t L, int32_t split, int32_t classes, fo_unit* out,
                              int32_t max_units);

/* ------------------------------------------------------------------ instrumentation
 * Kernel timing for benchmarks and tuning.  While enabled on a thread, every
 * MFMA GEMM and attention launch that thread enqueues is bracketed by two HIP
 * events on its stream (up to max_launches launches; later ones are not
 * recorded).  fo_profile_read synchronizes on the recorded events and returns
 * one entry per kernel: launches, summed duration, and summed algorithmic
 * FLOPs (2*M*N*K of the layer over valid rows only, not counting the extra
 * passes of compensated products) and executed MFMA FLOPs.  Reading clears
 * the records.  Errors: FO_EINVAL (max_launches < 0), FO_ENOMEM, FO_EHIP. */
typedef struct {
    char name[48];
    int64_t launches;
    double ms;           /* summed event-to-event time */
    double flops;        /* algorithmic */
    double mfma_flops;   /* executed on the matrix cores */
} fo_kernel_stat;
FO_API fo_status fo_profile_enable(int32_t max_launches);  /* 0 disables */
/* Fills up to `max` entries and returns how many kernels were seen (or < 0 on error). */
FO_API int32_t fo_profile_read(fo_kernel_stat* out, int32_t max);

/* ------------------------------------------------------------------ errors */
FO_API const char* fo_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* FEDOPTIMA_H */
