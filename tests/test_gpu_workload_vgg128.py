"""GPU tests of the 128-device workload loop: lognormal device rates, Poisson
arrivals per server step, each arrival an activation batch put into the HBM
pool under flow control (Alg. 2, Sec. 3.4.1) and a model message; pending
models are aggregated first in fused drains (Alg. 3, Alg. 4 aggregation
branch), then one batch is picked and trained on.  Checked against the oracle
scheduler, aggregation and server step through the C ABI:
  - every admission, pick, sequence number, slot id, counter, refusal count,
    peak occupancy and version bit for bit;
  - the bytes and labels in the slot of the batch in service are the ones
    pushed for that (device, sequence);
  - the global model equals the oracle's FIFO sequence of staleness-weighted
    mixes (fp64, rounded to fp32 after each) within 1e-4 normwise;
  - training: the step on each picked batch is compared with the oracle's
    step on the batch and labels pushed for that (device, sequence), run from
    the library's parameters just before the step (loss, logits, update): at
    every step of the small loop, and at sampled steps of the loop at the
    workload's own size (batch 64, 64 GiB pool = 32,768 slots of 2 MiB, past
    the step where the cap starts refusing arrivals).  A wrong slot or label
    moves the loss by far more than the bound.
The small loop hands each arrival over with its own put() calls, the loop at
workload scale with the batched calls (one per step for the activation
batches, one for the model messages)."""
import ctypes
import os

import numpy as np
import pytest

import fo_synth as S
import oracle
from oracle import aggregate as OA
from oracle.scheduler import TaskScheduler
from tests.gpu_util import announce, normwise, torch_cuda

pytestmark = pytest.mark.gpu
A = pytest.importorskip("paper_2504_13850_amd.api")

TOL = 2e-2
GRAD_TOL = 6e-2


def _d2h(torch, ptr, nbytes):
    """Device bytes at a raw pointer, through the process's HIP runtime (torch's)."""
    hip = ctypes.CDLL(os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so"))
    out = np.empty(nbytes, np.uint8)
    torch.cuda.synchronize()
    rc = hip.hipMemcpy(ctypes.c_void_p(out.ctypes.data), ctypes.c_void_p(ptr), ctypes.c_size_t(nbytes),
                       ctypes.c_int(2))  # hipMemcpyDeviceToHost
    assert rc == 0, rc
    return out


def _frob(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)


def _run_loop(B, steps, n_slots, bank_n, counts_sub, sample_steps=(), batched=False):
    """Runs the loop; returns a summary.  sample_steps: the steps whose
    training is compared with the oracle from the library's parameters;
    batched: each step's arrivals go through the batched put() calls."""
    torch = torch_cuda()
    cid = 5
    cfg = S.get_config(cid)
    K = cfg.n_devices
    stream = torch.cuda.current_stream()
    rates = S.make_arrival_rates(cid)
    counts = S.make_arrival_counts(cid, rates, steps, sub=counts_sub)
    acts = S.make_acts(cid, bank_n, batch=B, sub=7)
    labels = S.make_labels(cid, bank_n, batch=B, sub=7)
    acts_d = torch.from_numpy(acts.view(np.int16)).cuda()
    labels_d = torch.from_numpy(labels).cuda()
    slot_bytes = acts[0].nbytes
    g0 = S.make_global_vector(cid, sub=7)
    locs = S.make_local_vectors(cid, K, sub=7)
    gd = torch.from_numpy(g0.copy()).cuda()
    ld = torch.from_numpy(locs).cuda()
    model = A.fo_model_create(cid, B, S.init_params(cid), stream)
    q = A.fo_queues_create(K, slot_bytes, B, False, n_slots, stream)
    A.fo_set_max_delay(-1)
    sch = TaskScheduler(K, n_slots)
    dev_version = [0] * K
    bank_of = {}
    nxt = 0
    trained = drains = 0
    sampled = []
    ls_all, ss_all = [], []
    want, bank_i = [], []
    try:
        for t in range(steps):
            senders = []
            for k in np.nonzero(counts[t])[0].tolist():
                for _ in range(int(counts[t][k])):
                    i = nxt % bank_n
                    nxt += 1
                    ok, seq, _ = sch.put_act(k)
                    if batched:
                        want.append(ok)
                        bank_i.append(i)
                    else:
                        st = A.fo_queues_push(q, k, acts_d[i], labels_d[i])
                        assert (st == A.FO_OK) == ok, (t, k)
                    if ok:
                        bank_of[(k, seq)] = i
                    sch.put_model(k, dev_version[k])
                    if not batched:
                        A.fo_queues_push_model(q, k, ld[k], dev_version[k])
                    senders.append(k)
            if batched and senders:
                bi_ = np.array(bank_i, np.uint64)
                st = A.fo_queues_push_batch(q, senders, acts_d.data_ptr() + bi_ * slot_bytes,
                                            labels_d.data_ptr() + bi_ * (4 * B))
                assert st.tolist() == [A.FO_OK if ok else A.FO_FULL for ok in want], t
                ks_ = np.array(senders, np.int64)
                A.fo_queues_push_model_batch(q, senders, ld.data_ptr() + ks_ * (4 * ld.shape[1]), ld.shape[1],
                                             [dev_version[k] for k in senders])
            want, bank_i = [], []
            k = A.fo_pick_device(q)
            if k == -2:
                n0 = len(ls_all)
                while sch.q_model:
                    kind, kk, t_k = sch.get()
                    assert kind == "model"
                    ok, s = sch.aggregate_version(t_k)
                    assert ok
                    ls_all.append(kk)
                    ss_all.append(s)
                applied, skipped = A.fo_aggregate_pending_all(q, gd, 1.0)
                assert (applied, skipped) == (len(ls_all) - n0, 0)
                v = A.fo_queues_stats(q).version
                assert v == sch.t
                for kk in senders:
                    dev_version[kk] = v
                drains += 1
                k = A.fo_pick_device(q)
            r = sch.get()
            if r is None:
                assert k == -1
                continue
            assert r[0] == "act" and k == r[1], (t, k, r)
            fa, lab, seq, slot = A.fo_queues_in_service(q)
            assert (seq, slot) == (r[2], r[3]), (t, k, seq, slot, r)
            bi = bank_of[(k, seq)]
            got = _d2h(torch, fa.x, slot_bytes)
            assert np.array_equal(got, acts[bi].view(np.uint8).reshape(-1)), (k, seq, slot)
            got_lab = _d2h(torch, lab, 4 * B).view(np.int32)
            assert np.array_equal(got_lab, labels[bi]), (k, seq, slot)
            before = A.fo_model_read(model, A.FO_BUF_PARAMS) if t in sample_steps else None
            A.fo_server_step(model, fa, lab, k)
            A.fo_queues_release(q)
            sch.release()
            trained += 1
            if before is not None:
                announce(f"128-device loop: oracle check of step {t} (device {k}, seq {seq}, slot {slot})")
                rr = oracle.server_step(cid, before, acts[bi], labels[bi], lr=cfg.lr)
                loss = A.fo_model_read(model, A.FO_BUF_LOSS)[0]
                logits = A.fo_model_read(model, A.FO_BUF_LOGITS).reshape(B, cfg.n_classes)
                after = A.fo_model_read(model, A.FO_BUF_PARAMS).astype(np.float64)
                rec = dict(step=t, loss=abs(loss - rr["loss"]) / abs(rr["loss"]),
                           logits=normwise(logits, rr["logits"]),
                           update=_frob(after - before, rr["params"] - before))
                sampled.append(rec)
                assert rec["loss"] <= TOL and rec["logits"] <= TOL, rec
                assert rec["update"] <= GRAD_TOL, rec
        st = A.fo_queues_stats(q)
        assert A.fo_queues_counters(q, K) == sch.c
        assert (st.refused, st.peak_queued, st.queued, st.version) == (sch.refused, sch.peak_queued, sch.queued(),
                                                                       sch.t)
        assert trained == steps and drains == steps
        ref_g, _ = OA.mix_sequence(g0, [locs[kk] for kk in ls_all], [1.0] * len(ls_all), ss_all)
        assert normwise(gd.cpu().numpy(), ref_g) <= 1e-4
    finally:
        A.fo_queues_destroy(q)
        A.fo_model_destroy(model)
    return dict(refused=st.refused, peak=st.peak_queued, omega=st.omega, sampled=sampled)


def test_vgg128_loop_matches_oracle():
    """A small pool (600 slots) so that the cap binds within a few steps; batch 4;
    every step's training compared with the oracle."""
    announce("128-device loop, 12 steps, pool 600 slots, batch 4")
    out = _run_loop(B=4, steps=12, n_slots=600, bank_n=8, counts_sub=7, sample_steps=tuple(range(12)))
    assert out["refused"] > 0 and len(out["sampled"]) == 12


def test_vgg128_loop_workload_scale():
    """The workload's own sizes: batch 64, a 64 GiB pool of 2 MiB slots
    (32,768 slots, omega = 32,640), the benchmark's arrival table, run past
    step 161 where the cap starts refusing arrivals."""
    steps = 175
    announce(f"128-device loop at workload scale, {steps} steps, pool 32768 slots, batch 64")
    out = _run_loop(B=64, steps=steps, n_slots=(64 << 30) // (2 << 20), bank_n=16, counts_sub=0,
                    sample_steps=(0, steps - 1), batched=True)
    print(out)
    assert out["refused"] > 0 and out["peak"] >= out["omega"]
    assert len(out["sampled"]) == 2
