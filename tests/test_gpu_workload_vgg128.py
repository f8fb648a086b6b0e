"""GPU test of the 128-device workload loop: lognormal device rates, Poisson
arrivals per server step, each arrival an activation batch put into the HBM
pool under flow control (Alg. 2, Sec. 3.4.1) and a model message; pending
models are aggregated first in fused drains (Alg. 3, Alg. 4 aggregation
branch), then one batch is picked and trained on.  Checked against the oracle
scheduler and aggregation through the C ABI:
  - every admission, pick, sequence number, slot id, counter, refusal count,
    peak occupancy and version bit for bit;
  - the bytes in the slot of the batch in service are the bytes pushed for
    that (device, sequence);
  - the global model equals the oracle's FIFO sequence of staleness-weighted
    mixes (fp64, rounded to fp32 after each) within 1e-4 normwise."""
import ctypes
import os

import numpy as np
import pytest

import fo_synth as S
from oracle import aggregate as OA
from oracle.scheduler import TaskScheduler
from tests.gpu_util import announce, normwise, torch_cuda

pytestmark = pytest.mark.gpu
A = pytest.importorskip("paper_2504_13850_amd.api")


def _d2h(torch, ptr, nbytes):
    """Device bytes at a raw pointer, through the process's HIP runtime (torch's)."""
    hip = ctypes.CDLL(os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so"))
    out = np.empty(nbytes, np.uint8)
    torch.cuda.synchronize()
    rc = hip.hipMemcpy(ctypes.c_void_p(out.ctypes.data), ctypes.c_void_p(ptr), ctypes.c_size_t(nbytes),
                       ctypes.c_int(2))  # hipMemcpyDeviceToHost
    assert rc == 0, rc
    return out


def test_vgg128_loop_matches_oracle():
    torch = torch_cuda()
    cid = 5
    cfg = S.get_config(cid)
    K = cfg.n_devices
    B, steps, n_slots, bank_n = 4, 12, 600, 8  # a small pool: the cap binds within a few steps
    announce(f"128-device loop, {steps} steps, pool {n_slots} slots")
    stream = torch.cuda.current_stream()
    rates = S.make_arrival_rates(cid)
    counts = S.make_arrival_counts(cid, rates, steps, sub=7)
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
    ref_g = g0.copy()
    dev_version = [0] * K
    bank_of = {}
    nxt = 0
    trained = drains = 0
    try:
        for t in range(steps):
            senders = []
            for k in np.nonzero(counts[t])[0].tolist():
                for _ in range(int(counts[t][k])):
                    i = nxt % bank_n
                    nxt += 1
                    ok, seq, _ = sch.put_act(k)
                    st = A.fo_queues_push(q, k, acts_d[i], labels_d[i])
                    assert (st == A.FO_OK) == ok
                    if ok:
                        bank_of[(k, seq)] = i
                    sch.put_model(k, dev_version[k])
                    A.fo_queues_push_model(q, k, ld[k], dev_version[k])
                    senders.append(k)
            k = A.fo_pick_device(q)
            if k == -2:
                ls, ss = [], []
                while sch.q_model:
                    kind, kk, t_k = sch.get()
                    assert kind == "model"
                    ok, s = sch.aggregate_version(t_k)
                    assert ok
                    ls.append(locs[kk])
                    ss.append(s)
                ref_g, _ = OA.mix_sequence(ref_g, ls, [1.0] * len(ls), ss)
                applied, skipped = A.fo_aggregate_pending_all(q, gd, 1.0)
                assert (applied, skipped) == (len(ls), 0)
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
            assert r[0] == "act" and k == r[1]
            fa, lab, seq, slot = A.fo_queues_in_service(q)
            assert (seq, slot) == (r[2], r[3])
            got = _d2h(torch, fa.x, slot_bytes)
            assert np.array_equal(got, acts[bank_of[(k, seq)]].view(np.uint8).reshape(-1)), (k, seq, slot)
            A.fo_server_step(model, fa, lab, k)
            A.fo_queues_release(q)
            sch.release()
            trained += 1
        st = A.fo_queues_stats(q)
        assert A.fo_queues_counters(q, K) == sch.c
        assert (st.refused, st.peak_queued, st.queued, st.version) == (sch.refused, sch.peak_queued, sch.queued(),
                                                                       sch.t)
        assert st.refused > 0 and trained == steps and drains == steps
        assert np.isfinite(A.fo_model_read(model, A.FO_BUF_LOSS)[0])
        assert normwise(gd.cpu().numpy(), ref_g) <= 1e-4
    finally:
        A.fo_queues_destroy(q)
        A.fo_model_destroy(model)
