"""The concurrent server pipeline (fo_pipeline_run: Receiver and Compute
Engine threads of Sec. 5.1, flow control of Sec. 3.4.1, devices leaving and
rejoining under the dropout of Sec. 6.4) on the GPU, through the C ABI.

What a free-running concurrent run must satisfy, checked exactly:
* its pool event record replays through the oracle's Task Scheduler event by
  event (every admission or refusal, every pick's device, sequence number and
  slot, every aggregation's staleness and skip decision, every leave and
  rejoin), under both scheduling policies;
* the pipeline's counters agree with that record;
* the aggregated global model equals the oracle's mixing sequence over the
  record's aggregations (<= 1e-4 relative, as for sequential aggregation);
* the trained server model is bit-identical to a second model stepped
  sequentially through the same batches in the record's pick order, so the
  engine trained every picked batch exactly once, in order, with no slot
  overwritten while a step read it (pool and model on different streams).
The throughput retention R(p) = T(p) / T(0) of Sec. 6.4 is checked for its
two regimes: a server-bound system keeps its throughput when devices drop
out, a device-bound one loses about the share of devices away."""
import numpy as np
import pytest

import fo_synth as S
import oracle
from tests.gpu_util import announce, to_dev, torch_cuda
from tests.pool_log import EV_JOIN, EV_LEAVE, EV_MODEL, EV_PUSH, replay

pytestmark = pytest.mark.gpu
A = pytest.importorskip("paper_2504_13850_amd.api")

CID = 1
N_AGG = 4096


def _setup(torch, K, B, n_slots, bank_n, n_local, sub):
    cfg = S.get_config(CID)
    slot_bytes = B * int(np.prod(cfg.in_shape)) * 4
    model_stream = torch.cuda.current_stream()
    pool_stream = torch.cuda.Stream()
    theta = S.init_params(CID)
    m = A.fo_model_create(CID, B, theta, model_stream)
    q = A.fo_queues_create(K, slot_bytes, B, False, n_slots, pool_stream)
    xs = S.make_acts(CID, bank_n, batch=B, sub=sub)
    ls = S.make_labels(CID, bank_n, batch=B, sub=sub)
    loc = S.make_local_vectors(CID, n_local, n=N_AGG, sub=sub)
    g0 = S.make_global_vector(CID, n=N_AGG, sub=sub)
    bufs = dict(x=to_dev(xs), l=to_dev(ls), loc=to_dev(loc), g=to_dev(g0))
    return theta, m, q, xs, ls, loc, g0, bufs, model_stream


def _run(torch, K, B, n_slots, periods, seconds, p_drop, policy, D, sub, seed, bank_n=24, n_local=5, alpha=0.6,
         log_cap=2_000_000):
    theta, m, q, xs, ls, loc, g0, bufs, stream = _setup(torch, K, B, n_slots, bank_n, n_local, sub)
    A.fo_queues_set_policy(q, A.FO_SCHED_COUNTER if policy == "counter" else A.FO_SCHED_FIFO)
    A.fo_queues_log_enable(q, log_cap)
    A.fo_set_max_delay(-1 if D is None else D)
    try:
        st = A.fo_pipeline_run(q, m, bufs["g"], dict(
            seconds=seconds, iter_seconds=periods, H=4, p_drop=p_drop, interval_seconds=0.1, slow_max=2.0,
            seed=seed, bank_x=bufs["x"], bank_labels=bufs["l"], bank_n=bank_n, local_bank=bufs["loc"],
            n_local=n_local, alpha=alpha, max_inflight=2))
        torch.cuda.synchronize()
        log = A.fo_queues_log_read(q, log_cap)
        out = dict(st=st, log=log, qs=A.fo_queues_stats(q), theta=theta, xs=xs, ls=ls, loc=loc, g0=g0,
                   g=bufs["g"].cpu().numpy(), params=A.fo_model_read(m, A.FO_BUF_PARAMS),
                   c=A.fo_queues_counters(q, K), bank_n=bank_n, n_local=n_local, alpha=alpha)
    finally:
        A.fo_set_max_delay(-1)
        A.fo_queues_destroy(q)
        A.fo_model_destroy(m)
    assert log_cap < 1000 or len(out["log"]) < log_cap
    return out


@pytest.mark.parametrize("policy", ["counter", "fifo"])
def test_concurrent_run_is_a_valid_sequential_interleaving(policy):
    torch = torch_cuda()
    K, B, n_slots, D = 8, 8, 20, 3
    periods = 1e-3 * np.exp(np.random.default_rng(5).normal(0.0, 0.5, K))
    announce(f"pipeline policy={policy} K={K} B={B} 0.8 s, p=0.3")
    r = _run(torch, K, B, n_slots, periods, 0.8, 0.3, policy, D, sub=41, seed=9)
    st, log = r["st"], r["log"]
    print(f"steps={st.steps} samples={st.samples} aggs={st.aggregations} skipped={st.skipped} sent={st.sent} "
          f"not_sent={st.not_sent} models={st.models_sent} leaves={st.leaves} rejoins={st.rejoins} "
          f"idle={st.idle_seconds:.3f}/{st.wall_seconds:.3f} s events={len(log)}", flush=True)
    sch, picks, aggs = replay(log, K, n_slots, policy, D)
    # counters agree with the record
    typ, a = log[:, 0], log[:, 2]
    assert st.steps == len(picks) == r["qs"].picks and st.samples == B * st.steps
    assert st.sent == int(((typ == EV_PUSH) & (a == 1)).sum()) == r["qs"].admitted
    assert st.not_sent == int(((typ == EV_PUSH) & (a == 0)).sum()) == r["qs"].refused
    assert st.models_sent == int((typ == EV_MODEL).sum())
    assert st.aggregations == sum(1 for x in aggs if x[3]) and st.skipped == sum(1 for x in aggs if not x[3])
    assert st.leaves <= int((typ == EV_LEAVE).sum()) and st.rejoins == int((typ == EV_JOIN).sum())
    assert sch.c == r["c"] and sch.t == r["qs"].version
    assert st.steps > 100 and st.aggregations > 5 and st.leaves > 0 and st.not_sent > 0
    assert 0.0 <= st.idle_seconds <= st.wall_seconds
    # the global model: the oracle's mixing sequence over the record's aggregations
    locs = [r["loc"][(k + ri) % r["n_local"]] for k, ri, _, _ in aggs]
    ref, applied = oracle.mix_sequence(r["g0"], locs, [r["alpha"]] * len(aggs), [s for _, _, s, _ in aggs], D)
    assert applied == [x[3] for x in aggs]
    err = np.abs(r["g"].astype(np.float64) - ref).max() / np.abs(ref).max()
    assert err <= 1e-4, err
    # the server model: bit-identical to stepping the picked batches in order
    stream = torch.cuda.current_stream()
    m2 = A.fo_model_create(CID, B, r["theta"], stream)
    try:
        x_d, l_d = to_dev(r["xs"]), to_dev(r["ls"])
        for k, seq in picks:
            e = (k + seq) % r["bank_n"]
            A.fo_server_step(m2, (x_d[e], None, B), l_d[e], k)
        p2 = A.fo_model_read(m2, A.FO_BUF_PARAMS)
    finally:
        A.fo_model_destroy(m2)
    assert np.array_equal(p2, r["params"])
    assert not np.array_equal(p2, r["theta"])


def test_retention_under_dropout_follows_the_bottleneck():
    """R(0.5) for a server-bound system (devices send far faster than the
    server trains) stays near 1; for a device-bound one it falls to about the
    share of devices present."""
    torch = torch_cuda()
    K, B, n_slots = 16, 16, 40
    res = {}
    for regime, period in (("server-bound", 2e-4), ("device-bound", 2e-2)):
        periods = np.full(K, period)
        for p in (0.0, 0.5):
            announce(f"retention {regime} p={p}")
            r = _run(torch, K, B, n_slots, periods, 0.6, p, "counter", None, sub=43, seed=13, log_cap=1)
            res[(regime, p)] = r["st"].samples / r["st"].wall_seconds
    R_server = res[("server-bound", 0.5)] / res[("server-bound", 0.0)]
    R_device = res[("device-bound", 0.5)] / res[("device-bound", 0.0)]
    print(f"T: {res}  R(0.5) server-bound {R_server:.3f}, device-bound {R_device:.3f}", flush=True)
    assert R_server >= 0.85
    assert 0.2 <= R_device <= 0.8
