"""Pins for the oracle's aggregation and Task Scheduler (CPU only)."""
import itertools

import numpy as np
import pytest

import fo_synth as S
from oracle import aggregate as A
from oracle.scheduler import TaskScheduler
from tests.golden_io import fmt_get, read_trace, read_weights


# ----------------------------------------------------------------------------- aggregation
def test_weights_golden():
    for a, s, w in read_weights():
        assert A.weight(a, s) == w


def _vecs(n=10_000):
    g = S.make_global_vector(1, n)
    l = S.make_local_vectors(1, 4, n)
    return g, l


def test_alpha_zero_is_identity():
    g, l = _vecs()
    for s in range(4):
        out, ok = A.mix(g, l[0], 0.0, s)
        assert ok and out.tobytes() == g.tobytes()


def test_equal_models_reproduce_the_model():
    g, _ = _vecs()
    for a in (0.5, 1.0, 0.3):
        for s in range(5):
            out, _ = A.mix(g, g, a, s)
            assert out.tobytes() == g.tobytes()


def test_alpha_one_fresh_takes_local():
    g, l = _vecs()
    out, _ = A.mix(g, l[1], 1.0, 0)
    assert out.tobytes() == l[1].tobytes()


def test_max_delay_skips():
    g, l = _vecs()
    out, ok = A.mix(g, l[0], 1.0, 5, max_delay=4)
    assert not ok and out.tobytes() == g.tobytes()
    out, ok = A.mix(g, l[0], 1.0, 4, max_delay=4)
    assert ok and out.tobytes() != g.tobytes()


def test_sequence_matches_closed_form():
    """m sequential mixes = prod(1-w_i) g0 + sum_i w_i prod_{j>i}(1-w_j) l_i."""
    g, l = _vecs(2000)
    ws = [(0.5, 0), (0.5, 1), (0.5, 2), (0.5, 3)]
    out, _ = A.mix_sequence(g, l, [a for a, _ in ws], [s for _, s in ws])
    w = [a / (s + 1) for a, s in ws]
    ref = np.prod([1 - x for x in w]) * g.astype(np.float64)
    for i in range(4):
        ref = ref + w[i] * np.prod([1 - x for x in w[i + 1:]]) * l[i].astype(np.float64)
    # 4 roundings to fp32, each at most half an ulp of values of size <= max|.|
    bound = 4 * 2.0 ** -24 * max(np.abs(g).max(), np.abs(l).max())
    assert np.abs(out.astype(np.float64) - ref).max() <= bound


# ----------------------------------------------------------------------------- scheduler
def _run_trace(name, K, n_slots, with_slot, policy="counter"):
    sch = TaskScheduler(K, n_slots, policy=policy)
    for op, args, exp in read_trace(name):
        if op == "put_act":
            ok, seq, slot = sch.put_act(args[0])
            got = "refuse" if not ok else (f"admit seq={seq}" + (f" slot={slot}" if with_slot else ""))
        elif op == "put_model":
            sch.put_model(args[0], args[1])
            got = "-"
        elif op == "get":
            r = sch.get()
            if r is not None and r[0] == "act":
                r = r + (list(sch.c),)
            got = fmt_get(r, K, with_slot)
        elif op == "release":
            sch.release()
            got = "-"
        elif op in ("leave", "join"):
            sch.set_active(args[0], op == "join")
            got = "-"
        assert got == exp, (op, args, got, exp)
    return sch


def test_golden_scheduler_trace():
    _run_trace("sched_trace_k3.txt", 3, None, False)


def test_golden_flow_control_trace():
    sch = _run_trace("flow_trace_k2.txt", 2, 4, True)
    assert sch.refused == 3


def test_golden_fifo_leave_trace():
    sch = _run_trace("fifo_leave_trace_k3.txt", 3, 5, True, policy="fifo")
    assert sch.refused == 2 and sch.turn_on_signals == 5


def test_fifo_matches_one_global_queue_random_trace():
    """FIFO against an independent statement: one list of every admitted
    batch in admission order, served from its head; devices leave and rejoin
    at random and the memory bound of the flow control still holds."""
    K, n_slots = 5, 12
    rng = np.random.default_rng(11)
    sch = TaskScheduler(K, n_slots, policy="fifo")
    order = []
    active = [True] * K
    for step in range(2000):
        k = int(rng.integers(K))
        if rng.random() < 0.05:
            active[k] = not active[k]
            sch.set_active(k, active[k])
        for k in range(K):
            for _ in range(rng.poisson(0.8)):
                ok, seq, _ = sch.put_act(k)
                assert not (ok and not active[k])  # a device that left sends nothing
                if ok:
                    order.append((k, seq))
        assert sch.queued() <= sch.omega + K - 1
        r = sch.get()
        if order:
            assert r[:3] == ("act",) + order.pop(0)
            sch.release()
        else:
            assert r is None
    assert sch.refused > 0 and sch.turn_on_signals > 0


def test_counter_and_fifo_differ_on_skewed_arrivals():
    """Device 0 sends three batches per server step, device 1 one every third
    step, and the server trains on one batch per step, so a backlog builds.
    The counter policy serves device 1's batches as they come (c_1 = all 67
    of them); FIFO serves the backlog in arrival order, and device 1 gets
    only its share of the first 200 arrivals (the effect Sec. 6.5 measures)."""
    res = {}
    for policy in ("counter", "fifo"):
        sch = TaskScheduler(2, policy=policy)
        for step in range(200):
            for _ in range(3):
                sch.put_act(0)
            if step % 3 == 0:
                sch.put_act(1)
            sch.get()
            sch.release()
        res[policy] = list(sch.c)
    assert res["counter"] == [133, 67]
    assert res["fifo"][1] <= 20 and sum(res["fifo"]) == 200


def _brute_force_pick(queues, c):
    """Independent chooser: sort every non-empty device by (count, index)."""
    cands = sorted((c[k], k) for k in range(len(queues)) if queues[k])
    return None if not cands else cands[0][1]


@pytest.mark.parametrize("K", [1, 2, 3])
def test_brute_force_all_interleavings(K):
    alphabet = [("put", k) for k in range(K)] + [("get", None), ("model", None)]
    n = 0
    for length in range(1, 6 if K < 3 else 5):
        for seq in itertools.product(alphabet, repeat=length):
            sch = TaskScheduler(K)
            queues = [[] for _ in range(K)]
            models = []
            c = [0] * K
            nxt = [0] * K
            for op, k in seq:
                if op == "put":
                    sch.put_act(k)
                    queues[k].append(nxt[k])
                    nxt[k] += 1
                elif op == "model":
                    sch.put_model(0, 7)
                    models.append(7)
                else:
                    r = sch.get()
                    if models:
                        assert r == ("model", 0, models.pop(0))
                        continue
                    kk = _brute_force_pick(queues, c)
                    if kk is None:
                        assert r is None
                    else:
                        assert r[:3] == ("act", kk, queues[kk].pop(0))
                        c[kk] += 1
                n += 1
            assert sch.c == c
    assert n > 0


def test_always_nonempty_is_round_robin_and_balanced():
    K = 5
    sch = TaskScheduler(K)
    for _ in range(40):
        for k in range(K):
            sch.put_act(k)
    picks = []
    for _ in range(100):
        r = sch.get()
        picks.append(r[1])
        assert max(sch.c) - min(sch.c) <= 1
        for k in range(K):
            sch.put_act(k)
    assert picks == [i % K for i in range(100)]
    assert sum(sch.c) == 100


def test_flow_control_bounds_memory_random_trace():
    K, n_slots = 6, 14
    rng = np.random.default_rng(3)
    sch = TaskScheduler(K, n_slots)
    in_use_max = 0
    for step in range(3000):
        for k in range(K):
            for _ in range(rng.poisson(1.5 if k % 2 else 0.3)):
                sch.put_act(k)
        in_use = sch.queued() + (sch.in_service is not None)
        in_use_max = max(in_use_max, in_use)
        assert sch.queued() <= sch.omega + K - 1
        assert len(sch.free) + sch.queued() + (1 if sch.in_service is not None else 0) == n_slots
        r = sch.get()
        if r is not None:
            sch.release()
    assert in_use_max <= n_slots
    assert sch.refused > 0


def test_versions_and_max_delay():
    sch = TaskScheduler(2)
    assert sch.aggregate_version(0) == (True, 0) and sch.t == 1
    assert sch.aggregate_version(0, max_delay=0) == (False, 1) and sch.t == 1
    assert sch.aggregate_version(0, max_delay=1) == (True, 1) and sch.t == 2


def test_join_starts_at_zero_count():
    sch = TaskScheduler(2)
    for _ in range(3):
        sch.put_act(0)
        sch.put_act(1)
    for _ in range(4):
        sch.get()
    k = sch.add_device()
    sch.put_act(k)
    assert sch.get()[1] == k  # c_k = 0 is the smallest counter
