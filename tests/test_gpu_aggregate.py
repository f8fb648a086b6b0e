"""GPU parity of the aggregation kernels (Alg. 4, aggregation branch)
against the oracle, through the C ABI."""
import numpy as np
import pytest

import fo_synth as S
from oracle import aggregate as OA
from tests.gpu_util import announce, normwise, to_dev, torch_cuda

pytestmark = pytest.mark.gpu
A = pytest.importorskip("paper_2504_13850_amd.api")

TOL = 1e-4


def _vecs(n, m=4, sub=0):
    g = S.make_global_vector(1, n, sub=sub)
    l = S.make_local_vectors(1, m, n, sub=sub)
    return g, l


@pytest.mark.parametrize("n", [1, 3, 5, 1001, 4099, 10_000, 38_720, 157_504])
def test_single_mix_matches_oracle(n):
    torch = torch_cuda()
    announce(f"aggregate n={n}")
    g, l = _vecs(n)
    for alpha, s in [(0.5, 0), (0.5, 1), (0.5, 2), (0.5, 3), (1.0, 0), (1.0, 7), (0.3, 2)]:
        gd, ld = to_dev(g), to_dev(l[1])
        assert A.fo_async_aggregate(gd, ld, alpha, s) == A.FO_OK
        ref, _ = OA.mix(g, l[1], alpha, s)
        got = gd.cpu().numpy()
        assert normwise(got, ref) <= TOL, (alpha, s)
        # elementwise: one rounding of the difference and one of the FMA
        assert np.abs(got - ref).max() <= 4 * 2.0 ** -24 * (np.abs(g).max() + np.abs(l[1]).max())
    torch.cuda.synchronize()


def test_identities_bit_exact():
    torch_cuda()
    announce("aggregate identities")
    g, l = _vecs(10_007)
    gd = to_dev(g)
    for s in range(5):
        A.fo_async_aggregate(gd, to_dev(l[0]), 0.0, s)          # alpha = 0
        A.fo_async_aggregate(gd, to_dev(g.copy()), 0.7, s)      # equal models
    assert gd.cpu().numpy().tobytes() == g.tobytes()
    # alpha = 1, fresh model: the global becomes the local one up to the two
    # roundings of g + 1 * (l - g): |err| <= u (|l - g| + |l|), u = 2^-24,
    # which is at most one ulp of max(|l - g|, |l|)
    A.fo_async_aggregate(gd, to_dev(l[2]), 1.0, 0)
    got = gd.cpu().numpy()
    bound = np.spacing(np.maximum(np.abs(l[2] - g), np.abs(l[2])))
    assert np.all(np.abs(got - l[2]) <= bound)


def test_max_delay_skips_and_config1_sequence():
    torch_cuda()
    announce("aggregate max delay + config-1 sequence")
    g, l = _vecs(10_000)
    gd = to_dev(g)
    try:
        A.fo_set_max_delay(2)
        assert A.fo_async_aggregate(gd, to_dev(l[0]), 1.0, 3) == A.FO_SKIPPED
        assert gd.cpu().numpy().tobytes() == g.tobytes()
    finally:
        A.fo_set_max_delay(-1)
    # the tiny-CNN workload: alpha = 0.5, device k arrives with staleness k
    for k in range(4):
        A.fo_async_aggregate(gd, to_dev(l[k]), 0.5, k)
    ref, _ = OA.mix_sequence(g, l, [0.5] * 4, [0, 1, 2, 3])
    assert normwise(gd.cpu().numpy(), ref) <= TOL


@pytest.mark.parametrize("n,m", [(38_720, 5), (157_504, 70), (4097, 130)])
def test_fused_drain_equals_sequential_bit_exact(n, m):
    """fo_aggregate_pending_all applies every pending message in one pass per
    64 messages; it must equal m single fo_aggregate_pending calls bit for bit."""
    torch_cuda()
    announce(f"fused drain n={n} m={m}")
    g, l = _vecs(n, m)
    locs = [to_dev(l[i]) for i in range(m)]
    # message i arrives while the global version is i; its device version lags by 0..3
    lag = S.make_staleness(5, m, 3)
    versions = [max(0, i - int(lag[i])) for i in range(m)]
    outs = []
    for fused in (False, True):
        q = A.fo_queues_create(4, 0, 1, False, 16)
        try:
            gd = to_dev(g)
            for i in range(m):
                A.fo_queues_push_model(q, i % 4, locs[i], int(versions[i]))
            if fused:
                applied, skipped = A.fo_aggregate_pending_all(q, gd, 1.0)
                assert applied + skipped == m
            else:
                while A.fo_aggregate_pending(q, gd, 1.0)[0] != A.FO_EMPTY:
                    pass
            outs.append(gd.cpu().numpy())
            version = A.fo_queues_stats(q).version
        finally:
            A.fo_queues_destroy(q)
    assert outs[0].tobytes() == outs[1].tobytes()
    # and both follow the oracle's sequence of mixes
    stal = [i - versions[i] for i in range(m)]
    assert version == m
    ref, _ = OA.mix_sequence(g, l, [1.0] * m, stal)
    assert normwise(outs[1], ref) <= TOL


@pytest.mark.parametrize("n", [(1 << 26) + 3, 1 << 28])
def test_large_vector_sampled(n):
    """Large vectors, among them the benchmark's 2^28 elements (1 GiB each, the
    size the HBM figure is measured at, same call and launch shape): a random
    sample of elements plus the tail checked against the oracle's mix."""
    torch = torch_cuda()
    announce(f"aggregate n={n}")
    g = S.make_global_vector(1, n, sub=5)
    l = S.make_local_vectors(1, 1, n, sub=5)[0]
    gd, ld = to_dev(g), to_dev(l)
    A.fo_async_aggregate(gd, ld, 1.0, 3)
    rng = np.random.default_rng(5)
    idx = np.concatenate([rng.integers(0, n, 200_000), np.arange(n - 8, n)])
    outs = gd[torch.from_numpy(idx).cuda()].cpu().numpy()
    gs, ls = g[idx], l[idx]
    del gd, ld
    ref, applied = OA.mix(gs, ls, 1.0, 3)
    assert applied
    assert normwise(outs, ref) <= TOL
    # elementwise: within two fp32 roundings of the oracle's once-rounded mix
    assert np.all(np.abs(outs.astype(np.float64) - ref) <= 2 * 2.0 ** -24 * (np.abs(ls - gs) + np.abs(ref)) + 1e-45)
