"""The library's pre-processor (fo_net_units, fo_select_split,
fo_aux_network; Sec. 3.2.1 Eq. 6-8, Sec. 3.2.2) against the oracle, on the
CPU: every unit of every network field by field, the split and every cost
bit for bit (both sides evaluate the same fp64 expressions in the same
order), and the auxiliary networks."""
import time

import numpy as np
import pytest

from oracle import preproc as P

A = pytest.importorskip("paper_2504_13850_amd.api")

NETS = [(A.FO_NET_VGG5, "vgg5", 10, 32), (A.FO_NET_VGG16, "vgg16", 10, 32),
        (A.FO_NET_MOBILENETV3_LARGE, "mobilenetv3_large", 200, 64),
        (A.FO_NET_MOBILENETV3_LARGE, "mobilenetv3_large", 1000, 224),
        (A.FO_NET_TRANSFORMER6, "transformer6", 2, 64), (A.FO_NET_TRANSFORMER12, "transformer12", 2, 512)]


def _same(got, ref):
    d = got.as_dict()
    for key, v in ref.items():
        assert d[key] == v, (key, d[key], v)


@pytest.mark.parametrize("net,name,classes,hw", NETS)
def test_units_match_oracle(net, name, classes, hw):
    units = A.fo_net_units(net, classes, hw)
    ref = P.net_layers(name, classes, hw)
    assert len(units) == len(ref)
    for u, r in zip(units, ref):
        _same(u, r)


@pytest.mark.parametrize("net,name,classes,hw", NETS)
def test_split_and_aux_match_oracle(net, name, classes, hw):
    units = A.fo_net_units(net, classes, hw)
    ref = P.net_layers(name, classes, hw)
    rng = np.random.default_rng(net * 7 + hw)
    for trial in range(40):
        K = int(rng.integers(1, 129))
        o = rng.uniform(1e9, 2e12, K)   # device FLOP/s
        b = rng.uniform(2e6, 2e8, K)    # device bytes/s
        batch, nbytes = int(rng.choice([16, 32, 64])), int(rng.choice([2, 4]))
        l, costs = A.fo_select_split(units, batch, nbytes, o, b)
        lr, cr = P.select_split(ref, batch, nbytes, list(o), list(b))
        assert l == lr and costs.tolist() == cr
        if any(r["kind"] != P.POOL for r in ref[:l]):
            aux = A.fo_aux_network(units, l, classes)
            aux_r = P.aux_network(ref, l, classes)
            assert len(aux) == len(aux_r)
            for u, r in zip(aux, aux_r):
                _same(u, r)


def test_golden_split_through_the_library():
    from tests.test_oracle_preproc import _golden_split
    units_r, devs, costs, split = _golden_split()
    arr = (A.fo_unit * len(units_r))()
    for i, r in enumerate(units_r):
        for key, v in r.items():
            setattr(arr[i], key, v)
    l, c = A.fo_select_split(arr, 1, 1, [d[0] for d in devs], [d[1] for d in devs])
    assert l == split and c.tolist() == costs


def test_errors_and_speed():
    with pytest.raises(A.FoError):
        A.fo_net_units(99, 10, 32)
    with pytest.raises(A.FoError):
        A.fo_net_units(A.FO_NET_VGG16, 10, 30)  # needs five halvings
    units = A.fo_net_units(A.FO_NET_TRANSFORMER12, 2, 512)
    with pytest.raises(A.FoError):
        A.fo_select_split(units, 16, 4, [1e9, 0.0], [1e6, 1e6])
    with pytest.raises(A.FoError):
        A.fo_aux_network(units, 0, 2)
    # a 128-device selection is microseconds of host work (the paper bounds the
    # whole initialization stage by seconds)
    o, b = np.full(128, 1e10), np.full(128, 1e7)
    t0 = time.perf_counter()
    for _ in range(100):
        A.fo_select_split(units, 16, 4, o, b)
    assert (time.perf_counter() - t0) / 100 < 0.01
