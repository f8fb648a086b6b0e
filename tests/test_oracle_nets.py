"""Pins for the oracle's whole server networks and training step (CPU only).

* the flat parameter layout the oracle derives equals the workload description,
* loss, logits and every gradient equal an independent fp64 autograd
  implementation (PyTorch CPU),
* central finite differences of the loss on sampled parameters,
* closed forms: zero classifier gives loss ln C; lr = 0 leaves parameters
  unchanged; momentum buffer recursion; padded tokens never matter."""
import numpy as np
import pytest

import fo_synth as S
import oracle
from oracle import nets
from tests import torch_ref

SMALL_B = {1: 3, 2: 2, 3: 4, 4: 2, 5: 2, 6: 2, 7: 3, 8: 2, 9: 3, 10: 3}


def _inputs(cid, B, sub=7):
    acts = S.make_acts(cid, 1, batch=B, sub=sub)[0]
    labels = S.make_labels(cid, 1, batch=B, sub=sub)[0]
    lengths = S.make_lengths(cid, 1, batch=B, sub=sub)[0] if cid in (4, 7, 8) else None
    return acts, labels, lengths


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5, 6, 7, 8, 9, 10])
def test_layout_matches_workload(cid):
    a = [(n, tuple(s)) for n, s in nets.param_layout(cid)]
    b = [(n, tuple(s)) for n, s, _, _ in S.param_layout(cid)]
    assert a == b
    assert sum(int(np.prod(s)) for _, s in a) == S.param_count(cid)


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 6, 7, 8, 9, 10])
def test_step_matches_independent_autograd(cid):
    B = SMALL_B[cid]
    theta = S.init_params(cid)
    acts, labels, lengths = _inputs(cid, B)
    r = oracle.server_step(cid, theta, acts, labels, lengths)
    x = nets.decode_acts(acts, np.float64)
    tl, tz, tg = torch_ref.step(cid, theta, x, labels, lengths)
    assert abs(r["loss"] - tl) <= 1e-12 * abs(tl)
    np.testing.assert_allclose(r["logits"], tz, rtol=0, atol=1e-11 * np.abs(tz).max())
    # every gradient entry, normwise per tensor; a tensor whose gradient is zero
    # by construction (the bias of a batch norm whose output reaches the loss
    # only through later batch norms: config 10's first three bottlenecks) holds
    # round-off on both sides, so scales have a floor of 1e-6 of the largest
    off = 0
    gscale = np.abs(tg).max()
    for name, shape, _, _ in S.param_layout(cid):
        n = int(np.prod(shape))
        g, t = r["grads"][off:off + n], tg[off:off + n]
        scale = max(np.abs(t).max(), 1e-6 * gscale)
        assert np.abs(g - t).max() <= 1e-9 * scale + 1e-300, name
        off += n
    np.testing.assert_allclose(r["params"], theta - 0.01 * r["grads"], rtol=1e-15, atol=1e-18)


@pytest.mark.parametrize("cid,n_probe", [(1, 12), (3, 10), (6, 12), (7, 12), (9, 12), (10, 12)])
def test_step_gradient_finite_differences(cid, n_probe):
    B = 2
    theta = S.init_params(cid).astype(np.float64)
    acts, labels, lengths = _inputs(cid, B, sub=3)
    r = oracle.server_step(cid, theta, acts, labels, lengths)
    rng = np.random.default_rng(5)
    idx = rng.choice(theta.size, size=n_probe, replace=False)
    # also probe the last entries (classifier bias)
    idx = np.concatenate([idx, [theta.size - 1]])
    h = 1e-6
    gmax = np.abs(r["grads"]).max()
    for i in idx:
        tp, tm = theta.copy(), theta.copy()
        tp[i] += h
        tm[i] -= h
        lp = oracle.server_step(cid, tp, acts, labels, lengths)["loss"]
        lm = oracle.server_step(cid, tm, acts, labels, lengths)["loss"]
        num = (lp - lm) / (2 * h)
        assert abs(num - r["grads"][i]) <= 1e-6 * gmax, (i, num, r["grads"][i])


@pytest.mark.parametrize("cid,C", [(1, 10), (2, 10), (3, 100), (4, 2), (6, 10), (7, 2), (8, 2), (9, 10), (10, 200)])
def test_zero_classifier_gives_ln_c(cid, C):
    theta = S.init_params(cid).astype(np.float64)
    lay = S.param_layout(cid)
    nlast = sum(int(np.prod(s)) for _, s, _, _ in lay[-2:])
    theta[-nlast:] = 0.0
    acts, labels, lengths = _inputs(cid, SMALL_B[cid])
    r = oracle.server_step(cid, theta, acts, labels, lengths)
    assert r["loss"] == pytest.approx(np.log(C), abs=1e-15)
    np.testing.assert_array_equal(r["logits"], 0.0)


def test_lr_zero_and_momentum_recursion():
    cid = 3
    theta = S.init_params(cid).astype(np.float64)
    acts, labels, _ = _inputs(cid, 2)
    r0 = oracle.server_step(cid, theta, acts, labels, lr=0.0, momentum=0.9)
    np.testing.assert_array_equal(r0["params"], theta)
    r1 = oracle.server_step(cid, theta, acts, labels, lr=0.01, momentum=0.9)
    np.testing.assert_array_equal(r1["momentum"], r1["grads"])        # v_1 = g_1
    r2 = oracle.server_step(cid, r1["params"], acts, labels, lr=0.01, momentum=0.9, mom_buf=r1["momentum"])
    np.testing.assert_allclose(r2["momentum"], 0.9 * r1["grads"] + r2["grads"], rtol=1e-15)
    np.testing.assert_allclose(r2["params"], r1["params"] - 0.01 * r2["momentum"], rtol=1e-15)


@pytest.mark.parametrize("cid,lens", [(4, (40, 77)), (7, (5, 33)), (8, (17, 200))])
def test_padded_tokens_never_matter(cid, lens):
    theta = S.init_params(cid)
    acts, labels, lengths = _inputs(cid, 2)
    lengths = np.array(lens, np.int32)
    r = oracle.server_step(cid, theta, acts, labels, lengths)
    x2 = nets.decode_acts(acts, np.float64).copy()
    x2[0, lens[0]:] = 123.0
    x2[1, lens[1]:] = -55.0
    r2 = oracle.server_step(cid, theta, x2, labels, lengths)
    np.testing.assert_allclose(r2["logits"], r["logits"], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(r2["grads"], r["grads"], rtol=1e-9, atol=1e-12 * np.abs(r["grads"]).max())


def test_momentum_term_moves_the_second_update():
    """The multi-step GPU check compares the update of each step by relative
    Frobenius error (bound 6e-2).  A mistake planted in the oracle -- the
    momentum buffer dropped at step 2 -- moves that update by far more than
    the bound, so the check can see the mu v term of v <- mu v + g."""
    cid = 3
    theta = S.init_params(cid).astype(np.float64)
    acts, labels, _ = _inputs(cid, 4)
    a2 = S.make_acts(cid, 1, batch=4, sub=77)[0]
    l2 = S.make_labels(cid, 1, batch=4, sub=77)[0]
    r1 = oracle.server_step(cid, theta, acts, labels, lr=0.01, momentum=0.9)
    good = oracle.server_step(cid, r1["params"], a2, l2, lr=0.01, momentum=0.9, mom_buf=r1["momentum"])
    bad = oracle.server_step(cid, r1["params"], a2, l2, lr=0.01, momentum=0.9,
                             mom_buf=np.zeros_like(r1["momentum"]))
    d_good = good["params"] - r1["params"]
    d_bad = bad["params"] - r1["params"]
    assert np.linalg.norm(d_bad - d_good) / np.linalg.norm(d_good) > 0.6


def test_trajectory_amplifies_a_one_percent_step_error():
    """Why the multi-step GPU checks start each step from the library's own
    state: in the fp64 oracle alone, a 1% (relative Frobenius) perturbation of
    the first update -- the size of one bf16 step's error -- grows within two
    more VGG steps into a gradient difference above the 6e-2 bound of the GPU
    checks.  Comparing the two trajectories would measure the dynamics."""
    cid, B, sub = 2, 16, 23
    th = S.init_params(cid).astype(np.float64)
    acts = S.make_acts(cid, 3, batch=B, sub=sub)
    labels = S.make_labels(cid, 3, batch=B, sub=sub)
    r1 = oracle.server_step(cid, th, acts[0], labels[0])
    d = r1["params"] - th
    noise = np.random.default_rng(0).standard_normal(d.shape) * np.abs(d)
    noise *= 0.01 * np.linalg.norm(d) / np.linalg.norm(noise)
    pa, pb = r1["params"], th + d + noise
    worst = 0.0
    for i in (1, 2):
        ra = oracle.server_step(cid, pa, acts[i], labels[i])
        rb = oracle.server_step(cid, pb, acts[i], labels[i])
        off = 0
        for _, shape, _, _ in S.param_layout(cid):
            n = int(np.prod(shape))
            ga, gb = ra["grads"][off:off + n], rb["grads"][off:off + n]
            worst = max(worst, np.linalg.norm(ga - gb) / np.linalg.norm(ga))
            off += n
        pa, pb = ra["params"], rb["params"]
    assert worst > 0.06


def test_device_step_matches_independent_autograd_and_sends_its_activations():
    """The device-side iteration (Alg. 1): loss, logits and every gradient
    against torch fp64 autograd of the same two networks, the activations it
    sends against torch's forward of the device network alone, and the SGD
    step on device and auxiliary parameters."""
    cid, B = 6, 3
    theta = S.init_params(cid)
    x = S.make_acts(cid, 1, batch=B, sub=4)[0]
    labels = S.make_labels(cid, 1, batch=B, sub=4)[0]
    r = oracle.device_step(cid, theta, x, labels, lr=0.01)
    tl, tz, tg = torch_ref.step(cid, theta, x, labels)
    acts = torch_ref.forward.last_acts.detach().numpy()
    assert r["acts"].shape == (B, 64, 16, 16)
    np.testing.assert_allclose(r["acts"], acts, rtol=0, atol=1e-12 * np.abs(acts).max())
    assert abs(r["loss"] - tl) <= 1e-12 * abs(tl)
    np.testing.assert_allclose(r["grads"], tg, rtol=0, atol=1e-10 * np.abs(tg).max())
    np.testing.assert_allclose(r["params"], theta - 0.01 * r["grads"], rtol=1e-15, atol=1e-18)
    # the device step's loss is the server step's definition applied to these networks
    assert r["loss"] == pytest.approx(oracle.server_step(cid, theta, x, labels)["loss"], abs=1e-15)
