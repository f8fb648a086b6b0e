"""Pins for the oracle's layer definitions (CPU only).

Backward formulas are checked against central finite differences of the
forward in fp64; forwards are checked against brute-force loops, closed
forms and textbook identities."""
import numpy as np
import pytest
from scipy.signal import correlate

from oracle import layers as L

RNG = np.random.default_rng(12345)
FD_H = 1e-6
FD_TOL = 1e-6


def fd_check(fwd, x, dy, analytic, n_probe=25, rng=RNG):
    """Central differences of <fwd(x), dy> w.r.t. sampled entries of x."""
    flat = x.reshape(-1)
    idx = rng.choice(flat.size, size=min(n_probe, flat.size), replace=False)
    an = analytic.reshape(-1)
    scale = np.abs(an).max() + 1e-30
    for i in idx:
        old = flat[i]
        flat[i] = old + FD_H
        fp = np.sum(fwd() * dy)
        flat[i] = old - FD_H
        fm = np.sum(fwd() * dy)
        flat[i] = old
        num = (fp - fm) / (2 * FD_H)
        assert abs(num - an[i]) <= FD_TOL * scale + 1e-9 * abs(num), (i, num, an[i])


@pytest.mark.parametrize("stride,pad,k", [(1, 1, 3), (2, 1, 3), (2, 0, 1), (1, 0, 1)])
def test_conv_forward_brute_force(stride, pad, k):
    x = RNG.standard_normal((2, 3, 7, 6))
    w = RNG.standard_normal((4, 3, k, k))
    b = RNG.standard_normal(4)
    y = L.Conv2d(w, b, stride, pad).fwd(x)
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    for n in range(2):
        for co in range(4):
            full = sum(correlate(xp[n, ci], w[co, ci], mode="valid") for ci in range(3))
            np.testing.assert_allclose(y[n, co], full[::stride, ::stride] + b[co], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("stride,pad,k", [(1, 1, 3), (2, 1, 3), (2, 0, 1)])
def test_conv_backward_fd(stride, pad, k):
    x = RNG.standard_normal((2, 3, 6, 6))
    w = RNG.standard_normal((4, 3, k, k))
    b = RNG.standard_normal(4)
    conv = L.Conv2d(w, b, stride, pad)
    y = conv.fwd(x)
    dy = RNG.standard_normal(y.shape)
    dx = conv.bwd(dy)
    dw, db = conv.dw.copy(), conv.db.copy()
    fd_check(lambda: L.Conv2d(w, b, stride, pad).fwd(x), x, dy, dx)
    fd_check(lambda: L.Conv2d(w, b, stride, pad).fwd(x), w, dy, dw)
    fd_check(lambda: L.Conv2d(w, b, stride, pad).fwd(x), b, dy, db)


def test_conv1x1_is_matmul():
    x = RNG.standard_normal((3, 5, 4, 4))
    w = RNG.standard_normal((7, 5, 1, 1))
    y = L.Conv2d(w, None, 1, 0).fwd(x)
    ref = np.einsum("oc,nchw->nohw", w[:, :, 0, 0], x)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_relu_maxpool_gap_fd():
    x = RNG.standard_normal((2, 3, 4, 6))
    for mk in (L.MaxPool2, L.GlobalAvgPool, L.ReLU):
        m = mk()
        y = m.fwd(x)
        dy = RNG.standard_normal(y.shape)
        fd_check(lambda: mk().fwd(x), x, dy, m.bwd(dy))


def test_maxpool_first_max_on_ties():
    x = np.zeros((1, 1, 2, 2))
    x[0, 0, 0, 1] = 1.0
    x[0, 0, 1, 0] = 1.0          # tie between window positions 1 and 2
    m = L.MaxPool2()
    m.fwd(x)
    dx = m.bwd(np.ones((1, 1, 1, 1)))
    assert dx[0, 0, 0, 1] == 1.0 and dx.sum() == 1.0


def test_linear_fd():
    x = RNG.standard_normal((5, 7))
    w = RNG.standard_normal((3, 7))
    b = RNG.standard_normal(3)
    lin = L.Linear(w, b)
    y = lin.fwd(x)
    dy = RNG.standard_normal(y.shape)
    dx = lin.bwd(dy)
    fd_check(lambda: L.Linear(w, b).fwd(x), x, dy, dx)
    fd_check(lambda: L.Linear(w, b).fwd(x), w, dy, lin.dw)
    fd_check(lambda: L.Linear(w, b).fwd(x), b, dy, lin.db)


def test_cross_entropy_closed_forms():
    z = RNG.standard_normal((6, 10))
    y = RNG.integers(0, 10, 6)
    loss, dz = L.cross_entropy(z, y)
    np.testing.assert_allclose(dz.sum(1), 0.0, atol=1e-15)
    # direct definition -log softmax
    p = np.exp(z) / np.exp(z).sum(1, keepdims=True)
    assert abs(loss - np.mean(-np.log(p[np.arange(6), y]))) < 1e-13
    # equal logits: loss is exactly ln C
    for C in (2, 10, 100):
        l2, _ = L.cross_entropy(np.zeros((4, C)), np.zeros(4, int))
        assert abs(l2 - np.log(C)) < 1e-14
    # fd
    h = 1e-6
    for (i, j) in [(0, 0), (3, 7), (5, 9)]:
        zp, zm = z.copy(), z.copy()
        zp[i, j] += h
        zm[i, j] -= h
        num = (L.cross_entropy(zp, y)[0] - L.cross_entropy(zm, y)[0]) / (2 * h)
        assert abs(num - dz[i, j]) < 1e-8


def test_batchnorm_fd_and_identities():
    x = RNG.standard_normal((3, 4, 3, 2)) * 2 + 1
    g = RNG.standard_normal(4)
    b = RNG.standard_normal(4)
    bn = L.BatchNorm2d(g, b)
    y = bn.fwd(x)
    # normalised output: per-channel mean b, biased variance g^2 var/(var+eps)
    np.testing.assert_allclose(y.mean((0, 2, 3)), b, atol=1e-12)
    var = x.var(axis=(0, 2, 3))
    np.testing.assert_allclose(y.var(axis=(0, 2, 3)), g ** 2 * var / (var + 1e-5), rtol=1e-10)
    dy = RNG.standard_normal(y.shape)
    dx = bn.bwd(dy)
    np.testing.assert_allclose(dx.sum((0, 2, 3)), 0.0, atol=1e-12)
    fd_check(lambda: L.BatchNorm2d(g, b).fwd(x), x, dy, dx)
    fd_check(lambda: L.BatchNorm2d(g, b).fwd(x), g, dy, bn.dg)
    fd_check(lambda: L.BatchNorm2d(g, b).fwd(x), b, dy, bn.db)


def test_layernorm_fd_and_identities():
    x = RNG.standard_normal((2, 3, 8)) * 3 - 1
    g = RNG.standard_normal(8)
    b = RNG.standard_normal(8)
    ln = L.LayerNorm(g, b)
    y = ln.fwd(x)
    dy = RNG.standard_normal(y.shape)
    dx = ln.bwd(dy)
    np.testing.assert_allclose(dx.sum(-1), 0.0, atol=1e-12)
    fd_check(lambda: L.LayerNorm(g, b).fwd(x), x, dy, dx)
    fd_check(lambda: L.LayerNorm(g, b).fwd(x), g, dy, ln.dg)


def test_gelu_tanh_fd_and_values():
    x = RNG.standard_normal((4, 5)) * 2
    for mk in (L.GELU, L.Tanh):
        m = mk()
        y = m.fwd(x)
        dy = RNG.standard_normal(y.shape)
        fd_check(lambda: mk().fwd(x), x, dy, m.bwd(dy))
    # GELU(x) = x * Phi(x): Phi(0)=1/2, Phi(1)=0.8413447460685429
    g = L.GELU().fwd(np.array([0.0, 1.0, -1.0]))
    np.testing.assert_allclose(g, [0.0, 0.8413447460685429, -0.15865525393145707], rtol=1e-14)


def test_attention_fd_and_masking():
    B, Lq, d, H = 2, 5, 8, 2
    x = RNG.standard_normal((B, Lq, d))
    wqkv = RNG.standard_normal((3 * d, d)) * 0.3
    bqkv = RNG.standard_normal(3 * d) * 0.1
    wo = RNG.standard_normal((d, d)) * 0.3
    bo = RNG.standard_normal(d) * 0.1
    lengths = np.array([5, 3])

    def f():
        return L.MultiHeadAttention(wqkv, bqkv, wo, bo, H).fwd(x, lengths)

    att = L.MultiHeadAttention(wqkv, bqkv, wo, bo, H)
    y = att.fwd(x, lengths)
    dy = RNG.standard_normal(y.shape)
    dx = att.bwd(dy)
    fd_check(f, x, dy, dx)
    fd_check(f, wqkv, dy, att.qkv.dw)
    fd_check(f, bqkv, dy, att.qkv.db)
    fd_check(f, wo, dy, att.out.dw)
    # keys beyond the length do not influence any output of that sequence
    x2 = x.copy()
    x2[1, 3:] += 10.0
    y2 = L.MultiHeadAttention(wqkv, bqkv, wo, bo, H).fwd(x2, lengths)
    np.testing.assert_allclose(y2[1, :3], y[1, :3], rtol=1e-12, atol=1e-12)
    # single head, single valid key: output is that key's value through Wo
    one = L.MultiHeadAttention(wqkv, bqkv, wo, bo, 1).fwd(x[:1], np.array([1]))
    v0 = x[0, 0] @ wqkv[2 * d:].T + bqkv[2 * d:]
    np.testing.assert_allclose(one[0, 2], v0 @ wo.T + bo, rtol=1e-12)
