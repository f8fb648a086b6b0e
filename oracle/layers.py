"""Layer definitions of the server-side network M_s, forward and backward.

Test infrastructure (see package docstring).  Each layer is the textbook
definition written out directly; every backward formula is derived by hand
from the forward and checked against central finite differences in the
tests.  The paper's server networks are built from CONV, FC, pooling,
normalisation and transformer-encoder layers (Table 4, Sec. 5.1); the
per-layer conventions (padding, epsilon, GELU form, masking) are the
readings listed with the design notes of this repository.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

BN_EPS = 1e-5
LN_EPS = 1e-5


# ----------------------------------------------------------------------------- conv
class Conv2d:
    """Cross-correlation, NCHW input, weight [Cout, Cin, kh, kw], zero padding.

    Forward builds the explicit im2col matrix and multiplies; backward
    computes dW = dY^T cols, db = sum dY, and scatters dcols = dY W back
    (col2im)."""

    def __init__(self, w, b, stride=1, pad=1):
        self.w, self.b, self.s, self.p = w, b, stride, pad

    def fwd(self, x):
        B, C, H, W = x.shape
        Co, Ci, kh, kw = self.w.shape
        assert C == Ci
        s, p = self.s, self.p
        Ho = (H + 2 * p - kh) // s + 1
        Wo = (W + 2 * p - kw) // s + 1
        xp = np.zeros((B, C, H + 2 * p, W + 2 * p), x.dtype)
        xp[:, :, p:p + H, p:p + W] = x
        cols = np.empty((B, Ho, Wo, C, kh, kw), x.dtype)
        for i in range(kh):
            for j in range(kw):
                cols[..., i, j] = xp[:, :, i:i + s * Ho:s, j:j + s * Wo:s].transpose(0, 2, 3, 1)
        cols2 = cols.reshape(B * Ho * Wo, C * kh * kw)
        y = cols2 @ self.w.reshape(Co, -1).T
        if self.b is not None:
            y = y + self.b
        self.cache = (x.shape, cols2, Ho, Wo)
        return y.reshape(B, Ho, Wo, Co).transpose(0, 3, 1, 2)

    def bwd(self, dy, need_dx=True):
        (B, C, H, W), cols2, Ho, Wo = self.cache
        Co, Ci, kh, kw = self.w.shape
        s, p = self.s, self.p
        dy2 = dy.transpose(0, 2, 3, 1).reshape(B * Ho * Wo, Co)
        self.dw = (dy2.T @ cols2).reshape(self.w.shape)
        self.db = dy2.sum(0) if self.b is not None else None
        if not need_dx:
            return None
        dcols = (dy2 @ self.w.reshape(Co, -1)).reshape(B, Ho, Wo, C, kh, kw)
        dxp = np.zeros((B, C, H + 2 * p, W + 2 * p), dy.dtype)
        for i in range(kh):
            for j in range(kw):
                dxp[:, :, i:i + s * Ho:s, j:j + s * Wo:s] += dcols[..., i, j].transpose(0, 3, 1, 2)
        return dxp[:, :, p:p + H, p:p + W]


class DepthwiseConv2d:
    """One k x k filter per channel (groups = channels), NCHW input, weight
    [C, 1, k, k], zero padding k // 2, no bias.  y[b,c,o] = sum over the
    window of x[b,c,i] w[c,tap]; backward by the same sums read the other way."""

    def __init__(self, w, stride=1):
        self.w, self.s = w, stride

    def fwd(self, x):
        B, C, H, W = x.shape
        k = self.w.shape[-1]
        p, s = k // 2, self.s
        Ho, Wo = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
        xp = np.zeros((B, C, H + 2 * p, W + 2 * p), x.dtype)
        xp[:, :, p:p + H, p:p + W] = x
        y = np.zeros((B, C, Ho, Wo), x.dtype)
        for i in range(k):
            for j in range(k):
                y += xp[:, :, i:i + s * Ho:s, j:j + s * Wo:s] * self.w[None, :, 0, i, j, None, None]
        self.cache = (xp, x.shape, Ho, Wo)
        return y

    def bwd(self, dy, need_dx=True):
        xp, (B, C, H, W), Ho, Wo = self.cache
        k = self.w.shape[-1]
        p, s = k // 2, self.s
        self.dw = np.zeros_like(self.w)
        dxp = np.zeros_like(xp)
        for i in range(k):
            for j in range(k):
                win = xp[:, :, i:i + s * Ho:s, j:j + s * Wo:s]
                self.dw[:, 0, i, j] = (dy * win).sum(axis=(0, 2, 3))
                dxp[:, :, i:i + s * Ho:s, j:j + s * Wo:s] += dy * self.w[None, :, 0, i, j, None, None]
        return dxp[:, :, p:p + H, p:p + W] if need_dx else None


# ----------------------------------------------------------------------------- elementwise
class ReLU:
    def fwd(self, x):
        self.mask = x > 0
        return np.where(self.mask, x, 0.0).astype(x.dtype)

    def bwd(self, dy):
        return np.where(self.mask, dy, 0.0).astype(dy.dtype)


class GELU:
    """Exact GELU: 0.5 x (1 + erf(x / sqrt 2)); derivative Phi(x) + x phi(x)."""

    def fwd(self, x):
        self.x = x
        return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))

    def bwd(self, dy):
        x = self.x
        cdf = 0.5 * (1.0 + erf(x / np.sqrt(2.0)))
        pdf = np.exp(-0.5 * x * x) / np.sqrt(2.0 * np.pi)
        return dy * (cdf + x * pdf)


class HardSwish:
    """x ReLU6(x + 3) / 6; derivative 0 below -3, 1 above 3, (2x + 3) / 6 between."""

    def fwd(self, x):
        self.x = x
        return x * np.clip(x + 3.0, 0.0, 6.0) / 6.0

    def bwd(self, dy):
        x = self.x
        return dy * np.where(x < -3.0, 0.0, np.where(x > 3.0, 1.0, (2.0 * x + 3.0) / 6.0))


class HardSigmoid:
    """ReLU6(x + 3) / 6; derivative 1/6 strictly between -3 and 3, else 0."""

    def fwd(self, x):
        self.x = x
        return np.clip(x + 3.0, 0.0, 6.0) / 6.0

    def bwd(self, dy):
        x = self.x
        return dy * np.where((x > -3.0) & (x < 3.0), 1.0 / 6.0, 0.0)


class Tanh:
    def fwd(self, x):
        self.y = np.tanh(x)
        return self.y

    def bwd(self, dy):
        return dy * (1.0 - self.y * self.y)


# ----------------------------------------------------------------------------- pooling
class MaxPool2:
    """2x2 window, stride 2.  Backward routes each gradient to the first
    maximum of its window in row-major window order (np.argmax order)."""

    def fwd(self, x):
        B, C, H, W = x.shape
        win = x.reshape(B, C, H // 2, 2, W // 2, 2).transpose(0, 1, 2, 4, 3, 5).reshape(B, C, H // 2, W // 2, 4)
        self.idx = win.argmax(-1)
        self.shape = x.shape
        return np.take_along_axis(win, self.idx[..., None], -1)[..., 0]

    def bwd(self, dy):
        B, C, H, W = self.shape
        dwin = np.zeros((B, C, H // 2, W // 2, 4), dy.dtype)
        np.put_along_axis(dwin, self.idx[..., None], dy[..., None], -1)
        return dwin.reshape(B, C, H // 2, W // 2, 2, 2).transpose(0, 1, 2, 4, 3, 5).reshape(B, C, H, W)


class GlobalAvgPool:
    def fwd(self, x):
        self.shape = x.shape
        return x.mean(axis=(2, 3))

    def bwd(self, dy):
        B, C, H, W = self.shape
        return np.broadcast_to(dy[:, :, None, None] / (H * W), self.shape).copy()


# ----------------------------------------------------------------------------- linear
class Linear:
    """y = x W^T + b over the last axis; W is [out, in]."""

    def __init__(self, w, b):
        self.w, self.b = w, b

    def fwd(self, x):
        self.x = x
        return x @ self.w.T + self.b

    def bwd(self, dy, need_dx=True):
        x2 = self.x.reshape(-1, self.x.shape[-1])
        dy2 = dy.reshape(-1, dy.shape[-1])
        self.dw = dy2.T @ x2
        self.db = dy2.sum(0)
        return dy @ self.w if need_dx else None


# ----------------------------------------------------------------------------- loss
def cross_entropy(z, y):
    """Mean softmax cross-entropy over the batch (the server loss f_s, Eq. 5,
    averaged over one activation batch) and its gradient (softmax - onehot)/B."""
    B = z.shape[0]
    m = z.max(axis=1, keepdims=True)
    lse = m + np.log(np.exp(z - m).sum(axis=1, keepdims=True))
    loss = float(np.mean(lse[:, 0] - z[np.arange(B), y]))
    p = np.exp(z - lse)
    dz = p.copy()
    dz[np.arange(B), y] -= 1.0
    return loss, dz / B


# ----------------------------------------------------------------------------- norms
class BatchNorm2d:
    """Training-mode batch norm: statistics over (N, H, W), biased variance."""

    def __init__(self, g, b, eps=BN_EPS):
        self.g, self.b, self.eps = g, b, eps

    def fwd(self, x):
        mu = x.mean(axis=(0, 2, 3), keepdims=True)
        var = ((x - mu) ** 2).mean(axis=(0, 2, 3), keepdims=True)
        self.rstd = 1.0 / np.sqrt(var + self.eps)
        self.xhat = (x - mu) * self.rstd
        return self.g[None, :, None, None] * self.xhat + self.b[None, :, None, None]

    def bwd(self, dy):
        N = dy.shape[0] * dy.shape[2] * dy.shape[3]
        self.dg = (dy * self.xhat).sum(axis=(0, 2, 3))
        self.db = dy.sum(axis=(0, 2, 3))
        g = self.g[None, :, None, None]
        return g * self.rstd * (dy - self.db[None, :, None, None] / N
                                - self.xhat * self.dg[None, :, None, None] / N)


class LayerNorm:
    """Normalisation over the last axis, biased variance, affine."""

    def __init__(self, g, b, eps=LN_EPS):
        self.g, self.b, self.eps = g, b, eps

    def fwd(self, x):
        mu = x.mean(axis=-1, keepdims=True)
        var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
        self.rstd = 1.0 / np.sqrt(var + self.eps)
        self.xhat = (x - mu) * self.rstd
        return self.xhat * self.g + self.b

    def bwd(self, dy):
        d = dy.shape[-1]
        xh = self.xhat
        self.dg = (dy * xh).reshape(-1, d).sum(0)
        self.db = dy.reshape(-1, d).sum(0)
        dxh = dy * self.g
        return self.rstd * (dxh - dxh.mean(axis=-1, keepdims=True)
                            - xh * (dxh * xh).mean(axis=-1, keepdims=True))


# ----------------------------------------------------------------------------- attention
class MultiHeadAttention:
    """Self-attention with a fused [3d, d] input projection (query, key and
    value rows in that order), `heads` heads of width d/heads, scores scaled by
    1/sqrt(d/heads), keys at positions >= length masked to -inf, softmax over
    keys, output projection [d, d]."""

    def __init__(self, wqkv, bqkv, wo, bo, heads):
        self.qkv = Linear(wqkv, bqkv)
        self.out = Linear(wo, bo)
        self.h = heads

    def fwd(self, x, lengths):
        B, L, d = x.shape
        H, dh = self.h, d // self.h
        qkv = self.qkv.fwd(x)
        q = qkv[..., 0 * d:1 * d].reshape(B, L, H, dh).transpose(0, 2, 1, 3)
        k = qkv[..., 1 * d:2 * d].reshape(B, L, H, dh).transpose(0, 2, 1, 3)
        v = qkv[..., 2 * d:3 * d].reshape(B, L, H, dh).transpose(0, 2, 1, 3)
        scale = 1.0 / np.sqrt(dh)
        s = (q @ k.transpose(0, 1, 3, 2)) * scale
        keymask = np.arange(L)[None, :] >= np.asarray(lengths)[:, None]  # [B, L]
        s = np.where(keymask[:, None, None, :], -np.inf, s)
        m = s.max(axis=-1, keepdims=True)
        e = np.exp(s - m)
        p = e / e.sum(axis=-1, keepdims=True)
        o = p @ v
        self.cache = (q, k, v, p, scale, B, L, d, H, dh)
        return self.out.fwd(o.transpose(0, 2, 1, 3).reshape(B, L, d))

    def bwd(self, dy, need_dx=True):
        q, k, v, p, scale, B, L, d, H, dh = self.cache
        do = self.out.bwd(dy).reshape(B, L, H, dh).transpose(0, 2, 1, 3)
        dv = p.transpose(0, 1, 3, 2) @ do
        dp = do @ v.transpose(0, 1, 3, 2)
        ds = p * (dp - (dp * p).sum(axis=-1, keepdims=True))
        dq = (ds @ k) * scale
        dk = (ds.transpose(0, 1, 3, 2) @ q) * scale
        dqkv = np.concatenate([t.transpose(0, 2, 1, 3).reshape(B, L, d) for t in (dq, dk, dv)], axis=-1)
        return self.qkv.bwd(dqkv, need_dx)
