"""Seeded generators for weights, activation batches, labels, lengths,
device-side vectors, staleness values and arrival tables.

Every draw comes from ``numpy.random.default_rng(SeedSequence(1000 + cid,
spawn_key=(stream,)))`` so that the oracle and the HIP path consume the very
same bytes.  bf16 activations are produced as raw 16-bit patterns (the fp32
draw rounded to nearest-even), so both sides read identical values.
"""
from __future__ import annotations

import numpy as np

from .configs import get_config, param_layout

STREAMS = {
    "weights": 0, "acts": 1, "labels": 2, "lengths": 3, "arrivals": 4,
    "staleness": 5, "local": 6, "rates": 7, "global": 8,
}


def rng_for(cid: int, stream: str, sub: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence(1000 + cid, spawn_key=(STREAMS[stream], sub))
    return np.random.default_rng(ss)


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns uint16 bit patterns.
    Inputs here are finite draws, so NaN handling is not needed."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def f32_from_bf16_bits(h: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def init_params(cid: int, sub: int = 0) -> np.ndarray:
    """Flat fp32 parameter vector in the library layout.  Weights are
    Kaiming-uniform U(+-sqrt(6/fan_in)); biases and norm shifts 0; norm scales 1."""
    rng = rng_for(cid, "weights", sub)
    parts = []
    for _, shape, kind, fan_in in param_layout(cid):
        n = int(np.prod(shape))
        if kind == "kaiming":
            bound = np.sqrt(6.0 / fan_in)
            parts.append(rng.uniform(-bound, bound, size=n).astype(np.float32))
        elif kind == "zeros":
            parts.append(np.zeros(n, np.float32))
        elif kind == "ones":
            parts.append(np.ones(n, np.float32))
        else:  # pragma: no cover
            raise ValueError(kind)
    return np.concatenate(parts)


def make_acts(cid: int, n_batches: int, batch: int | None = None, sub: int = 0) -> np.ndarray:
    """Activation batches as sent by the devices.

    CNN configs: ReLU(N(0,1)) in NCHW, [n, B, C, H, W].  Transformer configs
    (4, 7, 8): hidden states N(0,1), [n, B, L, d].  Device side (config 6): normalised
    32x32 RGB images N(0,1), [n, B, 3, 32, 32], standing in for CIFAR-10.
    fp32 configs return float32; bf16 configs return the uint16 bit patterns
    of the bf16-rounded values."""
    cfg = get_config(cid)
    B = cfg.batch if batch is None else batch
    rng = rng_for(cid, "acts", sub)
    x = rng.standard_normal(size=(n_batches, B) + tuple(cfg.in_shape), dtype=np.float32)
    if cfg.family not in ("bert", "vgg_device", "tfsmall", "mbv3"):  # mbv3: a linear bottleneck's output
        np.maximum(x, 0.0, out=x)
    if cfg.dtype == "f32":
        return x
    return bf16_bits_from_f32(x)


def make_labels(cid: int, n_batches: int, batch: int | None = None, sub: int = 0) -> np.ndarray:
    cfg = get_config(cid)
    B = cfg.batch if batch is None else batch
    rng = rng_for(cid, "labels", sub)
    if cfg.family in ("bert", "tfsmall"):
        return (rng.random(size=(n_batches, B)) < 0.5).astype(np.int32)
    return rng.integers(0, cfg.n_classes, size=(n_batches, B), dtype=np.int64).astype(np.int32)


def make_lengths(cid: int, n_batches: int, batch: int | None = None, sub: int = 0,
                 lo: int | None = None, hi: int | None = None) -> np.ndarray:
    """Valid-token counts per sequence, uniform on [lo, hi] (default [32, L])."""
    cfg = get_config(cid)
    B = cfg.batch if batch is None else batch
    lo = cfg.extra.get("min_len", 1) if lo is None else lo
    hi = cfg.in_shape[0] if hi is None else hi
    rng = rng_for(cid, "lengths", sub)
    return rng.integers(lo, hi + 1, size=(n_batches, B), dtype=np.int64).astype(np.int32)


def make_local_vectors(cid: int, n_vectors: int, n: int | None = None, sub: int = 0,
                       std: float = 0.02) -> np.ndarray:
    """Flat device-side model vectors ~ N(0, std^2), fp32, [n_vectors, n]."""
    cfg = get_config(cid)
    n = cfg.agg_n if n is None else n
    rng = rng_for(cid, "local", sub)
    return (rng.standard_normal(size=(n_vectors, n), dtype=np.float32) * np.float32(std))


def make_global_vector(cid: int, n: int | None = None, sub: int = 0, std: float = 0.02) -> np.ndarray:
    cfg = get_config(cid)
    n = cfg.agg_n if n is None else n
    rng = rng_for(cid, "global", sub)
    return rng.standard_normal(size=n, dtype=np.float32) * np.float32(std)


def make_staleness(cid: int, count: int, hi: int, sub: int = 0) -> np.ndarray:
    """Staleness values uniform on {0, ..., hi}."""
    rng = rng_for(cid, "staleness", sub)
    return rng.integers(0, hi + 1, size=count, dtype=np.int64).astype(np.int32)


def make_arrival_rates(cid: int, K: int | None = None, sub: int = 0) -> np.ndarray:
    """Per-device arrival rates lambda_k ~ LogNormal(0, 1)."""
    cfg = get_config(cid)
    K = cfg.n_devices if K is None else K
    return rng_for(cid, "rates", sub).lognormal(0.0, 1.0, size=K)


def make_arrival_counts(cid: int, rates: np.ndarray, steps: int, sub: int = 0) -> np.ndarray:
    """Arrival events per (server step, device): Poisson(lambda_k), int32 [steps, K]."""
    rng = rng_for(cid, "arrivals", sub)
    return rng.poisson(lam=rates[None, :], size=(steps, rates.shape[0])).astype(np.int32)


__all__ = [
    "rng_for", "bf16_bits_from_f32", "f32_from_bf16_bits", "init_params", "make_acts",
    "make_labels", "make_lengths", "make_local_vectors", "make_global_vector",
    "make_staleness", "make_arrival_rates", "make_arrival_counts",
]
