"""Helpers shared by the GPU parity tests (marshalling and error metrics)."""
import numpy as np


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        import pytest
        pytest.skip("no GPU")
    return torch


def to_dev(x):
    torch = torch_cuda()
    t = torch.from_numpy(np.ascontiguousarray(x))
    return t.cuda()


def normwise(got, ref):
    """max_i |g_i - r_i| / max_i |r_i| (0 when both are zero)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.abs(ref).max() if ref.size else 0.0
    err = np.abs(got - ref).max() if ref.size else 0.0
    return 0.0 if scale == 0.0 and err == 0.0 else err / max(scale, 1e-300)


def per_tensor_errors(cid, got_flat, ref_flat, floor=0.0):
    """normwise error per parameter tensor; with floor > 0 a tensor's scale is
    at least floor times the largest gradient entry of the whole model (for
    gradients that are zero by construction and hold round-off only)."""
    import fo_synth as S
    out, off = {}, 0
    gscale = float(np.abs(np.asarray(ref_flat, np.float64)).max()) if floor > 0 else 0.0
    for name, shape, _, _ in S.param_layout(cid):
        n = int(np.prod(shape))
        got, ref = np.asarray(got_flat[off:off + n], np.float64), np.asarray(ref_flat[off:off + n], np.float64)
        scale = max(np.abs(ref).max(), floor * gscale)
        out[name] = np.abs(got - ref).max() / max(scale, 1e-300)
        off += n
    return out


def announce(msg):
    """Names the case before a GPU step, so a hard failure still says which."""
    print(f"[gpu-case] {msg}", flush=True)
