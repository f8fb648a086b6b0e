"""GPU test of fo_gemm_bf16_noalloc, the variant of fo_gemm_bf16 for callers
that cannot allocate: its split-K partials live in a fixed array of the
library instead of a caller workspace.  Through the C ABI, two calls in a
row (the second smaller, on different data, so partials left by the first
would show) must give the existing entry point's result bit for bit, and
both must match a plain fp64 product within 1e-5 (normwise); a product
whose partials exceed the array is refused before anything launches."""
import numpy as np
import pytest

import fo_synth as S
from tests.gpu_util import announce, normwise, to_dev, torch_cuda

pytestmark = pytest.mark.gpu
A = pytest.importorskip("paper_2504_13850_amd.api")

MAX_FLOATS = 4 << 20


def _bf16(rng, shape):
    h = S.bf16_bits_from_f32(rng.standard_normal(shape).astype(np.float32))
    return h, S.f32_from_bf16_bits(h).astype(np.float64)


def _case(torch, M, N, K, splits, la, lb, seed):
    rng = np.random.default_rng(seed)
    a, av = _bf16(rng, (M, K))
    b, bv = _bf16(rng, (N, K))
    Ad = to_dev((a if la == 0 else np.ascontiguousarray(a.T)).view(np.int16))
    Bd = to_dev((b if lb == 0 else np.ascontiguousarray(b.T)).view(np.int16))
    lda = K if la == 0 else M
    ldb = K if lb == 0 else N
    C0 = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    C1 = torch.full((M, N), 7.0, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(splits * M * N, 1), dtype=torch.float32, device="cuda")
    A.fo_gemm_bf16(M, N, K, la, Ad, None, lda, lb, Bd, None, ldb, C0, N, splits, ws)
    A.fo_gemm_bf16_noalloc(M, N, K, la, Ad, None, lda, lb, Bd, None, ldb, C1, N, splits)
    got0, got1 = C0.cpu().numpy(), C1.cpu().numpy()
    assert got1.tobytes() == got0.tobytes(), (M, N, K, splits)
    assert normwise(got1, av @ bv.T) <= 1e-5


def test_noalloc_matches_workspace_entry_point():
    torch = torch_cuda()
    announce("gemm noalloc: 768x768x4096 s=4 then 100x70x333 s=3")
    _case(torch, 768, 768, 4096, 4, 1, 1, 1)   # weight-gradient layout, 2.4M floats of partials
    _case(torch, 100, 70, 333, 3, 1, 1, 2)     # smaller, ragged, after the first
    _case(torch, 200, 130, 96, 1, 0, 0, 3)     # unsplit: no scratch at all


def test_noalloc_refuses_more_than_its_scratch():
    torch = torch_cuda()
    announce("gemm noalloc: oversized request refused")
    M, N, splits = 1024, 1024, 5  # 5.2M floats of partials > 4M
    assert splits * M * N > MAX_FLOATS
    d = torch.zeros(16, dtype=torch.int16, device="cuda")  # never read: the call is refused first
    C = torch.zeros(16, dtype=torch.float32, device="cuda")
    with pytest.raises(A.FoError) as e:
        A.fo_gemm_bf16_noalloc(M, N, 64, 0, d, None, 64, 0, d, None, 64, C, N, splits)
    assert e.value.status == A.FO_EINVAL and "16 MiB" in str(e.value)
