"""GPU tests of the MFMA GEMM and implicit-GEMM convolution passes in
isolation, through the kernel-level C entry points, against plain fp64
references (a matrix product; the oracle's convolution forward, input
gradient and weight gradient).  Shapes cover several tiles, ragged edges in
every dimension, both operand layouts, compensated products and split-K."""
import numpy as np
import pytest

import fo_synth as S
from oracle import layers as OL
from tests.gpu_util import announce, normwise, to_dev, torch_cuda

pytestmark = pytest.mark.gpu
A = pytest.importorskip("paper_2504_13850_amd.api")


def _bf16(rng, shape, scale=1.0):
    x = (rng.standard_normal(shape) * scale).astype(np.float32)
    h = S.bf16_bits_from_f32(x)
    return h, S.f32_from_bf16_bits(h).astype(np.float64)


def _split(rng, shape):
    """A value with exact (hi, lo) bf16 parts: x = hi + lo."""
    hi, hv = _bf16(rng, shape)
    lo, lv = _bf16(rng, shape, 2.0 ** -9)
    return hi, lo, hv + lv


def _dev16(h):
    return to_dev(h.view(np.int16))


@pytest.mark.parametrize("M,N,K,la,lb", [
    (256, 256, 256, 0, 0), (200, 130, 96, 0, 0), (129, 257, 70, 0, 1), (64, 10, 512, 0, 1),
    (512, 768, 3072, 0, 0), (300, 200, 1000, 1, 1), (10, 512, 64, 1, 1), (3, 5, 7, 0, 0), (1, 1, 1, 1, 0),
    # k-major, rows in whole chunks of 8 (the weight-gradient kernel with copies
    # into LDS): ragged row tiles and K tails of every depth
    (264, 136, 1000, 1, 1), (776, 392, 70, 1, 1), (8, 8, 5, 1, 1), (128, 1152, 4097, 1, 1),
    # row-major A times k-major B with every dimension in chunks of 8 (the
    # input-gradient kernel with copies into LDS)
    (264, 136, 1000, 0, 1), (776, 392, 72, 0, 1), (8, 8, 8, 0, 1), (2496, 768, 2304, 0, 1)])
def test_gemm_plain(M, N, K, la, lb):
    torch = torch_cuda()
    announce(f"gemm {M}x{N}x{K} layouts {la}{lb}")
    rng = np.random.default_rng(M * 7 + N * 3 + K)
    a, av = _bf16(rng, (M, K))
    b, bv = _bf16(rng, (N, K))
    Ad = _dev16(a if la == 0 else np.ascontiguousarray(a.T))
    Bd = _dev16(b if lb == 0 else np.ascontiguousarray(b.T))
    C = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    A.fo_gemm_bf16(M, N, K, la, Ad, None, K if la == 0 else M, lb, Bd, None, K if lb == 0 else N, C, N)
    ref = av @ bv.T
    assert normwise(C.cpu().numpy(), ref) <= 1e-5


@pytest.mark.parametrize("M,N,K,splits,la", [(256, 384, 1024, 4, 1), (100, 70, 333, 3, 1), (768, 768, 4096, 8, 1),
                                             (2496, 768, 3072, 2, 0), (264, 136, 1000, 3, 0)])
def test_gemm_split_k(M, N, K, splits, la):
    torch = torch_cuda()
    announce(f"gemm split-K {M}x{N}x{K} s={splits} A layout {la}")
    rng = np.random.default_rng(K)
    a, av = _bf16(rng, (K, M))      # k-major B (and A when la = 1), as in weight and input gradients
    b, bv = _bf16(rng, (K, N))
    Ad = _dev16(a) if la == 1 else _dev16(np.ascontiguousarray(a.T))
    C = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    ws = torch.empty(splits * M * N, dtype=torch.float32, device="cuda")
    A.fo_gemm_bf16(M, N, K, la, Ad, None, M if la == 1 else K, 1, _dev16(b), None, N, C, N, splits, ws)
    assert normwise(C.cpu().numpy(), av.T @ bv) <= 1e-5


@pytest.mark.parametrize("M,N,K,with_alo", [(256, 256, 768, True), (130, 300, 96, True), (64, 512, 512, False)])
def test_gemm_compensated(M, N, K, with_alo):
    """hi.hi + hi.lo + lo.hi reproduces the product of the unrounded values
    to about 16 significant bits (the omitted lo.lo term is ~2^-18)."""
    torch = torch_cuda()
    announce(f"gemm compensated {M}x{N}x{K}")
    rng = np.random.default_rng(N)
    if with_alo:
        ah, al, av = _split(rng, (M, K))
    else:
        ah, av = _bf16(rng, (M, K))
        al = None
    bh, bl, bv = _split(rng, (N, K))
    C = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    A.fo_gemm_bf16(M, N, K, 0, _dev16(ah), None if al is None else _dev16(al), K, 0, _dev16(bh), _dev16(bl), K, C, N)
    assert normwise(C.cpu().numpy(), av @ bv.T) <= 2e-5


@pytest.mark.parametrize("M,N,K,splits,with_alo", [(300, 200, 1000, 3, True), (129, 640, 2048, 4, True),
                                                    (256, 130, 512, 2, False)])
def test_gemm_compensated_split_k(M, N, K, splits, with_alo):
    """The single-pass compensated product with K slices (fp32 partials, reduction pass)."""
    torch = torch_cuda()
    announce(f"gemm compensated split-K {M}x{N}x{K} s={splits}")
    rng = np.random.default_rng(M + K)
    if with_alo:
        ah, al, av = _split(rng, (M, K))
    else:
        ah, av = _bf16(rng, (M, K))
        al = None
    bh, bl, bv = _split(rng, (N, K))
    C = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    ws = torch.empty(splits * M * N, dtype=torch.float32, device="cuda")
    A.fo_gemm_bf16(M, N, K, 0, _dev16(ah), None if al is None else _dev16(al), K, 0, _dev16(bh), _dev16(bl), K, C, N,
                   splits, ws)
    assert normwise(C.cpu().numpy(), av @ bv.T) <= 2e-5


CONVS = [  # (Bn, H, Ci, Co, k, stride, pad)
    (2, 16, 64, 128, 3, 1, 1), (3, 8, 128, 256, 3, 1, 1), (2, 4, 256, 512, 3, 1, 1), (2, 2, 512, 512, 3, 1, 1),
    (32, 2, 512, 512, 3, 1, 1), (2, 16, 64, 128, 3, 2, 1), (4, 4, 256, 512, 3, 2, 1), (2, 16, 64, 128, 1, 2, 0),
    (3, 4, 256, 512, 1, 2, 0), (1, 2, 512, 512, 3, 1, 1)]


def _conv_case(case, seed):
    Bn, H, Ci, Co, k, st, pad = case
    rng = np.random.default_rng(seed)
    x, xv = _bf16(rng, (Bn, H, H, Ci))
    w, wv = _bf16(rng, (Co, k, k, Ci), 0.05)
    Ho = (H + 2 * pad - k) // st + 1
    dy, dyv = _bf16(rng, (Bn, Ho, Ho, Co))
    conv = OL.Conv2d(wv.transpose(0, 3, 1, 2), None, st, pad)
    y = conv.fwd(xv.transpose(0, 3, 1, 2))
    dx = conv.bwd(dyv.transpose(0, 3, 1, 2))
    return (x, w, dy), (y.transpose(0, 2, 3, 1), dx.transpose(0, 2, 3, 1), conv.dw.transpose(0, 2, 3, 1)), Ho


@pytest.mark.parametrize("case", CONVS)
def test_conv_passes(case):
    torch = torch_cuda()
    Bn, H, Ci, Co, k, st, pad = case
    announce(f"conv {case}")
    (x, w, dy), (y_ref, dx_ref, dw_ref), Ho = _conv_case(case, sum(case))
    xd, wd, dyd = _dev16(x), _dev16(w), _dev16(dy)
    for splits in (1, 4):  # split-K forward and input gradient: fp32 partials, epilogue in the reduction
        ws = torch.empty(splits * Bn * H * H * max(Ci, Co), dtype=torch.float32, device="cuda")
        y = torch.zeros((Bn, Ho, Ho, Co), dtype=torch.float32, device="cuda")
        A.fo_conv2d_bf16(0, Bn, H, H, Ci, Co, k, st, pad, xd, None, None, wd, None, y, splits, ws)
        assert normwise(y.cpu().numpy(), y_ref) <= 1e-5, splits
        dx = torch.zeros((Bn, H, H, Ci), dtype=torch.float32, device="cuda")
        A.fo_conv2d_bf16(1, Bn, H, H, Ci, Co, k, st, pad, dyd, None, None, wd, None, dx, splits, ws)
        assert normwise(dx.cpu().numpy(), dx_ref) <= 1e-5, splits
    for splits in (1, 4):
        dw = torch.zeros((Co, k, k, Ci), dtype=torch.float32, device="cuda")
        rows, cols = Co, k * k * Ci
        ws = torch.empty(splits * rows * cols, dtype=torch.float32, device="cuda")
        if Bn * Ho * Ho < splits * 32:
            continue
        A.fo_conv2d_bf16(2, Bn, H, H, Ci, Co, k, st, pad, dyd, None, xd, None, None, dw, splits, ws)
        assert normwise(dw.cpu().numpy(), dw_ref) <= 1e-5, splits
