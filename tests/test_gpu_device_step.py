"""GPU parity of the device-side training iteration (Alg. 1, config 6: the
device network of the VGG-16 split and its auxiliary network) against the
fp64 oracle, through the C ABI, and of the hand-over of its activations to
the server (Alg. 2 put(), Alg. 3 get(), Alg. 4 training step).

Graded as the server's bf16 path: the local loss and the auxiliary logits
within 2e-2 (normwise for logits).  The activations the device sends are the
bf16 roundings of a compensated (about 16-bit) forward, so each must lie
within 2^-8 of the oracle's value relative to the largest activation of its
batch (normwise 4e-3).  Gradients and the update: relative Frobenius error per
tensor <= 6e-2 (bf16 backward)."""
import numpy as np
import pytest

import fo_synth as S
import oracle
from tests.gpu_util import announce, normwise, to_dev, torch_cuda

pytestmark = pytest.mark.gpu
A = pytest.importorskip("paper_2504_13850_amd.api")

CID = 6
TOL = 2e-2
ACT_TOL = 2.0 ** -8
GRAD_TOL = 6e-2


def _frob(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)


def _check(out, theta_before, r, B):
    acts = S.f32_from_bf16_bits(out["acts"].reshape(B, 64, 16, 16)).astype(np.float64)
    assert abs(out["loss"] - r["loss"]) <= TOL * abs(r["loss"]), (out["loss"], r["loss"])
    assert normwise(out["logits"], r["logits"]) <= TOL
    assert normwise(acts, r["acts"]) <= ACT_TOL
    off = 0
    for name, shape, _, _ in S.param_layout(CID):
        n = int(np.prod(shape))
        e = _frob(out["grads"][off:off + n], r["grads"][off:off + n])
        assert e <= GRAD_TOL, (name, e)
        off += n
    assert _frob(out["params"] - theta_before, r["params"] - theta_before) <= GRAD_TOL


def _step(torch, model, x, labels, B):
    out_d = torch.empty(B * 64 * 16 * 16, dtype=torch.int16, device="cuda")
    A.fo_device_step(model, to_dev(x), to_dev(labels), B, out_d)
    return dict(loss=A.fo_model_read(model, A.FO_BUF_LOSS)[0],
                logits=A.fo_model_read(model, A.FO_BUF_LOGITS).reshape(B, 10),
                grads=A.fo_model_read(model, A.FO_BUF_GRADS),
                params=A.fo_model_read(model, A.FO_BUF_PARAMS).astype(np.float64),
                acts=out_d.cpu().numpy().view(np.uint16))


@pytest.mark.parametrize("B,sub", [(64, 1), (5, 2), (1, 3)])
def test_device_step_parity(B, sub):
    torch = torch_cuda()
    announce(f"device step B={B}")
    theta = S.init_params(CID)
    x = S.make_acts(CID, 1, batch=B, sub=sub)[0]
    labels = S.make_labels(CID, 1, batch=B, sub=sub)[0]
    model = A.fo_model_create(CID, 64, theta, torch.cuda.current_stream())
    try:
        out = _step(torch, model, x, labels, B)
    finally:
        A.fo_model_destroy(model)
    r = oracle.device_step(CID, theta, x, labels, lr=0.01)
    _check(out, theta.astype(np.float64), r, B)


def test_device_steps_in_a_row():
    """Three local iterations on fresh batches (Alg. 1's inner loop), each
    checked from the library's parameters just before it."""
    torch = torch_cuda()
    announce("device step chain of 3, B=64")
    B = 64
    xs = S.make_acts(CID, 3, batch=B, sub=11)
    ls = S.make_labels(CID, 3, batch=B, sub=11)
    model = A.fo_model_create(CID, B, S.init_params(CID), torch.cuda.current_stream())
    try:
        prev = S.init_params(CID).astype(np.float64)
        for i in range(3):
            out = _step(torch, model, xs[i], ls[i], B)
            r = oracle.device_step(CID, prev, xs[i], ls[i], lr=0.01)
            _check(out, prev, r, B)
            prev = out["params"]
    finally:
        A.fo_model_destroy(model)


def test_devices_feed_the_server():
    """Four simulated devices each run a local iteration and put their
    activations into the server's pool; the scheduler picks them in
    round-robin order and the server (config 2) trains on each.  Every server
    step is compared with the oracle's server step on the activations that
    device sent (bit-identical to what the pool holds), so the two halves of
    the split meet through the library alone; the server never returns a
    gradient to the devices."""
    torch = torch_cuda()
    announce("four devices -> pool -> server (config 2)")
    K, B = 4, 16
    stream = torch.cuda.current_stream()
    dev = A.fo_model_create(CID, B, S.init_params(CID), stream)
    srv = A.fo_model_create(2, B, S.init_params(2), stream)
    q = A.fo_queues_create(K, B * 64 * 16 * 16 * 2, B, False, K + 4, stream)
    sent = {}
    try:
        xs = S.make_acts(CID, K, batch=B, sub=21)
        ls = S.make_labels(CID, K, batch=B, sub=21)
        lab_d = to_dev(ls)
        for k in range(K):  # devices share one model object here; each trains on its own batch
            out_d = torch.empty(B * 64 * 16 * 16, dtype=torch.int16, device="cuda")
            A.fo_device_step(dev, to_dev(xs[k]), lab_d[k], B, out_d)
            assert A.fo_queues_push(q, k, out_d, lab_d[k]) == A.FO_OK
            sent[k] = out_d.cpu().numpy().view(np.uint16).reshape(B, 64, 16, 16).copy()
        theta = S.init_params(2).astype(np.float64)
        order = []
        while True:
            k = A.fo_pick_device(q)
            if k < 0:
                break
            order.append(k)
            fa, lab, _, _ = A.fo_queues_in_service(q)
            A.fo_server_step(srv, fa, lab, k)
            A.fo_queues_release(q)
            r = oracle.server_step(2, theta, sent[k], ls[k], lr=0.01)
            loss = A.fo_model_read(srv, A.FO_BUF_LOSS)[0]
            assert abs(loss - r["loss"]) <= TOL * abs(r["loss"]), (k, loss, r["loss"])
            assert normwise(A.fo_model_read(srv, A.FO_BUF_LOGITS).reshape(B, 10), r["logits"]) <= TOL
            theta = A.fo_model_read(srv, A.FO_BUF_PARAMS).astype(np.float64)
        assert order == [0, 1, 2, 3]
    finally:
        A.fo_queues_destroy(q)
        A.fo_model_destroy(srv)
        A.fo_model_destroy(dev)


def test_device_and_server_models_are_not_interchangeable():
    torch = torch_cuda()
    announce("device / server entry points refuse the other kind of model")
    stream = torch.cuda.current_stream()
    dev = A.fo_model_create(CID, 4, S.init_params(CID), stream)
    srv = A.fo_model_create(2, 4, S.init_params(2), stream)
    try:
        x = torch.zeros(4 * 3 * 32 * 32, dtype=torch.float32, device="cuda")
        lab = torch.zeros(4, dtype=torch.int32, device="cuda")
        out = torch.empty(4 * 64 * 16 * 16, dtype=torch.int16, device="cuda")
        with pytest.raises(A.FoError):
            A.fo_device_step(srv, x, lab, 4, out)
        with pytest.raises(A.FoError):
            A.fo_server_step(dev, (out, None, 4), lab, 0)
    finally:
        A.fo_model_destroy(dev)
        A.fo_model_destroy(srv)
