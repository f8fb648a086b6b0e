"""GPU parity of the fp32 tiny-CNN server step (config 1) against the fp64
oracle, through the C ABI: loss, logits, every gradient tensor and the
parameter update, per step of a round-robin trace drawn by the scheduler."""
import numpy as np
import pytest

import fo_synth as S
import oracle
from oracle import layers as OL
from oracle import nets as ON
from tests.gpu_util import announce, normwise, per_tensor_errors, to_dev, torch_cuda

pytestmark = pytest.mark.gpu
A = pytest.importorskip("paper_2504_13850_amd.api")

CID = 1
TOL = 1e-4


def _pool_margin(cid, theta, acts):
    """Smallest gap between the winner and the runner-up of any 2x2 pool
    window with a positive winner, relative to the winner (a near tie could
    route a gradient differently at fp32)."""
    P = ON.unpack(cid, theta, np.float64)
    x = ON.decode_acts(acts, np.float64)
    y = OL.ReLU().fwd(OL.Conv2d(P["conv1.w"], P["conv1.b"]).fwd(x))
    B, C, H, W = y.shape
    win = np.sort(y.reshape(B, C, H // 2, 2, W // 2, 2).transpose(0, 1, 2, 4, 3, 5).reshape(-1, 4), axis=1)
    pos = win[:, 3] > 0
    return np.min((win[pos, 3] - win[pos, 2]) / win[pos, 3])


def _check_step(model, theta, acts, labels, B):
    ref = oracle.server_step(CID, theta, acts, labels, lr=0.01)
    loss = A.fo_model_read(model, A.FO_BUF_LOSS)[0]
    logits = A.fo_model_read(model, A.FO_BUF_LOGITS).reshape(B, 10)
    grads = A.fo_model_read(model, A.FO_BUF_GRADS)
    params = A.fo_model_read(model, A.FO_BUF_PARAMS)
    assert abs(loss - ref["loss"]) <= TOL * abs(ref["loss"])
    assert normwise(logits, ref["logits"]) <= TOL
    errs = per_tensor_errors(CID, grads, ref["grads"])
    assert max(errs.values()) <= TOL, errs
    dtheta = params.astype(np.float64) - theta.astype(np.float64)
    assert normwise(dtheta, ref["params"] - theta) <= 10 * TOL  # Δθ carries fp32 cancellation
    return params


@pytest.mark.parametrize("B", [16, 3, 1])
def test_single_step_parity(B):
    torch = torch_cuda()
    announce(f"config 1 step B={B}")
    theta = S.init_params(CID)
    # first seed whose pooling windows have no near tie (a tie closer than the
    # fp32 rounding of the conv could route a gradient to the other element)
    sub = next(k for k in range(B, B + 50)
               if _pool_margin(CID, theta, S.make_acts(CID, 1, batch=B, sub=k)[0]) > 1e-5)
    acts = S.make_acts(CID, 1, batch=B, sub=sub)[0]
    labels = S.make_labels(CID, 1, batch=B, sub=sub)[0]
    model = A.fo_model_create(CID, 16, theta, torch.cuda.current_stream())
    try:
        A.fo_server_step(model, (to_dev(acts), None, B), to_dev(labels), 0)
        _check_step(model, theta, acts, labels, B)
        assert A.fo_model_steps(model, 0) == 1
    finally:
        A.fo_model_destroy(model)


def test_round_robin_trace_through_pool():
    """4 devices, one batch each, drawn by fo_pick_device in round-robin order
    (equal counters, lowest index first); each step checked against the oracle
    continuing from the previous oracle parameters."""
    torch = torch_cuda()
    announce("config 1 pool trace")
    K, B = 4, 16
    theta = S.init_params(CID)
    acts = S.make_acts(CID, K)
    labels = S.make_labels(CID, K)
    stream = torch.cuda.current_stream()
    slot_bytes = acts[0].nbytes
    q = A.fo_queues_create(K, slot_bytes, B, False, K + 4, stream)
    model = A.fo_model_create(CID, B, theta, stream)
    try:
        for k in (3, 1, 0, 2):  # arrival order does not matter: the counters decide
            st = A.fo_queues_push(q, k, acts[k], labels[k], None, on_host=True)
            assert st == A.FO_OK
        order = []
        cur = theta.copy()
        while True:
            k = A.fo_pick_device(q)
            if k < 0:
                break
            order.append(k)
            fa, lab_ptr, seq, slot = A.fo_queues_in_service(q)
            A.fo_server_step(model, fa, lab_ptr, k)
            A.fo_queues_release(q)
            new = _check_step(model, cur, acts[k], labels[k], B)
            cur = new
        assert order == [0, 1, 2, 3]
        assert A.fo_queues_counters(q, K) == [1, 1, 1, 1]
    finally:
        A.fo_model_destroy(model)
        A.fo_queues_destroy(q)


def test_checkpoint_write_read_roundtrip():
    torch = torch_cuda()
    announce("config 1 checkpoint")
    theta = S.init_params(CID)
    model = A.fo_model_create(CID, 4, theta, torch.cuda.current_stream())
    try:
        assert A.fo_model_read(model, A.FO_BUF_PARAMS).tobytes() == theta.tobytes()
        t2 = (theta * 0.5).astype(np.float32)
        A.fo_model_write(model, A.FO_BUF_PARAMS, t2)
        assert A.fo_model_read(model, A.FO_BUF_PARAMS).tobytes() == t2.tobytes()
        with pytest.raises(A.FoError):
            A.fo_model_read(model, A.FO_BUF_LOSS)  # no step yet
    finally:
        A.fo_model_destroy(model)
