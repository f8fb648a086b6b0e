"""Multi-step GPU parity: consecutive server steps on fresh seeded batches,
each compared with the oracle chained on its own state.

One training iteration of Alg. 4 updates the parameters (and, for the
ResNet workload, the momentum buffer v <- mu v + g, theta <- theta - lr v).
A single step from a zero buffer cannot show the mu v term (v_1 = g_1), so
these tests run three steps in a row on three different batches and, after
every step, compare the library's state with the oracle's state after the
same number of steps, the oracle starting each step from its own parameters
and momentum buffer:

  graded:   loss and logits of the step (2e-2, normwise for logits);
  checked:  every gradient tensor, the update of the step
            (theta_i - theta_{i-1}) and the momentum buffer, by relative
            Frobenius error <= 6e-2 (bf16 gradients; a dropped or mis-scaled
            term moves them by O(1)).

A wrong momentum coefficient changes the step-2 update by about mu |v_1| /
|v_2|, which is of order one here."""
import numpy as np
import pytest

import fo_synth as S
import oracle
from tests.gpu_util import announce, normwise, to_dev, torch_cuda

pytestmark = pytest.mark.gpu
A = pytest.importorskip("paper_2504_13850_amd.api")

TOL = 2e-2
GRAD_TOL = 6e-2
N_STEPS = 3


def _frob(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)


def _worst_tensor(cid, got, ref):
    worst, name, off = -1.0, None, 0
    for nm, shape, _, _ in S.param_layout(cid):
        n = int(np.prod(shape))
        e = _frob(got[off:off + n], ref[off:off + n])
        if e > worst:
            worst, name = e, nm
        off += n
    return name, worst


def _chain(cid, B, sub, with_lengths=False):
    torch = torch_cuda()
    cfg = S.get_config(cid)
    theta = S.init_params(cid)
    acts = S.make_acts(cid, N_STEPS, batch=B, sub=sub)
    labels = S.make_labels(cid, N_STEPS, batch=B, sub=sub)
    lengths = S.make_lengths(cid, N_STEPS, batch=B, sub=sub) if with_lengths else [None] * N_STEPS
    model = A.fo_model_create(cid, B, theta, torch.cuda.current_stream())
    ref_theta = theta.astype(np.float64)
    ref_mom = None
    prev = theta.astype(np.float64)
    report = []
    try:
        for i in range(N_STEPS):
            x = to_dev(acts[i] if cfg.dtype == "f32" else acts[i].view(np.int16))
            lab = to_dev(labels[i])
            ln = to_dev(lengths[i]) if with_lengths else None
            A.fo_server_step(model, (x, ln, B), lab, i)
            loss = A.fo_model_read(model, A.FO_BUF_LOSS)[0]
            logits = A.fo_model_read(model, A.FO_BUF_LOGITS).reshape(B, cfg.n_classes)
            grads = A.fo_model_read(model, A.FO_BUF_GRADS)
            params = A.fo_model_read(model, A.FO_BUF_PARAMS).astype(np.float64)
            r = oracle.server_step(cid, ref_theta, acts[i], labels[i], lengths[i], lr=cfg.lr,
                                   momentum=cfg.momentum, mom_buf=ref_mom)
            e_loss = abs(loss - r["loss"]) / abs(r["loss"])
            e_logit = normwise(logits, r["logits"])
            gname, e_grad = _worst_tensor(cid, grads, r["grads"])
            e_upd = _frob(params - prev, r["params"] - ref_theta)
            rec = dict(step=i + 1, loss=e_loss, logits=e_logit, grad=(gname, e_grad), update=e_upd)
            if cfg.momentum:
                rec["momentum"] = _frob(A.fo_model_read(model, A.FO_BUF_MOMENTUM), r["momentum"])
            report.append(rec)
            assert e_loss <= TOL, rec
            assert e_logit <= TOL, rec
            assert e_grad <= GRAD_TOL, rec
            assert e_upd <= GRAD_TOL, rec
            if cfg.momentum:
                assert rec["momentum"] <= GRAD_TOL, rec
            prev = params
            ref_theta = r["params"]
            ref_mom = r["momentum"]
    finally:
        A.fo_model_destroy(model)
    print(report)
    return report


def test_resnet_momentum_chain():
    """ResNet-18 split at its workload batch (32), SGD with momentum 0.9:
    from step 2 on the update carries mu v."""
    announce("config 3 chain of 3 steps B=32")
    _chain(3, 32, 21)


def test_vgg_chain():
    """VGG-16 split at its workload batch (64), plain SGD."""
    announce("config 2 chain of 3 steps B=64")
    _chain(2, 64, 23)


def test_transformer_chain():
    """BERT-base-shaped encoder, plain SGD, lengths drawn like the workload
    (uniform on [32, 128]); batch 12 keeps the fp64 oracle to seconds per step."""
    announce("config 4 chain of 3 steps B=12")
    _chain(4, 12, 24, with_lengths=True)
