"""Graph replay of the server and device steps (fo_set_graph_mode) against
direct launches.

With graph mode on, fo_server_step (fo_device_step) replays a HIP graph
captured once per batch size, after setting the arguments of its first
launch, which stores the batch's pointers for the other kernels.  Every kernel of
the step is deterministic (no atomics), so a replayed step must give results
bit-identical to the same step launched kernel by kernel.  Each case runs one
model per mode through the same sequence of batches: several replays at one
batch size, a smaller (ragged) batch that captures a second graph, then the
first size again; every batch lives in a fresh device tensor (the caller's
pointers change between replays), and unrelated eager work plus a device
synchronisation sit between consecutive steps."""
import numpy as np
import pytest

import fo_synth as S
from tests.gpu_util import announce, to_dev, torch_cuda

pytestmark = pytest.mark.gpu
A = pytest.importorskip("paper_2504_13850_amd.api")


def _batch(cid, B, sub):
    cfg = S.get_config(cid)
    acts = S.make_acts(cid, 1, batch=B, sub=sub)[0]
    if cfg.dtype != "f32":
        acts = acts.view(np.int16)
    labels = S.make_labels(cid, 1, batch=B, sub=sub)[0]
    lengths = S.make_lengths(cid, 1, batch=B, sub=sub)[0] if cfg.family in ("bert", "tfsmall") else None
    return acts, labels, lengths


def _read_all(model, cfg, B):
    out = dict(loss=A.fo_model_read(model, A.FO_BUF_LOSS),
               logits=A.fo_model_read(model, A.FO_BUF_LOGITS)[:B * cfg.n_classes],
               grads=A.fo_model_read(model, A.FO_BUF_GRADS),
               params=A.fo_model_read(model, A.FO_BUF_PARAMS))
    if cfg.momentum:
        out["mom"] = A.fo_model_read(model, A.FO_BUF_MOMENTUM)
    return out


def _eager_noise(torch, step):
    """Unrelated work on torch's stream between steps."""
    g = torch.Generator(device="cuda").manual_seed(1000 + step)
    a = torch.randn(512, 512, device="cuda", generator=g)
    b = torch.zeros(512, 512, device="cuda")
    b.copy_(a @ a.T)
    b.zero_()
    return float(a.sum().item())


@pytest.mark.parametrize("cid,Bmax", [(1, 8), (2, 8), (3, 8), (4, 6), (5, 8), (6, 8), (7, 8), (8, 4), (9, 8), (10, 8)])
def test_graph_replay_matches_direct_launches(cid, Bmax):
    torch = torch_cuda()
    cfg = S.get_config(cid)
    theta = S.init_params(cid)
    sizes = [Bmax, Bmax, Bmax, Bmax // 2 + 1, Bmax // 2 + 1, Bmax]
    stream = torch.cuda.current_stream()
    graph = direct = None
    try:
        graph = A.fo_model_create(cid, Bmax, theta, stream)
        direct = A.fo_model_create(cid, Bmax, theta, stream)
        for step, B in enumerate(sizes):
            announce(f"graph replay cid={cid} step={step} B={B}")
            acts, labels, lengths = _batch(cid, B, sub=step + 1)
            outs = []
            for mode, model in ((True, graph), (False, direct)):
                A.fo_set_graph_mode(mode)
                x, lab = to_dev(acts), to_dev(labels)
                ln = to_dev(lengths) if lengths is not None else None
                if cid == 6:  # the device step: its activations are compared too
                    out = torch.empty(B * 64 * 16 * 16, dtype=torch.int16, device="cuda")
                    A.fo_device_step(model, x, lab, B, out)
                    outs.append(_read_all(model, cfg, B))
                    outs[-1]["acts"] = out.cpu().numpy()
                    del out
                else:
                    A.fo_server_step(model, (x, ln, B), lab, step % 3)
                    outs.append(_read_all(model, cfg, B))
                del x, lab, ln
                _eager_noise(torch, step)
                torch.cuda.synchronize()
            got, ref = outs
            for k in ref:
                assert np.array_equal(got[k], ref[k]), f"cid={cid} step={step} B={B}: {k} differs"
            assert np.isfinite(ref["loss"]).all()
        assert A.fo_model_steps(graph, -1) == len(sizes) == A.fo_model_steps(direct, -1)
    finally:
        A.fo_set_graph_mode(True)
        for model in (graph, direct):
            if model is not None:
                A.fo_model_destroy(model)
