"""A second, independent statement of the server networks written with
PyTorch's CPU autograd in fp64.  Used only to pin the oracle (forward values
and every gradient); it never touches the HIP library."""
import numpy as np
import torch
import torch.nn.functional as F

from fo_synth import param_layout


def _params(cid, flat):
    out, off = {}, 0
    for name, shape, _, _ in param_layout(cid):
        n = int(np.prod(shape))
        t = torch.tensor(np.asarray(flat[off:off + n], np.float64).reshape(shape), requires_grad=True)
        out[name] = t
        off += n
    return out


def _w4(t):  # flat [Co, kh, kw, Ci] -> torch [Co, Ci, kh, kw]
    return t.permute(0, 3, 1, 2)


def forward(cid, P, x, lengths=None):
    if cid == 1:
        h = F.max_pool2d(F.relu(F.conv2d(x, _w4(P["conv1.w"]), P["conv1.b"], padding=1)), 2)
        h = F.relu(F.conv2d(h, _w4(P["conv2.w"]), P["conv2.b"], padding=1)).mean((2, 3))
        return F.linear(h, P["fc.w"], P["fc.b"])
    if cid in (2, 5):
        h, i = x, 0
        for v in [128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512, "M"]:
            if v == "M":
                h = F.max_pool2d(h, 2)
            else:
                h = F.relu(F.conv2d(h, _w4(P[f"conv{i}.w"]), P[f"conv{i}.b"], padding=1))
                i += 1
        h = h.flatten(1)
        h = F.relu(F.linear(h, P["fc0.w"], P["fc0.b"]))
        h = F.relu(F.linear(h, P["fc1.w"], P["fc1.b"]))
        return F.linear(h, P["fc2.w"], P["fc2.b"])
    if cid == 3:
        def bn(h, n):
            return F.batch_norm(h, None, None, P[n + ".g"], P[n + ".b"], training=True, eps=1e-5)
        h = x
        for st in (2, 3, 4):
            for bi in range(2):
                p = f"layer{st}.{bi}"
                s = 2 if bi == 0 else 1
                o = F.relu(bn(F.conv2d(h, _w4(P[p + ".conv1.w"]), stride=s, padding=1), p + ".bn1"))
                o = bn(F.conv2d(o, _w4(P[p + ".conv2.w"]), padding=1), p + ".bn2")
                sc = bn(F.conv2d(h, _w4(P[p + ".ds.w"]), stride=2), p + ".dsbn") if bi == 0 else h
                h = F.relu(o + sc)
        return F.linear(h.mean((2, 3)), P["fc.w"], P["fc.b"])
    if cid == 10:
        from oracle.nets import MBV3_TAIL

        def hswish(t):  # x ReLU6(x + 3) / 6, differentiated exactly by autograd
            return t * torch.clamp(t + 3.0, 0.0, 6.0) / 6.0

        def hsigmoid(t):
            return torch.clamp(t + 3.0, 0.0, 6.0) / 6.0

        def bn(h, n):
            return F.batch_norm(h, None, None, P[n + ".g"], P[n + ".b"], training=True, eps=1e-5)
        h, ci = x, 80
        for j, (k, e, co, se, st) in enumerate(MBV3_TAIL):
            p = f"b{j}"
            t = hswish(bn(F.conv2d(h, _w4(P[p + ".expand.w"])), p + ".bn1"))
            t = hswish(bn(F.conv2d(t, _w4(P[p + ".dw.w"]), stride=st, padding=k // 2, groups=e), p + ".bn2"))
            if se:
                sq = F.relu(F.linear(t.mean((2, 3)), P[p + ".se.fc1.w"], P[p + ".se.fc1.b"]))
                t = t * hsigmoid(F.linear(sq, P[p + ".se.fc2.w"], P[p + ".se.fc2.b"]))[:, :, None, None]
            t = bn(F.conv2d(t, _w4(P[p + ".proj.w"])), p + ".bn3")
            h = t + h if st == 1 and ci == co else t
            ci = co
        h = hswish(bn(F.conv2d(h, _w4(P["last.w"])), "last_bn")).mean((2, 3))
        return F.linear(hswish(F.linear(h, P["fc1.w"], P["fc1.b"])), P["fc2.w"], P["fc2.b"])
    if cid == 9:
        h = F.batch_norm(F.conv2d(x, _w4(P["conv.w"]), padding=1), None, None, P["bn.g"], P["bn.b"],
                         training=True, eps=1e-5)
        h = F.max_pool2d(F.relu(h), 2).flatten(1)
        return F.linear(F.relu(F.linear(h, P["fc1.w"], P["fc1.b"])), P["fc2.w"], P["fc2.b"])
    if cid == 6:  # device network, then the auxiliary network on its output
        xi = F.max_pool2d(F.relu(F.conv2d(F.relu(F.conv2d(x, _w4(P["conv1.w"]), P["conv1.b"], padding=1)),
                                          _w4(P["conv2.w"]), P["conv2.b"], padding=1)), 2)
        forward.last_acts = xi
        h = F.relu(F.conv2d(xi, _w4(P["aux.conv.w"]), P["aux.conv.b"], padding=1)).mean((2, 3))
        return F.linear(h, P["aux.fc.w"], P["aux.fc.b"])
    if cid in (7, 8):
        B, L, d = x.shape
        H = 5 if cid == 7 else 50
        dh = d // H
        mask = torch.arange(L)[None, :] >= torch.as_tensor(lengths)[:, None]
        h = x
        for li in range(6 if cid == 7 else 12):
            p = f"enc{li}"
            qkv = F.linear(h, P[p + ".qkv.w"], P[p + ".qkv.b"])
            q, k, v = (qkv[..., i * d:(i + 1) * d].reshape(B, L, H, dh).transpose(1, 2) for i in range(3))
            s = torch.matmul(q, k.transpose(-1, -2)) / dh ** 0.5
            s = s.masked_fill(mask[:, None, None, :], float("-inf"))
            o = torch.matmul(torch.softmax(s, -1), v).transpose(1, 2).reshape(B, L, d)
            h = F.layer_norm(h + F.linear(o, P[p + ".o.w"], P[p + ".o.b"]), (d,), P[p + ".ln1.g"], P[p + ".ln1.b"], 1e-5)
            f = F.linear(F.relu(F.linear(h, P[p + ".ffn1.w"], P[p + ".ffn1.b"])), P[p + ".ffn2.w"], P[p + ".ffn2.b"])
            h = F.layer_norm(h + f, (d,), P[p + ".ln2.g"], P[p + ".ln2.b"], 1e-5)
        return F.linear(h[:, 0], P["cls.w"], P["cls.b"])
    if cid == 4:
        B, L, d = x.shape
        H, dh = 12, 64
        mask = torch.arange(L)[None, :] >= torch.as_tensor(lengths)[:, None]
        h = x
        for li in range(10):
            p = f"enc{li}"
            qkv = F.linear(h, P[p + ".qkv.w"], P[p + ".qkv.b"])
            q, k, v = (qkv[..., i * d:(i + 1) * d].reshape(B, L, H, dh).transpose(1, 2) for i in range(3))
            s = torch.matmul(q, k.transpose(-1, -2)) / 8.0
            s = s.masked_fill(mask[:, None, None, :], float("-inf"))
            o = torch.matmul(torch.softmax(s, -1), v).transpose(1, 2).reshape(B, L, d)
            h = F.layer_norm(h + F.linear(o, P[p + ".o.w"], P[p + ".o.b"]), (d,), P[p + ".ln1.g"], P[p + ".ln1.b"], 1e-5)
            f = F.linear(F.gelu(F.linear(h, P[p + ".ffn1.w"], P[p + ".ffn1.b"])), P[p + ".ffn2.w"], P[p + ".ffn2.b"])
            h = F.layer_norm(h + f, (d,), P[p + ".ln2.g"], P[p + ".ln2.b"], 1e-5)
        pooled = torch.tanh(F.linear(h[:, 0], P["pool.w"], P["pool.b"]))
        return F.linear(pooled, P["cls.w"], P["cls.b"])
    raise ValueError(cid)


def step(cid, flat, x, labels, lengths=None):
    """Returns (loss, logits, flat gradient) from torch autograd in fp64."""
    P = _params(cid, flat)
    xt = torch.tensor(np.asarray(x, np.float64))
    z = forward(cid, P, xt, lengths)
    loss = F.cross_entropy(z, torch.tensor(np.asarray(labels, np.int64)))
    loss.backward()
    g = np.concatenate([P[n].grad.numpy().reshape(-1) for n, _, _, _ in param_layout(cid)])
    return float(loss), z.detach().numpy(), g
