"""Pre-processor of the initialization stage (Sec. 3.2.1, Eq. 6-8; auxiliary
network of Sec. 3.2.2), written plainly.

Test infrastructure (see package docstring).  Readings taken where the
paper is silent:

* Layer tables.  A network is a list of units that can be split after: a
  convolution (with its normalisation and activation), a pooling layer, a
  fully connected layer, a MobileNetV3 bottleneck block, an embedding, a
  transformer encoder layer.  Blocks are never cut (the paper splits only at
  sequential connections).  fwd_flops counts the multiply-adds of
  convolutions and matrix products (2 FLOPs each) of one sample's forward
  pass; normalisation, activations, pooling and softmax are not counted.
  out_elems is the number of output values of one sample.
* Eq. 6-8 inputs.  O_l = 3 x fwd_flops(l) x batch (forward, input gradient
  and weight gradient of one training iteration); S_l = out_elems(l) x batch x
  bytes per value (what a device sends if the split follows layer l).  The
  split l ranges over 1..L as in Eq. 8; ties go to the smallest l.
* Architectures.  VGG-5 (Table 4): conv3-32, pool, conv3-64, pool, conv3-64,
  pool, fc-128, fc-X on 32x32x3 inputs; each convolution is followed by a
  batch norm and carries no bias (the norm's shift makes one redundant).  MobileNetV3-Large (Table 4, with the bottleneck expansions, strides,
  squeeze-excitation placement and activations of its own definition,
  Howard et al., 2019): squeeze width = the expansion / 4 rounded to a
  multiple of 8 as in that definition; the last two layers after the global
  pool are fully connected.  Transformer-6/12 (Table 4): EMB-100 (lookup, no
  FLOPs; its table size is not given, so it counts no parameters), encoder
  layers with d = 100, the given heads and FFN width, post-norm, then fc-X on
  the first token.  VGG-16 on 32x32 inputs: the thirteen 3x3 convolutions
  with five pools and fc 512-512-X, as the server workloads use it.
* Auxiliary network (Sec. 3.2.2, default option): one unit of the same kind
  as the last unit of M_d that has parameters (pools are skipped), with that
  unit's width, stride 1, then a classifier: global average pool and fc-X
  after a spatial unit, fc-X on the first token after an encoder, fc-X after
  a fully connected unit.  After an embedding the auxiliary network is the
  classifier alone.
"""
from __future__ import annotations

CONV, POOL, FC, BNECK, EMB, ENC = 1, 2, 3, 4, 6, 7
NETS = {"vgg5": 1, "mobilenetv3_large": 2, "transformer6": 3, "transformer12": 4, "vgg16": 5}


def _div8(v):
    """Round v to a multiple of 8 (at least 8), never below 90% of v."""
    n = max(8, int(v + 4) // 8 * 8)
    return n + 8 if n < 0.9 * v else n


def _layer(kind, k=0, stride=1, c_in=0, c_out=0, h=0, w=0, expand=0, heads=0, hidden=0, norm=0, se=0, params=0,
           flops=0.0, out=0.0):
    return dict(kind=kind, k=k, stride=stride, c_in=c_in, c_out=c_out, h_out=h, w_out=w, expand=expand,
                heads=heads, hidden=hidden, norm=norm, se=se, params=params, fwd_flops=float(flops),
                out_elems=float(out))


def conv(k, stride, c_in, c_out, h_in, w_in, bias=True, bn=True):
    ho, wo = (h_in + 2 * (k // 2) - k) // stride + 1, (w_in + 2 * (k // 2) - k) // stride + 1
    params = k * k * c_in * c_out + (c_out if bias else 0) + (2 * c_out if bn else 0)
    return _layer(CONV, k, stride, c_in, c_out, ho, wo, norm=int(bn), params=params,
                  flops=2 * k * k * c_in * c_out * ho * wo, out=c_out * ho * wo)


def pool(c, h_in, w_in, size=2):
    if size == 0:  # global average
        return _layer(POOL, 0, 1, c, c, 1, 1, out=c)
    return _layer(POOL, size, size, c, c, h_in // size, w_in // size, out=c * (h_in // size) * (w_in // size))


def fc(c_in, c_out):
    return _layer(FC, 0, 1, c_in, c_out, 1, 1, params=c_in * c_out + c_out, flops=2 * c_in * c_out, out=c_out)


def bneck(k, expand, c_in, c_out, se, stride, h_in, w_in):
    """Expansion 1x1 (absent when expand == c_in), depthwise k x k, optional
    squeeze-excitation, projection 1x1; batch norm after each convolution."""
    ho, wo = (h_in + 2 * (k // 2) - k) // stride + 1, (w_in + 2 * (k // 2) - k) // stride + 1
    params = flops = 0
    if expand != c_in:
        params += c_in * expand + 2 * expand
        flops += 2 * c_in * expand * h_in * w_in
    params += k * k * expand + 2 * expand
    flops += 2 * k * k * expand * ho * wo
    if se:
        s = _div8(expand // 4)
        params += expand * s + s + s * expand + expand
        flops += 2 * (expand * s + s * expand)
    params += expand * c_out + 2 * c_out
    flops += 2 * expand * c_out * ho * wo
    return _layer(BNECK, k, stride, c_in, c_out, ho, wo, expand=expand, norm=1, se=int(se), params=params,
                  flops=flops, out=c_out * ho * wo)


def emb(d, seq):
    return _layer(EMB, 0, 1, 0, d, seq, 1, out=d * seq)


def enc(d, heads, hidden, seq):
    params = 4 * d * d + 4 * d + 2 * d + d * hidden + hidden + hidden * d + d + 2 * d
    flops = 2 * seq * d * 3 * d + 2 * seq * seq * d * 2 + 2 * seq * d * d + 2 * seq * d * hidden * 2
    return _layer(ENC, 0, 1, d, d, seq, 1, heads=heads, hidden=hidden, norm=1, params=params, flops=flops,
                  out=d * seq)


MBV3_LARGE = [  # (kernel, expansion, out channels, squeeze-excitation, stride)
    (3, 16, 16, False, 1), (3, 64, 24, False, 2), (3, 72, 24, False, 1), (5, 72, 40, True, 2),
    (5, 120, 40, True, 1), (5, 120, 40, True, 1), (3, 240, 80, False, 2), (3, 200, 80, False, 1),
    (3, 184, 80, False, 1), (3, 184, 80, False, 1), (3, 480, 112, True, 1), (3, 672, 112, True, 1),
    (5, 672, 160, True, 2), (5, 960, 160, True, 1), (5, 960, 160, True, 1),
]


def net_layers(net: str, classes: int, in_hw: int):
    """The unit table of a network: in_hw is the image side (CNNs) or the
    sequence length (transformers)."""
    L = []
    if net == "vgg5":
        h = in_hw
        for c_in, c_out in ((3, 32), (32, 64), (64, 64)):
            L.append(conv(3, 1, c_in, c_out, h, h, bias=False))
            L.append(pool(c_out, h, h))
            h //= 2
        L.append(fc(64 * h * h, 128))
        L.append(fc(128, classes))
    elif net == "vgg16":
        h, c = in_hw, 3
        for v in (64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512, "M"):
            if v == "M":
                L.append(pool(c, h, h))
                h //= 2
            else:
                L.append(conv(3, 1, c, v, h, h, bn=False))
                c = v
        L += [fc(c * h * h, 512), fc(512, 512), fc(512, classes)]
    elif net == "mobilenetv3_large":
        L.append(conv(3, 2, 3, 16, in_hw, in_hw, bias=False))
        h, c = L[-1]["h_out"], 16
        for k, e, o, se, s in MBV3_LARGE:
            L.append(bneck(k, e, c, o, se, s, h, h))
            h, c = L[-1]["h_out"], o
        L.append(conv(1, 1, c, 960, h, h, bias=False))
        L.append(pool(960, h, h, size=0))
        L.append(fc(960, 1280))
        L.append(fc(1280, classes))
    elif net in ("transformer6", "transformer12"):
        n, heads = (6, 5) if net == "transformer6" else (12, 50)
        L.append(emb(100, in_hw))
        for _ in range(n):
            L.append(enc(100, heads, 100, in_hw))
        L.append(fc(100, classes))
    else:
        raise ValueError(net)
    return L


def split_costs(layers, batch, act_bytes, o, b):
    """Eq. 6-8: for every split l (1-based), max over devices of
    max(sum_{i<=l} O_i / o_k, S_l / b_k)."""
    costs, prefix = [], 0.0
    for lay in layers:
        prefix += 3.0 * lay["fwd_flops"] * batch
        S = lay["out_elems"] * batch * act_bytes
        costs.append(max(max(prefix / ok, S / bk) for ok, bk in zip(o, b)))
    return costs


def select_split(layers, batch, act_bytes, o, b):
    costs = split_costs(layers, batch, act_bytes, o, b)
    best = min(range(len(costs)), key=lambda i: (costs[i], i))
    return best + 1, costs


def aux_network(layers, l, classes):
    """The default auxiliary network for the split after unit l (1-based)."""
    last = next((lay for lay in reversed(layers[:l]) if lay["kind"] != POOL), None)
    if last is None:
        raise ValueError("no unit with parameters before the split")
    out = layers[l - 1]
    kind = last["kind"]
    if kind == CONV:
        h, w, c = out["h_out"], out["w_out"], out["c_out"]
        u = conv(last["k"], 1, c, c, h, w, bias=True, bn=bool(last["norm"]))
        return [u, pool(c, h, w, size=0), fc(c, classes)]
    if kind == BNECK:
        h, w, c = out["h_out"], out["w_out"], out["c_out"]
        u = bneck(last["k"], last["expand"], c, c, bool(last["se"]), 1, h, w)
        return [u, pool(c, h, w, size=0), fc(c, classes)]
    if kind == ENC:
        return [enc(last["c_out"], last["heads"], last["hidden"], last["h_out"]), fc(last["c_out"], classes)]
    if kind == EMB:
        return [fc(last["c_out"], classes)]
    if kind == FC:
        return [fc(last["c_out"], last["c_out"]), fc(last["c_out"], classes)]
    raise ValueError(kind)

