"""Server-side networks M_s of the server configurations and one training
iteration of the activation branch of Algorithm 4 (forward of M_s, the loss
f_s, the backward pass, then theta_s <- theta_s - gamma_s * grad).

Test infrastructure (see package docstring).  The flat parameter order (the
"library layout") is derived here from the architecture on its own; a test
compares it with the workload description and with the library.  Convolution
weights sit in the flat vector as [Cout][kh][kw][Cin] and are turned into the
[Cout][Cin][kh][kw] form that ``layers.Conv2d`` expects when unpacked.

The server never returns an activation gradient to the devices (the devices
train on their local auxiliary loss instead, Sec. 3.1 and Alg. 1), so the
first server layer's input gradient is not computed.
"""
from __future__ import annotations

import numpy as np

from . import layers as Lyr

# architecture constants per configuration id (from the workload descriptions)
VGG_PLAN = [128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512, "M"]
RESNET_STAGES = [(2, 128, 2), (3, 256, 2), (4, 512, 2)]  # (stage, channels, blocks)
BERT = dict(d=768, heads=12, ffn=3072, layers=10, classes=2)
# the paper's Transformer-6 and Transformer-12 (Table 4) after their embedding
TFSMALL = {7: dict(d=100, heads=5, ffn=100, layers=6), 8: dict(d=100, heads=50, ffn=100, layers=12)}
FAMILY = {1: "cnn", 2: "vgg", 3: "resnet", 4: "bert", 5: "vgg", 6: "vgg_device", 7: "tfsmall", 8: "tfsmall",
          9: "vgg5", 10: "mbv3"}
IN_CH = {1: 32, 2: 64, 3: 64, 5: 64, 6: 3, 9: 64, 10: 80}
CLASSES = {1: 10, 2: 10, 3: 100, 4: 2, 5: 10, 6: 10, 7: 2, 8: 2, 9: 10, 10: 200}
# MobileNetV3-Large's last eight bottlenecks (its own definition): kernel,
# expansion, output channels, squeeze-excitation, stride; all hard-swish
MBV3_TAIL = [(3, 200, 80, False, 1), (3, 184, 80, False, 1), (3, 184, 80, False, 1), (3, 480, 112, True, 1),
             (3, 672, 112, True, 1), (5, 672, 160, True, 2), (5, 960, 160, True, 1), (5, 960, 160, True, 1)]


def se_width(e):
    """Squeeze width: e / 4 to a multiple of 8, at least 8, not below 90% of e / 4."""
    v = e // 4
    n = max(8, int(v + 4) // 8 * 8)
    return n + 8 if n < 0.9 * v else n


def param_layout(cid: int):
    """[(name, shape in the flat vector)] in flat order."""
    fam = FAMILY[cid]
    out = []

    def conv(n, co, ci, k, bias=True):
        out.append((n + ".w", (co, k, k, ci)))
        if bias:
            out.append((n + ".b", (co,)))

    def lin(n, o, i):
        out.append((n + ".w", (o, i)))
        out.append((n + ".b", (o,)))

    def norm(n, c):
        out.append((n + ".g", (c,)))
        out.append((n + ".b", (c,)))

    if fam == "cnn":
        conv("conv1", 64, 32, 3)
        conv("conv2", 64, 64, 3)
        lin("fc", 10, 64)
    elif fam == "mbv3":
        ci = IN_CH[cid]
        for j, (k, e, co, se, _) in enumerate(MBV3_TAIL):
            p = f"b{j}"
            conv(p + ".expand", e, ci, 1, bias=False)
            norm(p + ".bn1", e)
            out.append((p + ".dw.w", (e, k, k, 1)))
            norm(p + ".bn2", e)
            if se:
                lin(p + ".se.fc1", se_width(e), e)
                lin(p + ".se.fc2", e, se_width(e))
            conv(p + ".proj", co, e, 1, bias=False)
            norm(p + ".bn3", co)
            ci = co
        conv("last", 960, ci, 1, bias=False)
        norm("last_bn", 960)
        lin("fc1", 1280, 960)
        lin("fc2", CLASSES[cid], 1280)
    elif fam == "vgg5":
        # the server part of VGG-5 (Table 4) after its second pool: CONV-3-64 with
        # batch norm (no bias), pool, FC-128, FC-X on [64, 8, 8] inputs
        conv("conv", 64, IN_CH[cid], 3, bias=False)
        norm("bn", 64)
        lin("fc1", 128, 64 * 4 * 4)
        lin("fc2", CLASSES[cid], 128)
    elif fam == "vgg_device":
        # device network M_d: VGG-16's first block; auxiliary network: one layer
        # of the type of M_d's last layer, then a dense classifier (Sec. 3.2.2)
        conv("conv1", 64, IN_CH[cid], 3)
        conv("conv2", 64, 64, 3)
        conv("aux.conv", 64, 64, 3)
        lin("aux.fc", CLASSES[cid], 64)
    elif fam == "vgg":
        ci, n = IN_CH[cid], 0
        for v in VGG_PLAN:
            if v != "M":
                conv(f"conv{n}", v, ci, 3)
                ci, n = v, n + 1
        lin("fc0", 512, 512)
        lin("fc1", 512, 512)
        lin("fc2", CLASSES[cid], 512)
    elif fam == "resnet":
        ci = IN_CH[cid]
        for st, c, nb in RESNET_STAGES:
            for bi in range(nb):
                p = f"layer{st}.{bi}"
                conv(p + ".conv1", c, ci if bi == 0 else c, 3, bias=False)
                norm(p + ".bn1", c)
                conv(p + ".conv2", c, c, 3, bias=False)
                norm(p + ".bn2", c)
                if bi == 0:
                    conv(p + ".ds", c, ci, 1, bias=False)
                    norm(p + ".dsbn", c)
            ci = c
        lin("fc", CLASSES[cid], 512)
    else:
        arch = BERT if fam == "bert" else TFSMALL[cid]
        d, f = arch["d"], arch["ffn"]
        for li in range(arch["layers"]):
            p = f"enc{li}"
            lin(p + ".qkv", 3 * d, d)
            lin(p + ".o", d, d)
            norm(p + ".ln1", d)
            lin(p + ".ffn1", f, d)
            lin(p + ".ffn2", d, f)
            norm(p + ".ln2", d)
        if fam == "bert":
            lin("pool", d, d)
        lin("cls", CLASSES[cid], d)
    return out


def unpack(cid, flat, dt):
    P, off = {}, 0
    for name, shape in param_layout(cid):
        n = int(np.prod(shape))
        a = np.asarray(flat[off:off + n], dtype=dt).reshape(shape)
        if len(shape) == 4:  # [Co, kh, kw, Ci] -> [Co, Ci, kh, kw]
            a = a.transpose(0, 3, 1, 2).copy()
        P[name] = a
        off += n
    assert off == len(flat), (off, len(flat))
    return P


def pack(cid, G):
    parts = []
    for name, shape in param_layout(cid):
        g = G[name]
        if len(shape) == 4:
            g = g.transpose(0, 2, 3, 1)
        parts.append(np.asarray(g).reshape(-1))
    return np.concatenate(parts)


# ----------------------------------------------------------------------------- networks
class _Net:
    def grads(self):
        return self.G


class CNN(_Net):
    """conv3x3 32->64 + ReLU, maxpool2, conv3x3 64->64 + ReLU, global average
    pool, linear 64->10."""

    def __init__(self, P):
        self.c1 = Lyr.Conv2d(P["conv1.w"], P["conv1.b"])
        self.r1, self.mp = Lyr.ReLU(), Lyr.MaxPool2()
        self.c2 = Lyr.Conv2d(P["conv2.w"], P["conv2.b"])
        self.r2, self.gap = Lyr.ReLU(), Lyr.GlobalAvgPool()
        self.fc = Lyr.Linear(P["fc.w"], P["fc.b"])

    def fwd(self, x, lengths=None):
        h = self.mp.fwd(self.r1.fwd(self.c1.fwd(x)))
        h = self.gap.fwd(self.r2.fwd(self.c2.fwd(h)))
        return self.fc.fwd(h)

    def bwd(self, dz):
        dh = self.gap.bwd(self.fc.bwd(dz))
        dh = self.mp.bwd(self.c2.bwd(self.r2.bwd(dh)))
        self.c1.bwd(self.r1.bwd(dh), need_dx=False)
        self.G = {"conv1.w": self.c1.dw, "conv1.b": self.c1.db, "conv2.w": self.c2.dw,
                  "conv2.b": self.c2.db, "fc.w": self.fc.dw, "fc.b": self.fc.db}


class DeviceVGG(_Net):
    """The device-side network M_d of the VGG-16 split (conv3x3 3->64 + ReLU,
    conv3x3 64->64 + ReLU, 2x2 max pool; its output xi is the activation batch
    the device sends to the server) followed by the auxiliary network on xi
    (conv3x3 64->64 + ReLU, global average pool, dense 64 -> classes), which
    gives the device its local loss f_d (Alg. 1, Sec. 3.2.2)."""

    def __init__(self, P):
        self.c1, self.r1 = Lyr.Conv2d(P["conv1.w"], P["conv1.b"]), Lyr.ReLU()
        self.c2, self.r2 = Lyr.Conv2d(P["conv2.w"], P["conv2.b"]), Lyr.ReLU()
        self.mp = Lyr.MaxPool2()
        self.ca, self.ra = Lyr.Conv2d(P["aux.conv.w"], P["aux.conv.b"]), Lyr.ReLU()
        self.gap = Lyr.GlobalAvgPool()
        self.fc = Lyr.Linear(P["aux.fc.w"], P["aux.fc.b"])

    def fwd(self, x, lengths=None):
        self.xi = self.mp.fwd(self.r2.fwd(self.c2.fwd(self.r1.fwd(self.c1.fwd(x)))))
        return self.fc.fwd(self.gap.fwd(self.ra.fwd(self.ca.fwd(self.xi))))

    def bwd(self, dz):
        dxi = self.ca.bwd(self.ra.bwd(self.gap.bwd(self.fc.bwd(dz))))
        dh = self.c2.bwd(self.r2.bwd(self.mp.bwd(dxi)))
        self.c1.bwd(self.r1.bwd(dh), need_dx=False)  # the input is data: no gradient
        self.G = {"conv1.w": self.c1.dw, "conv1.b": self.c1.db, "conv2.w": self.c2.dw, "conv2.b": self.c2.db,
                  "aux.conv.w": self.ca.dw, "aux.conv.b": self.ca.db, "aux.fc.w": self.fc.dw,
                  "aux.fc.b": self.fc.db}


class VGG(_Net):
    """VGG-16 after its second convolution and first pool: ten 3x3 convs
    with ReLU and four 2x2 max pools, then 512-512-classes linear layers with
    ReLU between them."""

    def __init__(self, P, cid):
        self.seq, n = [], 0
        for v in VGG_PLAN:
            if v == "M":
                self.seq.append(("pool", Lyr.MaxPool2()))
            else:
                self.seq.append((f"conv{n}", Lyr.Conv2d(P[f"conv{n}.w"], P[f"conv{n}.b"])))
                self.seq.append(("relu", Lyr.ReLU()))
                n += 1
        self.fcs = [Lyr.Linear(P[f"fc{i}.w"], P[f"fc{i}.b"]) for i in range(3)]
        self.frelu = [Lyr.ReLU(), Lyr.ReLU()]

    def fwd(self, x, lengths=None):
        h = x
        for _, l in self.seq:
            h = l.fwd(h)
        h = h.reshape(h.shape[0], -1)
        for i in range(2):
            h = self.frelu[i].fwd(self.fcs[i].fwd(h))
        return self.fcs[2].fwd(h)

    def bwd(self, dz):
        G = {}
        dh = self.fcs[2].bwd(dz)
        for i in (1, 0):
            dh = self.fcs[i].bwd(self.frelu[i].bwd(dh))
        for i in range(3):
            G[f"fc{i}.w"], G[f"fc{i}.b"] = self.fcs[i].dw, self.fcs[i].db
        dh = dh.reshape(dh.shape[0], -1, 1, 1)  # the last pool leaves 1x1 maps
        for idx in range(len(self.seq) - 1, -1, -1):
            name, l = self.seq[idx]
            if name.startswith("conv"):
                dh = l.bwd(dh, need_dx=idx > 0)
                G[name + ".w"], G[name + ".b"] = l.dw, l.db
            else:
                dh = l.bwd(dh)
        self.G = G


class BasicBlock:
    """ReLU(BN(conv3x3(ReLU(BN(conv3x3_s(x))))) + shortcut(x)); shortcut is
    BN(conv1x1_s(x)) when the shape changes, else x.  Convs carry no bias."""

    def __init__(self, P, p, stride, down):
        self.c1 = Lyr.Conv2d(P[p + ".conv1.w"], None, stride=stride, pad=1)
        self.b1 = Lyr.BatchNorm2d(P[p + ".bn1.g"], P[p + ".bn1.b"])
        self.r1 = Lyr.ReLU()
        self.c2 = Lyr.Conv2d(P[p + ".conv2.w"], None, stride=1, pad=1)
        self.b2 = Lyr.BatchNorm2d(P[p + ".bn2.g"], P[p + ".bn2.b"])
        self.r2 = Lyr.ReLU()
        self.down = down
        if down:
            self.cd = Lyr.Conv2d(P[p + ".ds.w"], None, stride=stride, pad=0)
            self.bd = Lyr.BatchNorm2d(P[p + ".dsbn.g"], P[p + ".dsbn.b"])
        self.p = p

    def fwd(self, x):
        h = self.r1.fwd(self.b1.fwd(self.c1.fwd(x)))
        h = self.b2.fwd(self.c2.fwd(h))
        sc = self.bd.fwd(self.cd.fwd(x)) if self.down else x
        return self.r2.fwd(h + sc)

    def bwd(self, dy, need_dx, G):
        p = self.p
        ds = self.r2.bwd(dy)
        dh = self.b2.bwd(ds)
        dh = self.c2.bwd(dh)
        dh = self.b1.bwd(self.r1.bwd(dh))
        dx = self.c1.bwd(dh, need_dx=need_dx)
        G[p + ".conv1.w"], G[p + ".bn1.g"], G[p + ".bn1.b"] = self.c1.dw, self.b1.dg, self.b1.db
        G[p + ".conv2.w"], G[p + ".bn2.g"], G[p + ".bn2.b"] = self.c2.dw, self.b2.dg, self.b2.db
        if self.down:
            dsc = self.cd.bwd(self.bd.bwd(ds), need_dx=need_dx)
            G[p + ".ds.w"], G[p + ".dsbn.g"], G[p + ".dsbn.b"] = self.cd.dw, self.bd.dg, self.bd.db
        else:
            dsc = ds
        return dx + dsc if need_dx else None


class ResNet(_Net):
    """ResNet-18 stages 2-4 (two BasicBlocks each, the first with stride 2
    and a 1x1 projection shortcut), global average pool, linear 512->classes."""

    def __init__(self, P, cid):
        self.blocks = []
        for st, c, nb in RESNET_STAGES:
            for bi in range(nb):
                self.blocks.append(BasicBlock(P, f"layer{st}.{bi}", 2 if bi == 0 else 1, bi == 0))
        self.gap = Lyr.GlobalAvgPool()
        self.fc = Lyr.Linear(P["fc.w"], P["fc.b"])

    def fwd(self, x, lengths=None):
        h = x
        for b in self.blocks:
            h = b.fwd(h)
        return self.fc.fwd(self.gap.fwd(h))

    def bwd(self, dz):
        G = {}
        dh = self.gap.bwd(self.fc.bwd(dz))
        G["fc.w"], G["fc.b"] = self.fc.dw, self.fc.db
        for i in range(len(self.blocks) - 1, -1, -1):
            dh = self.blocks[i].bwd(dh, i > 0, G)
        self.G = G


class EncoderLayer:
    """Post-LN transformer encoder layer: h = LN1(x + MHA(x));
    y = LN2(h + W2 act(W1 h + b1) + b2), act = GELU (BERT) or ReLU (the
    paper's own transformers, as in the original encoder)."""

    def __init__(self, P, p, heads, act="gelu"):
        self.att = Lyr.MultiHeadAttention(P[p + ".qkv.w"], P[p + ".qkv.b"], P[p + ".o.w"], P[p + ".o.b"], heads)
        self.ln1 = Lyr.LayerNorm(P[p + ".ln1.g"], P[p + ".ln1.b"])
        self.f1 = Lyr.Linear(P[p + ".ffn1.w"], P[p + ".ffn1.b"])
        self.act = Lyr.GELU() if act == "gelu" else Lyr.ReLU()
        self.f2 = Lyr.Linear(P[p + ".ffn2.w"], P[p + ".ffn2.b"])
        self.ln2 = Lyr.LayerNorm(P[p + ".ln2.g"], P[p + ".ln2.b"])
        self.p = p

    def fwd(self, x, lengths):
        h = self.ln1.fwd(x + self.att.fwd(x, lengths))
        return self.ln2.fwd(h + self.f2.fwd(self.act.fwd(self.f1.fwd(h))))

    def bwd(self, dy, need_dx, G):
        p = self.p
        du = self.ln2.bwd(dy)
        dh = du + self.f1.bwd(self.act.bwd(self.f2.bwd(du)))
        dv = self.ln1.bwd(dh)
        dx = self.att.bwd(dv, need_dx)
        G[p + ".ln2.g"], G[p + ".ln2.b"] = self.ln2.dg, self.ln2.db
        G[p + ".ffn2.w"], G[p + ".ffn2.b"] = self.f2.dw, self.f2.db
        G[p + ".ffn1.w"], G[p + ".ffn1.b"] = self.f1.dw, self.f1.db
        G[p + ".ln1.g"], G[p + ".ln1.b"] = self.ln1.dg, self.ln1.db
        G[p + ".o.w"], G[p + ".o.b"] = self.att.out.dw, self.att.out.db
        G[p + ".qkv.w"], G[p + ".qkv.b"] = self.att.qkv.dw, self.att.qkv.db
        return dv + dx if need_dx else None


class Bert(_Net):
    """Encoder layers, then the pooler tanh(W_p h_0 + b_p) on the first token
    and a linear classifier."""

    def __init__(self, P, nlayers=None):
        n = BERT["layers"] if nlayers is None else nlayers
        self.layers = [EncoderLayer(P, f"enc{i}", BERT["heads"]) for i in range(n)]
        self.pool = Lyr.Linear(P["pool.w"], P["pool.b"])
        self.tanh = Lyr.Tanh()
        self.cls = Lyr.Linear(P["cls.w"], P["cls.b"])

    def fwd(self, x, lengths):
        h = x
        for l in self.layers:
            h = l.fwd(h, lengths)
        self.hshape = h.shape
        return self.cls.fwd(self.tanh.fwd(self.pool.fwd(h[:, 0, :])))

    def bwd(self, dz):
        G = {}
        dp = self.pool.bwd(self.tanh.bwd(self.cls.bwd(dz)))
        G["cls.w"], G["cls.b"] = self.cls.dw, self.cls.db
        G["pool.w"], G["pool.b"] = self.pool.dw, self.pool.db
        dh = np.zeros(self.hshape, dp.dtype)
        dh[:, 0, :] = dp
        for i in range(len(self.layers) - 1, -1, -1):
            dh = self.layers[i].bwd(dh, i > 0, G)
        self.G = G


class Bottleneck:
    """MobileNetV3 bottleneck: expansion 1x1 conv, BN, hard-swish; depthwise
    k x k conv (stride s), BN, hard-swish; squeeze-excitation (global mean,
    fc, ReLU, fc, hard-sigmoid, channel scale) when present; projection 1x1
    conv, BN; plus the input when the stride is 1 and the widths agree."""

    def __init__(self, P, p, k, e, ci, co, se, stride):
        self.p, self.se, self.res = p, se, stride == 1 and ci == co
        self.ex = Lyr.Conv2d(P[p + ".expand.w"], None, pad=0)
        self.bn1, self.a1 = Lyr.BatchNorm2d(P[p + ".bn1.g"], P[p + ".bn1.b"]), Lyr.HardSwish()
        self.dw = Lyr.DepthwiseConv2d(P[p + ".dw.w"], stride)
        self.bn2, self.a2 = Lyr.BatchNorm2d(P[p + ".bn2.g"], P[p + ".bn2.b"]), Lyr.HardSwish()
        if se:
            self.f1, self.r = Lyr.Linear(P[p + ".se.fc1.w"], P[p + ".se.fc1.b"]), Lyr.ReLU()
            self.f2, self.hs = Lyr.Linear(P[p + ".se.fc2.w"], P[p + ".se.fc2.b"]), Lyr.HardSigmoid()
        self.pr = Lyr.Conv2d(P[p + ".proj.w"], None, pad=0)
        self.bn3 = Lyr.BatchNorm2d(P[p + ".bn3.g"], P[p + ".bn3.b"])

    def fwd(self, x):
        h = self.a2.fwd(self.bn2.fwd(self.dw.fwd(self.a1.fwd(self.bn1.fwd(self.ex.fwd(x))))))
        if self.se:
            self.h = h
            self.s = self.hs.fwd(self.f2.fwd(self.r.fwd(self.f1.fwd(h.mean(axis=(2, 3))))))
            h = h * self.s[:, :, None, None]
        y = self.bn3.fwd(self.pr.fwd(h))
        return y + x if self.res else y

    def bwd(self, dy, need_dx, G):
        p = self.p
        dh = self.pr.bwd(self.bn3.bwd(dy))
        G[p + ".proj.w"], G[p + ".bn3.g"], G[p + ".bn3.b"] = self.pr.dw, self.bn3.dg, self.bn3.db
        if self.se:
            h, s = self.h, self.s
            ds = (dh * h).sum(axis=(2, 3))
            dm = self.f1.bwd(self.r.bwd(self.f2.bwd(self.hs.bwd(ds))))
            G[p + ".se.fc1.w"], G[p + ".se.fc1.b"] = self.f1.dw, self.f1.db
            G[p + ".se.fc2.w"], G[p + ".se.fc2.b"] = self.f2.dw, self.f2.db
            dh = dh * s[:, :, None, None] + dm[:, :, None, None] / (h.shape[2] * h.shape[3])
        dh = self.dw.bwd(self.bn2.bwd(self.a2.bwd(dh)))
        G[p + ".dw.w"], G[p + ".bn2.g"], G[p + ".bn2.b"] = self.dw.dw, self.bn2.dg, self.bn2.db
        dx = self.ex.bwd(self.bn1.bwd(self.a1.bwd(dh)), need_dx)
        G[p + ".expand.w"], G[p + ".bn1.g"], G[p + ".bn1.b"] = self.ex.dw, self.bn1.dg, self.bn1.db
        if not need_dx:
            return None
        return dx + dy if self.res else dx


class MBV3Server(_Net):
    """MobileNetV3-Large after its seventh bottleneck: eight bottlenecks, conv
    1x1 to 960 + BN + hard-swish, global mean, fc 1280 + hard-swish, fc X."""

    def __init__(self, P, cid):
        self.blocks, ci = [], IN_CH[cid]
        for j, (k, e, co, se, st) in enumerate(MBV3_TAIL):
            self.blocks.append(Bottleneck(P, f"b{j}", k, e, ci, co, se, st))
            ci = co
        self.last = Lyr.Conv2d(P["last.w"], None, pad=0)
        self.lbn, self.la = Lyr.BatchNorm2d(P["last_bn.g"], P["last_bn.b"]), Lyr.HardSwish()
        self.gap = Lyr.GlobalAvgPool()
        self.fc1, self.fa, self.fc2 = Lyr.Linear(P["fc1.w"], P["fc1.b"]), Lyr.HardSwish(), Lyr.Linear(P["fc2.w"], P["fc2.b"])

    def fwd(self, x, lengths=None):
        h = x
        for b in self.blocks:
            h = b.fwd(h)
        g = self.gap.fwd(self.la.fwd(self.lbn.fwd(self.last.fwd(h))))
        return self.fc2.fwd(self.fa.fwd(self.fc1.fwd(g)))

    def bwd(self, dz):
        G = {}
        dg = self.fc1.bwd(self.fa.bwd(self.fc2.bwd(dz)))
        G["fc2.w"], G["fc2.b"], G["fc1.w"], G["fc1.b"] = self.fc2.dw, self.fc2.db, self.fc1.dw, self.fc1.db
        dh = self.last.bwd(self.lbn.bwd(self.la.bwd(self.gap.bwd(dg))))
        G["last.w"], G["last_bn.g"], G["last_bn.b"] = self.last.dw, self.lbn.dg, self.lbn.db
        for i in range(len(self.blocks) - 1, -1, -1):
            dh = self.blocks[i].bwd(dh, i > 0, G)
        self.G = G


class VGG5Server(_Net):
    """conv3x3 (no bias) -> BN (train) -> ReLU -> maxpool 2x2 -> flatten (C, H, W)
    -> fc1 -> ReLU -> fc2."""

    def __init__(self, P):
        self.conv = Lyr.Conv2d(P["conv.w"], None)
        self.bn = Lyr.BatchNorm2d(P["bn.g"], P["bn.b"])
        self.r1, self.pool = Lyr.ReLU(), Lyr.MaxPool2()
        self.fc1, self.r2, self.fc2 = Lyr.Linear(P["fc1.w"], P["fc1.b"]), Lyr.ReLU(), Lyr.Linear(P["fc2.w"], P["fc2.b"])

    def fwd(self, x, lengths=None):
        p = self.pool.fwd(self.r1.fwd(self.bn.fwd(self.conv.fwd(x))))
        self.pshape = p.shape
        return self.fc2.fwd(self.r2.fwd(self.fc1.fwd(p.reshape(p.shape[0], -1))))

    def bwd(self, dz):
        dp = self.fc1.bwd(self.r2.bwd(self.fc2.bwd(dz))).reshape(self.pshape)
        self.conv.bwd(self.bn.bwd(self.r1.bwd(self.pool.bwd(dp))), need_dx=False)
        self.G = {"conv.w": self.conv.dw, "bn.g": self.bn.dg, "bn.b": self.bn.db,
                  "fc1.w": self.fc1.dw, "fc1.b": self.fc1.db, "fc2.w": self.fc2.dw, "fc2.b": self.fc2.db}


class SmallTransformer(_Net):
    """The server part of Transformer-6/12 (Table 4) split after EMB-100: the
    encoder layers (ReLU FFN) and FC-X on the first token."""

    def __init__(self, P, cid):
        a = TFSMALL[cid]
        self.layers = [EncoderLayer(P, f"enc{i}", a["heads"], act="relu") for i in range(a["layers"])]
        self.cls = Lyr.Linear(P["cls.w"], P["cls.b"])

    def fwd(self, x, lengths):
        h = x
        for l in self.layers:
            h = l.fwd(h, lengths)
        self.hshape = h.shape
        return self.cls.fwd(h[:, 0, :])

    def bwd(self, dz):
        G = {}
        d0 = self.cls.bwd(dz)
        G["cls.w"], G["cls.b"] = self.cls.dw, self.cls.db
        dh = np.zeros(self.hshape, d0.dtype)
        dh[:, 0, :] = d0
        for i in range(len(self.layers) - 1, -1, -1):
            dh = self.layers[i].bwd(dh, i > 0, G)
        self.G = G


def build(cid, P):
    fam = FAMILY[cid]
    if fam == "tfsmall":
        return SmallTransformer(P, cid)
    if fam == "vgg5":
        return VGG5Server(P)
    if fam == "mbv3":
        return MBV3Server(P, cid)
    if fam == "cnn":
        return CNN(P)
    if fam == "vgg_device":
        return DeviceVGG(P)
    if fam == "vgg":
        return VGG(P, cid)
    if fam == "resnet":
        return ResNet(P, cid)
    return Bert(P)


# ----------------------------------------------------------------------------- inputs
def decode_acts(acts, dt):
    """Activations as the devices sent them: fp32 arrays pass through;
    uint16 arrays are bf16 bit patterns, widened exactly (bits << 16)."""
    a = np.asarray(acts)
    if a.dtype == np.uint16:
        a = (a.astype(np.uint32) << np.uint32(16)).view(np.float32)
    return a.astype(dt)


# ----------------------------------------------------------------------------- training step
def sgd_update(params, grads, lr, momentum=0.0, mom_buf=None):
    """theta <- theta - lr * g (Alg. 4).  With momentum mu (config 3):
    v <- mu v + g (v starts at 0, so the first v is g), theta <- theta - lr v."""
    if momentum == 0.0:
        return params - lr * grads, None
    v = grads.copy() if mom_buf is None else momentum * mom_buf + grads
    return params - lr * v, v


def server_forward(cid, params_flat, acts, lengths=None, dt=np.float64):
    P = unpack(cid, params_flat, dt)
    net = build(cid, P)
    return net.fwd(decode_acts(acts, dt), lengths)


def server_step(cid, params_flat, acts, labels, lengths=None, lr=0.01, momentum=0.0,
                mom_buf=None, dt=np.float64):
    """One activation-branch iteration of Algorithm 4 on one batch.

    Returns a dict with the loss, the logits, the flat gradient, the updated
    flat parameters and (for momentum) the updated buffer, all in ``dt``."""
    P = unpack(cid, params_flat, dt)
    net = build(cid, P)
    z = net.fwd(decode_acts(acts, dt), lengths)
    loss, dz = Lyr.cross_entropy(z, np.asarray(labels))
    net.bwd(dz)
    g = pack(cid, net.grads()).astype(dt)
    theta = np.asarray(params_flat, dtype=dt)
    new, v = sgd_update(theta, g, lr, momentum, None if mom_buf is None else np.asarray(mom_buf, dt))
    return {"loss": loss, "logits": z, "grads": g, "params": new, "momentum": v}


def device_step(cid, params_flat, x, labels, lr=0.01, dt=np.float64):
    """One local training iteration of a device (Alg. 1): forward of the
    device network M_dk on the mini-batch, its output activations xi (what
    the device sends), forward of the auxiliary network on xi, the local loss
    f_d, backward through both networks and the SGD step with rate gamma_d on
    theta_dk and the auxiliary parameters.  Returns server_step's dict plus
    "acts" (xi, [B, 64, 16, 16])."""
    P = unpack(cid, params_flat, dt)
    net = build(cid, P)
    z = net.fwd(np.asarray(x, dtype=dt))
    loss, dz = Lyr.cross_entropy(z, np.asarray(labels))
    net.bwd(dz)
    g = pack(cid, net.grads()).astype(dt)
    new, _ = sgd_update(np.asarray(params_flat, dtype=dt), g, lr)
    return {"loss": loss, "logits": z, "grads": g, "params": new, "acts": net.xi}
