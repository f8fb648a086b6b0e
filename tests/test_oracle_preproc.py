"""Pins of the pre-processor oracle (Sec. 3.2.1, Eq. 6-8; auxiliary network
of Sec. 3.2.2): every unit's forward FLOPs and parameter count against torch
modules written independently here (FLOPs counted by torch's own FLOP
counter), MobileNetV3-Large's published parameter count, a hand-derived
split, properties of the argmin-max rule, and the auxiliary network that the
VGG-16 split of the server workloads yields (config 6's)."""
import os

import numpy as np
import pytest
import torch
import torch.nn as nn
import torch.nn.functional as F
from torch.utils.flop_counter import FlopCounterMode

import fo_synth as S
from oracle import preproc as P
from tests.golden_io import GOLDEN


def _flops(mod, x):
    with FlopCounterMode(display=False) as fc:
        with torch.no_grad():
            y = mod(x)
    return fc.get_total_flops(), y


def _nparams(mod):
    return sum(p.numel() for p in mod.parameters())


class _SE(nn.Module):
    def __init__(self, e, s):
        super().__init__()
        self.a, self.b = nn.Conv2d(e, s, 1), nn.Conv2d(s, e, 1)

    def forward(self, x):
        return x * F.hardsigmoid(self.b(F.relu(self.a(F.adaptive_avg_pool2d(x, 1)))))


class _Bneck(nn.Module):
    def __init__(self, k, e, ci, co, se, s):
        super().__init__()
        layers = []
        if e != ci:
            layers += [nn.Conv2d(ci, e, 1, bias=False), nn.BatchNorm2d(e), nn.Hardswish()]
        layers += [nn.Conv2d(e, e, k, s, k // 2, groups=e, bias=False), nn.BatchNorm2d(e), nn.Hardswish()]
        if se:
            layers.append(_SE(e, P._div8(e // 4)))
        layers += [nn.Conv2d(e, co, 1, bias=False), nn.BatchNorm2d(co)]
        self.body = nn.Sequential(*layers)
        self.res = s == 1 and ci == co

    def forward(self, x):
        y = self.body(x)
        return x + y if self.res else y


class _Enc(nn.Module):
    def __init__(self, d, heads, hidden):
        super().__init__()
        self.h = heads
        self.qkv, self.o = nn.Linear(d, 3 * d), nn.Linear(d, d)
        self.f1, self.f2 = nn.Linear(d, hidden), nn.Linear(hidden, d)
        self.n1, self.n2 = nn.LayerNorm(d), nn.LayerNorm(d)

    def forward(self, x):
        B, L, d = x.shape
        q, k, v = (t.reshape(B, L, self.h, d // self.h).transpose(1, 2) for t in self.qkv(x).split(d, -1))
        a = torch.softmax(q @ k.transpose(-1, -2) / (d // self.h) ** 0.5, -1) @ v
        x = self.n1(x + self.o(a.transpose(1, 2).reshape(B, L, d)))
        return self.n2(x + self.f2(F.gelu(self.f1(x))))


def _torch_units(net, classes, hw):
    """The same networks as torch modules, unit by unit, with their inputs."""
    units = []
    if net in ("vgg5", "vgg16"):
        plan = ((32, "M", 64, "M", 64, "M") if net == "vgg5" else
                (64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512, "M"))
        c, h = 3, hw
        for v in plan:
            if v == "M":
                units.append((nn.MaxPool2d(2), (c, h, h)))
                h //= 2
            else:
                bn = [nn.BatchNorm2d(v)] if net == "vgg5" else []
                units.append((nn.Sequential(nn.Conv2d(c, v, 3, 1, 1, bias=net != "vgg5"), *bn, nn.ReLU()), (c, h, h)))
                c = v
        widths = (128,) if net == "vgg5" else (512, 512)
        n_in = c * h * h
        for wd in widths + (classes,):
            units.append((nn.Linear(n_in, wd), (n_in,)))
            n_in = wd
    elif net == "mobilenetv3_large":
        units.append((nn.Sequential(nn.Conv2d(3, 16, 3, 2, 1, bias=False), nn.BatchNorm2d(16), nn.Hardswish()),
                      (3, hw, hw)))
        c, h = 16, (hw + 1) // 2
        for k, e, o, se, s in P.MBV3_LARGE:
            units.append((_Bneck(k, e, c, o, se, s), (c, h, h)))
            c, h = o, (h + 2 * (k // 2) - k) // s + 1
        units.append((nn.Sequential(nn.Conv2d(c, 960, 1, bias=False), nn.BatchNorm2d(960), nn.Hardswish()),
                      (c, h, h)))
        units.append((nn.AdaptiveAvgPool2d(1), (960, h, h)))
        units.append((nn.Linear(960, 1280), (960,)))
        units.append((nn.Linear(1280, classes), (1280,)))
    else:
        n, heads = (6, 5) if net == "transformer6" else (12, 50)
        units.append((nn.Identity(), (hw, 100)))  # the embedding lookup: no FLOPs
        for _ in range(n):
            units.append((_Enc(100, heads, 100), (hw, 100)))
        units.append((nn.Linear(100, classes), (100,)))
    return units


@pytest.mark.parametrize("net,classes,hw", [("vgg5", 10, 32), ("vgg16", 10, 32), ("mobilenetv3_large", 200, 64),
                                            ("transformer6", 2, 64), ("transformer12", 2, 32)])
def test_unit_tables_match_torch_modules(net, classes, hw):
    ours = P.net_layers(net, classes, hw)
    ref = _torch_units(net, classes, hw)
    assert len(ours) == len(ref)
    for i, (u, (mod, shape)) in enumerate(zip(ours, ref)):
        mod.eval()
        fl, y = _flops(mod, torch.zeros((1,) + shape))
        assert u["fwd_flops"] == fl, (net, i, u["fwd_flops"], fl)
        assert u["params"] == _nparams(mod), (net, i)
        assert u["out_elems"] == y.numel(), (net, i)


def test_mobilenetv3_large_published_parameter_count():
    """5,483,032 parameters at 1000 classes: the count of the architecture's
    reference implementation (its paper quotes 5.4M)."""
    assert sum(u["params"] for u in P.net_layers("mobilenetv3_large", 1000, 224)) == 5_483_032


def _golden_split():
    units, devs, costs, split = [], [], None, None
    for line in open(os.path.join(GOLDEN, "split_k2.txt")):
        t = line.split()
        if not t or t[0].startswith("#"):
            continue
        kv = {a.split("=")[0]: float(a.split("=")[1]) for a in t[1:] if "=" in a}
        if t[0] == "unit":
            units.append(P._layer(P.FC, flops=kv["f"], out=kv["s"]))
        elif t[0] == "device":
            devs.append((kv["o"], kv["b"]))
        elif t[0] == "costs":
            costs = [float(v) for v in t[1:]]
        elif t[0] == "split":
            split = int(t[1])
    return units, devs, costs, split


def test_golden_split():
    units, devs, costs, split = _golden_split()
    l, c = P.select_split(units, 1, 1, [d[0] for d in devs], [d[1] for d in devs])
    assert c == costs and l == split


def test_split_rule_properties():
    rng = np.random.default_rng(3)
    L = P.net_layers("vgg16", 10, 32)
    for _ in range(50):
        K = int(rng.integers(1, 9))
        o = list(rng.uniform(1e9, 1e12, K))
        b = list(rng.uniform(1e6, 1e9, K))
        l, c = P.select_split(L, 16, 4, o, b)
        # brute force over every split and device
        brute = []
        for j in range(len(L)):
            Osum = sum(3.0 * u["fwd_flops"] * 16 for u in L[:j + 1])
            S = L[j]["out_elems"] * 16 * 4
            brute.append(max(max(Osum / ok, S / bk) for ok, bk in zip(o, b)))
        assert np.allclose(c, brute, rtol=1e-12) and c[l - 1] == min(c) and l == c.index(min(c)) + 1
        # the device order does not matter
        perm = rng.permutation(K)
        assert P.select_split(L, 16, 4, [o[i] for i in perm], [b[i] for i in perm])[0] == l
    # unlimited bandwidth: the least training work wins (the first unit);
    # unlimited compute: the smallest output wins
    assert P.select_split(L, 16, 4, [1e12], [1e300])[0] == 1
    l, _ = P.select_split(L, 16, 4, [1e300], [1e6])
    outs = [u["out_elems"] for u in L]
    assert outs[l - 1] == min(outs) and l == outs.index(min(outs)) + 1


def test_aux_network_of_the_vgg16_split_is_config_6s():
    """Splitting VGG-16 after its first block (conv 64, conv 64, pool: the
    server workloads' split) gives the auxiliary network of config 6:
    conv3x3 64->64 with bias, global average pool, fc 64->10."""
    L = P.net_layers("vgg16", 10, 32)
    aux = P.aux_network(L, 3, 10)
    assert [u["kind"] for u in aux] == [P.CONV, P.POOL, P.FC]
    assert (aux[0]["k"], aux[0]["c_in"], aux[0]["c_out"], aux[0]["h_out"]) == (3, 64, 64, 16)
    lay = {name: int(np.prod(shape)) for name, shape, _, _ in S.param_layout(6)}
    assert sum(u["params"] for u in aux) == lay["aux.conv.w"] + lay["aux.conv.b"] + lay["aux.fc.w"] + lay["aux.fc.b"]
    device = sum(u["params"] for u in L[:3])
    assert device + sum(u["params"] for u in aux) == S.param_count(6)


@pytest.mark.parametrize("net,l,kinds", [("mobilenetv3_large", 5, [P.BNECK, P.POOL, P.FC]),
                                         ("transformer6", 3, [P.ENC, P.FC]), ("transformer6", 1, [P.FC]),
                                         ("vgg5", 7, [P.FC, P.FC])])
def test_aux_network_kinds(net, l, kinds):
    L = P.net_layers(net, 10, 32)
    aux = P.aux_network(L, l, 10)
    assert [u["kind"] for u in aux] == kinds
    assert aux[-1]["c_out"] == 10
