"""Workload descriptions for the server-side configurations (and the device side of one).

Each configuration is a split of a network between devices and the server:
the devices send the activations of their last layer, and the server trains
the remaining layers (the server-side network M_s of Sec. 3.1, trained in the
activation branch of Algorithm 4).  The shapes below stand in for the paper's
workloads (image classification on CIFAR-10 / Tiny ImageNet, sentiment
analysis on SST-2 / IMDB, Sec. 5.1); no dataset is read.

``param_layout`` fixes the order and shape of every server parameter inside
the flat fp32 vector exchanged with the library (the "library layout").
Convolution weights are stored as [Cout][kh][kw][Cin]; linear weights as
[out][in]; the fused attention input projection as [3*d][d] with the query,
key and value rows in that order.  Both the oracle and the HIP library derive
this order independently from the architecture; tests compare the three.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple


@dataclass(frozen=True)
class ConfigSpec:
    cid: int
    name: str
    family: str              # "cnn" (C1), "vgg" (C2, C5), "resnet" (C3), "bert" (C4), "vgg_device" (6),
                             # "tfsmall" (7, 8)
    batch: int
    in_shape: Tuple[int, ...]  # per-sample activation shape at the boundary (NCHW or [L, d])
    n_classes: int
    n_devices: int
    dtype: str               # "f32" or "bf16" (activations and GEMM operands)
    lr: float
    momentum: float          # 0.0 = plain SGD
    agg_n: int               # length of the flat device-side vector aggregated (0 = none)
    agg_alpha: float
    steps: int
    extra: dict = field(default_factory=dict)


CONFIGS = {
    1: ConfigSpec(1, "tiny-cnn-fp32", "cnn", 16, (32, 16, 16), 10, 4, "f32",
                  0.01, 0.0, 10_000, 0.5, 4),
    2: ConfigSpec(2, "vgg16-split-bf16", "vgg", 64, (64, 16, 16), 10, 16, "bf16",
                  0.01, 0.0, 0, 1.0, 100),
    3: ConfigSpec(3, "resnet18-split-bf16", "resnet", 32, (64, 16, 16), 100, 32, "bf16",
                  0.01, 0.9, 157_504, 1.0, 100, {"max_staleness": 8}),
    4: ConfigSpec(4, "bert-base-split-bf16", "bert", 32, (128, 768), 2, 16, "bf16",
                  0.01, 0.0, 0, 1.0, 100,
                  {"layers": 10, "heads": 12, "ffn": 3072, "min_len": 32}),
    5: ConfigSpec(5, "vgg16-split-128dev-bf16", "vgg", 64, (64, 16, 16), 10, 128, "bf16",
                  0.01, 0.0, 38_720, 1.0, 1000,
                  {"pool_bytes": 64 << 30, "bank": 256}),
    # The device side of the VGG-16 split of configurations 2 and 5 (Alg. 1):
    # device network conv1-2 of VGG-16 plus its auxiliary network, trained on
    # CIFAR-10-shaped 32x32 RGB inputs (fp32 at the boundary) against the local
    # loss; its output activations are the [64,16,16] batches the server trains on.
    6: ConfigSpec(6, "vgg16-device-side", "vgg_device", 64, (3, 32, 32), 10, 16, "f32",
                  0.01, 0.0, 0, 1.0, 100, {"server_config": 2}),
    # The paper's own transformers (Table 4), split after the embedding (the
    # split the pre-processor chooses for them): the server trains every
    # encoder layer (d = 100, FFN 100, ReLU, post-norm) and the classifier on the
    # first token, in fp32.  Transformer-6 (5 heads of width 20) on SST-2-shaped
    # batches of 64 tokens; Transformer-12 (50 heads of width 2) on IMDB-shaped
    # batches of 256 tokens.
    7: ConfigSpec(7, "transformer6-split-fp32", "tfsmall", 16, (64, 100), 2, 8, "f32",
                  0.01, 0.0, 0, 1.0, 100, {"layers": 6, "heads": 5, "ffn": 100, "min_len": 4}),
    8: ConfigSpec(8, "transformer12-split-fp32", "tfsmall", 16, (256, 100), 2, 16, "f32",
                  0.01, 0.0, 0, 1.0, 100, {"layers": 12, "heads": 50, "ffn": 100, "min_len": 16}),
    # The paper's VGG-5 (Table 4) on CIFAR-10, split after its second pool (the
    # split the pre-processor chooses for Raspberry-Pi-class devices): the server
    # trains conv3x3 64->64 with training-mode batch norm and ReLU, a 2x2 max
    # pool, fc 1024->128 with ReLU and fc 128->10, in fp32, on [64, 8, 8] inputs.
    9: ConfigSpec(9, "vgg5-split-fp32", "vgg5", 32, (64, 8, 8), 10, 8, "f32",
                  0.01, 0.0, 0, 1.0, 100),
    # The paper's MobileNetV3-Large (Table 4) on Tiny ImageNet (64x64, 200
    # classes), split after its seventh bottleneck (the split the pre-processor
    # chooses for Jetson-class devices): the server trains the last eight
    # bottlenecks (hard-swish, four with squeeze-excitation, one stride 2), the
    # 1x1 convolution to 960 channels, the global pool and fc 960-1280-200, in
    # fp32, on [80, 4, 4] inputs.
    10: ConfigSpec(10, "mobilenetv3l-split-fp32", "mbv3", 32, (80, 4, 4), 200, 16, "f32",
                   0.01, 0.0, 0, 1.0, 100),
}

# The server part of MobileNetV3-Large after its seventh bottleneck:
# (kernel, expansion, output channels, squeeze-excitation, stride)
MBV3_SERVER = [(3, 200, 80, False, 1), (3, 184, 80, False, 1), (3, 184, 80, False, 1), (3, 480, 112, True, 1),
               (3, 672, 112, True, 1), (5, 672, 160, True, 2), (5, 960, 160, True, 1), (5, 960, 160, True, 1)]


def squeeze_width(e: int) -> int:
    """The squeeze-excitation width of an expansion e: e / 4 rounded to a
    multiple of 8 (at least 8, never below 90% of e / 4)."""
    v = e // 4
    n = max(8, int(v + 4) // 8 * 8)
    return n + 8 if n < 0.9 * v else n


def get_config(cid: int) -> ConfigSpec:
    if cid not in CONFIGS:
        raise ValueError(f"unknown config {cid}")
    return CONFIGS[cid]


# (name, shape, init kind, fan_in). kinds: "kaiming" = U(+-sqrt(6/fan_in)), "zeros", "ones"
Entry = Tuple[str, Tuple[int, ...], str, int]

VGG_SERVER_CONVS = [128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512, "M"]


def _conv(name: str, cout: int, cin: int, k: int, bias: bool) -> List[Entry]:
    out = [(name + ".w", (cout, k, k, cin), "kaiming", cin * k * k)]
    if bias:
        out.append((name + ".b", (cout,), "zeros", 0))
    return out


def _linear(name: str, nout: int, nin: int) -> List[Entry]:
    return [(name + ".w", (nout, nin), "kaiming", nin), (name + ".b", (nout,), "zeros", 0)]


def _norm(name: str, c: int) -> List[Entry]:
    return [(name + ".g", (c,), "ones", 0), (name + ".b", (c,), "zeros", 0)]


def param_layout(cid: int) -> List[Entry]:
    cfg = get_config(cid)
    lay: List[Entry] = []
    if cfg.family == "cnn":
        lay += _conv("conv1", 64, 32, 3, True)
        lay += _conv("conv2", 64, 64, 3, True)
        lay += _linear("fc", 10, 64)
    elif cfg.family == "vgg":
        cin, i = cfg.in_shape[0], 0
        for v in VGG_SERVER_CONVS:
            if v == "M":
                continue
            lay += _conv(f"conv{i}", v, cin, 3, True)
            cin, i = v, i + 1
        lay += _linear("fc0", 512, 512)
        lay += _linear("fc1", 512, 512)
        lay += _linear("fc2", cfg.n_classes, 512)
    elif cfg.family == "resnet":
        cin = cfg.in_shape[0]
        for li, c in ((2, 128), (3, 256), (4, 512)):
            for bi in range(2):
                p = f"layer{li}.{bi}"
                lay += _conv(p + ".conv1", c, cin if bi == 0 else c, 3, False)
                lay += _norm(p + ".bn1", c)
                lay += _conv(p + ".conv2", c, c, 3, False)
                lay += _norm(p + ".bn2", c)
                if bi == 0:
                    lay += _conv(p + ".ds", c, cin, 1, False)
                    lay += _norm(p + ".dsbn", c)
            cin = c
        lay += _linear("fc", cfg.n_classes, 512)
    elif cfg.family == "mbv3":
        cin = cfg.in_shape[0]
        for j, (k, e, co, se, _) in enumerate(MBV3_SERVER):
            p = f"b{j}"
            lay += _conv(p + ".expand", e, cin, 1, False)
            lay += _norm(p + ".bn1", e)
            lay += [(p + ".dw.w", (e, k, k, 1), "kaiming", k * k)]
            lay += _norm(p + ".bn2", e)
            if se:
                s = squeeze_width(e)
                lay += _linear(p + ".se.fc1", s, e)
                lay += _linear(p + ".se.fc2", e, s)
            lay += _conv(p + ".proj", co, e, 1, False)
            lay += _norm(p + ".bn3", co)
            cin = co
        lay += _conv("last", 960, cin, 1, False)
        lay += _norm("last_bn", 960)
        lay += _linear("fc1", 1280, 960)
        lay += _linear("fc2", cfg.n_classes, 1280)
    elif cfg.family == "vgg5":
        lay += _conv("conv", 64, cfg.in_shape[0], 3, False)
        lay += _norm("bn", 64)
        lay += _linear("fc1", 128, 64 * 4 * 4)
        lay += _linear("fc2", cfg.n_classes, 128)
    elif cfg.family == "vgg_device":
        lay += _conv("conv1", 64, 3, 3, True)
        lay += _conv("conv2", 64, 64, 3, True)
        lay += _conv("aux.conv", 64, 64, 3, True)
        lay += _linear("aux.fc", cfg.n_classes, 64)
    elif cfg.family in ("bert", "tfsmall"):
        d, f = cfg.in_shape[1], cfg.extra["ffn"]
        for li in range(cfg.extra["layers"]):
            p = f"enc{li}"
            lay += _linear(p + ".qkv", 3 * d, d)
            lay += _linear(p + ".o", d, d)
            lay += _norm(p + ".ln1", d)
            lay += _linear(p + ".ffn1", f, d)
            lay += _linear(p + ".ffn2", d, f)
            lay += _norm(p + ".ln2", d)
        if cfg.family == "bert":
            lay += _linear("pool", d, d)
        lay += _linear("cls", cfg.n_classes, d)
    else:  # pragma: no cover
        raise ValueError(cfg.family)
    return lay


def param_count(cid: int) -> int:
    n = 0
    for _, shape, _, _ in param_layout(cid):
        k = 1
        for s in shape:
            k *= s
        n += k
    return n
