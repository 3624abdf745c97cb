"""Conv2d task tables and tuning configurations.

The paper tunes every conv2d operator of a model as its own task (section 4,
evaluation set-up: ResNet-18 gives 12 such tasks, and its skip-connection
1x1 convolutions are the light operators 2, 5, 8 and 11 in Fig. 5). The paper
lists counts, not shapes; the tables below are the standard ImageNet
architectures at 224x224 input:

* ResNet-18 (batch 1): 12 distinct conv shapes, with a 1x1 projection at the
  first unit of every stage (four projections, task positions 2, 5, 8, 11
  counted from 0).
* ResNet-50 (batch 1): the 22 distinct bottleneck 1x1/3x3 shapes, stride on
  the 3x3 convolution, stem excluded.
* MobileNet-v2 (batch 16): 10 distinct depthwise 3x3 shapes (fp32, NCHW)
  and 19 distinct pointwise 1x1 shapes (bf16 NHWC, fp32 output).

Each configuration fixes the task list, data recipe, candidate count, CU
fractions and measurement protocol so that runs are comparable.
"""
from __future__ import annotations

from dataclasses import dataclass, field, asdict
from typing import List, Tuple

DT_F32 = 0
DT_BF16 = 1
LAYOUT_NCHW = 0
LAYOUT_NHWC = 1

FAM_DIRECT_F32 = 1
FAM_DEPTHWISE_F32 = 2
FAM_IGEMM_BF16 = 3
FAM_IGEMM_F32 = 4
FAMILY_NAMES = {1: "direct_f32", 2: "depthwise_f32", 3: "igemm_mfma_bf16", 4: "igemm_mfma_f32"}
# knob index of the reduction split per family (depthwise has none)
SPLIT_KNOB = {1: 7, 3: 7, 4: 9}


def split_of(s) -> int:
    """How many ways schedule s splits its reduction (1: not split)."""
    i = SPLIT_KNOB.get(int(s.family))
    return 1 if i is None else int(s.knob[i])


@dataclass(frozen=True)
class Op:
    """One conv2d task: shapes, precision and layout (fields mirror ``ct_op``)."""
    name: str
    n: int
    c: int
    h: int
    w: int
    k: int
    r: int
    s: int
    stride_h: int = 1
    stride_w: int = 1
    pad_h: int = 0
    pad_w: int = 0
    dil_h: int = 1
    dil_w: int = 1
    groups: int = 1
    dtype: int = DT_F32
    layout: int = LAYOUT_NCHW

    @property
    def oh(self) -> int:
        return max((self.h + 2 * self.pad_h - self.dil_h * (self.r - 1) - 1) // self.stride_h + 1, 0)

    @property
    def ow(self) -> int:
        return max((self.w + 2 * self.pad_w - self.dil_w * (self.s - 1) - 1) // self.stride_w + 1, 0)

    @property
    def cg(self) -> int:
        return self.c // self.groups

    def x_shape(self) -> Tuple[int, ...]:
        if self.layout == LAYOUT_NCHW:
            return (self.n, self.c, self.h, self.w)
        return (self.n, self.h, self.w, self.c)

    def w_shape(self) -> Tuple[int, ...]:
        if self.layout == LAYOUT_NCHW:
            return (self.k, self.cg, self.r, self.s)
        return (self.k, self.r, self.s, self.cg)

    def y_shape(self) -> Tuple[int, ...]:
        if self.layout == LAYOUT_NCHW:
            return (self.n, self.k, self.oh, self.ow)
        return (self.n, self.oh, self.ow, self.k)

    def flops(self) -> int:
        """2 * N * K * OH * OW * Cg * R * S (padded taps counted)."""
        return 2 * self.n * self.k * self.oh * self.ow * self.cg * self.r * self.s

    def bytes_moved(self) -> int:
        """Compulsory HBM bytes: x and w read once, y (always fp32) written once."""
        el = 2 if self.dtype == DT_BF16 else 4
        nx = self.n * self.c * self.h * self.w
        nw = self.k * self.cg * self.r * self.s
        ny = self.n * self.k * self.oh * self.ow
        return el * (nx + nw) + 4 * ny

    def families(self) -> Tuple[int, ...]:
        """Kernel families whose layout/precision contract fits this task."""
        if self.dtype == DT_BF16:
            if (self.layout == LAYOUT_NHWC and self.r == 1 and self.s == 1 and self.groups == 1
                    and self.pad_h == 0 and self.pad_w == 0):
                return (FAM_IGEMM_BF16,)
            return ()
        if self.layout != LAYOUT_NCHW:
            return ()
        if self.groups == 1:
            return (FAM_DIRECT_F32, FAM_IGEMM_F32)
        if self.groups == self.c and self.k == self.c:
            return (FAM_DEPTHWISE_F32,)
        return ()

    def as_tuple(self) -> Tuple[int, ...]:
        return (self.n, self.c, self.h, self.w, self.k, self.r, self.s, self.stride_h,
                self.stride_w, self.pad_h, self.pad_w, self.dil_h, self.dil_w, self.groups,
                self.dtype, self.layout)


def conv(name, n, c, h, k, rs, stride=1, pad=None, groups=1, dtype=DT_F32, layout=LAYOUT_NCHW):
    pad = rs // 2 if pad is None else pad
    return Op(name, n, c, h, h, k, rs, rs, stride, stride, pad, pad, 1, 1, groups, dtype, layout)


def resnet18(n: int = 1) -> List[Op]:
    return [
        conv("r18.1", n, 3, 224, 64, 7, 2, 3),
        conv("r18.2", n, 64, 56, 64, 3, 1),
        conv("r18.3", n, 64, 56, 64, 1, 1),
        conv("r18.4", n, 64, 56, 128, 3, 2),
        conv("r18.5", n, 128, 28, 128, 3, 1),
        conv("r18.6", n, 64, 56, 128, 1, 2),
        conv("r18.7", n, 128, 28, 256, 3, 2),
        conv("r18.8", n, 256, 14, 256, 3, 1),
        conv("r18.9", n, 128, 28, 256, 1, 2),
        conv("r18.10", n, 256, 14, 512, 3, 2),
        conv("r18.11", n, 512, 7, 512, 3, 1),
        conv("r18.12", n, 256, 14, 512, 1, 2),
    ]


def resnet50(n: int = 1) -> List[Op]:
    spec = [  # (C, H, K, RS, stride)
        (64, 56, 64, 1, 1), (64, 56, 64, 3, 1), (64, 56, 256, 1, 1), (256, 56, 64, 1, 1),
        (256, 56, 128, 1, 1), (128, 56, 128, 3, 2), (128, 28, 512, 1, 1), (256, 56, 512, 1, 2),
        (512, 28, 128, 1, 1), (128, 28, 128, 3, 1), (512, 28, 256, 1, 1), (256, 28, 256, 3, 2),
        (256, 14, 1024, 1, 1), (512, 28, 1024, 1, 2), (1024, 14, 256, 1, 1), (256, 14, 256, 3, 1),
        (1024, 14, 512, 1, 1), (512, 14, 512, 3, 2), (512, 7, 2048, 1, 1), (1024, 14, 2048, 1, 2),
        (2048, 7, 512, 1, 1), (512, 7, 512, 3, 1),
    ]
    return [conv("r50.%d" % (i + 1), n, c, h, k, rs, s) for i, (c, h, k, rs, s) in enumerate(spec)]


# How many convolutions of the network have each distinct shape (ResNet-18
# under the four-projection reading: 21 convolutions; ResNet-50 bottlenecks,
# stem excluded: 52). Used to weigh per-layer latencies into a model total.
MULTIPLICITY = {
    "r18.1": 1, "r18.2": 4, "r18.3": 1, "r18.4": 1, "r18.5": 3, "r18.6": 1,
    "r18.7": 1, "r18.8": 3, "r18.9": 1, "r18.10": 1, "r18.11": 3, "r18.12": 1,
    **{"r50.%d" % (i + 1): m for i, m in enumerate(
        [1, 3, 4, 2, 1, 1, 4, 1, 3, 3, 1, 1, 6, 1, 5, 5, 1, 1, 3, 1, 2, 2])},
}


def multiplicity(name: str) -> int:
    """Occurrences of a layer shape in its network (1 if not tabulated)."""
    return MULTIPLICITY.get(name, 1)


def mobilenet_v2_depthwise(n: int = 16) -> List[Op]:
    spec = [(32, 112, 1), (96, 112, 2), (144, 56, 1), (144, 56, 2), (192, 28, 1), (192, 28, 2),
            (384, 14, 1), (576, 14, 1), (576, 14, 2), (960, 7, 1)]
    return [conv("dw%d" % (i + 1), n, c, h, c, 3, s, 1, groups=c) for i, (c, h, s) in enumerate(spec)]


def mobilenet_v2_pointwise(n: int = 16) -> List[Op]:
    spec = [(32, 16, 112), (16, 96, 112), (96, 24, 56), (24, 144, 56), (144, 24, 56), (144, 32, 28),
            (32, 192, 28), (192, 32, 28), (192, 64, 14), (64, 384, 14), (384, 64, 14), (384, 96, 14),
            (96, 576, 14), (576, 96, 14), (576, 160, 7), (160, 960, 7), (960, 160, 7), (960, 320, 7),
            (320, 1280, 7)]
    return [conv("pw%d" % (i + 1), n, c, h, k, 1, 1, 0, dtype=DT_BF16, layout=LAYOUT_NHWC)
            for i, (c, k, h) in enumerate(spec)]


@dataclass(frozen=True)
class Protocol:
    """Timing protocol: warm-up launches, repeats, launches per repeat (one event pair each)."""
    warmup: int = 2
    repeats: int = 5
    launches: int = 10
    timeout_ms: float = 1000.0


@dataclass
class TuneConfig:
    config_id: int
    name: str
    ops: List[Op]
    n_candidates: int
    fractions: Tuple[float, ...]
    dist: str = "uniform"
    seed: int = 0
    clients: int = 1
    top_t: int = 8
    eps: float = 0.01
    stage1: Protocol = field(default_factory=Protocol)
    stage2: Protocol = field(default_factory=lambda: Protocol(2, 21, 10))

    def describe(self) -> dict:
        d = asdict(self)
        d["ops"] = [o.name for o in self.ops]
        return d


def config(config_id: int) -> TuneConfig:
    """The five workload configurations, by number (1-5)."""
    if config_id == 1:
        return TuneConfig(1, "single conv 64->64 3x3 56x56 fp32", [conv("c1", 1, 64, 56, 64, 3, 1)],
                          64, (1.0,))
    if config_id == 2:
        return TuneConfig(2, "ResNet-18 b1 conv set fp32", resnet18(1), 256, (0.25, 0.5, 1.0))
    if config_id == 3:
        return TuneConfig(3, "ResNet-18 cross-evaluation fp32", resnet18(1), 256,
                          (0.125, 0.25, 0.5, 0.75, 1.0), dist="normal")
    if config_id == 4:
        return TuneConfig(4, "ResNet-50 b1 bottleneck convs, 4 clients at 25% against 1 client at 100%",
                          resnet50(1), 512, (0.25, 1.0), clients=4)
    if config_id == 5:
        return TuneConfig(5, "MobileNet-v2 b16 dw fp32 + pw bf16",
                          mobilenet_v2_depthwise(16) + mobilenet_v2_pointwise(16), 1024, (0.5, 1.0))
    raise ValueError("configs are numbered 1-5")
