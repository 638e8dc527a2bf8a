"""Layer shapes of the YOLOv8m-class detector's Conv+BN+SiLU blocks.

Shapes only: no arithmetic of the method lives here.  The detector is the one
trained in the paper's case study (Sec. 6.1: CSP backbone, PAN-FPN neck,
decoupled head, SiLU, strides 8/16/32, 25.9M parameters), at YOLOv8m scale
(width 0.75, depth 0.67): channel widths 48/96/192/384/576, C2f repeats
2/4/4/2 in the backbone and 2 in the neck.

A C2f(c1 -> c2, n) block is: cv1 1x1 c1->c2, split into two c2/2 halves, n
bottlenecks of two 3x3 convs at c2/2 (residual in the backbone only), concat of
(2+n) halves, cv2 1x1 -> c2.  SPPF is cv1 1x1 C->C/2, three 5x5 max-pools,
concat 4*C/2, cv2 1x1 -> C.  All 3x3 convs use pad 1, all 1x1 convs pad 0.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional


@dataclass(frozen=True)
class ConvLayer:
    name: str
    ci: int
    co: int
    h: int  # input spatial size (square)
    k: int
    s: int

    @property
    def p(self) -> int:
        return self.k // 2

    @property
    def ho(self) -> int:
        return (self.h + 2 * self.p - self.k) // self.s + 1

    def gemm_flops(self, n: int) -> float:
        """2 * N*Ho*Wo * Co * Ci*kh*kw: one pass (fwd, dgrad and wgrad each cost this)."""
        return 2.0 * n * self.ho * self.ho * self.co * self.ci * self.k * self.k

    def params(self) -> int:
        return self.co * self.ci * self.k * self.k


def _c2f(prefix: str, c1: int, c2: int, n: int, h: int, out: List[ConvLayer]) -> None:
    half = c2 // 2
    out.append(ConvLayer(f"{prefix}.cv1", c1, c2, h, 1, 1))
    for i in range(n):
        out.append(ConvLayer(f"{prefix}.m{i}.cv1", half, half, h, 3, 1))
        out.append(ConvLayer(f"{prefix}.m{i}.cv2", half, half, h, 3, 1))
    out.append(ConvLayer(f"{prefix}.cv2", (2 + n) * half, c2, h, 1, 1))


def backbone_neck_layers() -> List[ConvLayer]:
    """The 65 Conv+BN+SiLU layers of the backbone and neck at a 640x640 input."""
    L: List[ConvLayer] = []
    L.append(ConvLayer("b0", 3, 48, 640, 3, 2))
    L.append(ConvLayer("b1", 48, 96, 320, 3, 2))
    _c2f("b2", 96, 96, 2, 160, L)
    L.append(ConvLayer("b3", 96, 192, 160, 3, 2))
    _c2f("b4", 192, 192, 4, 80, L)
    L.append(ConvLayer("b5", 192, 384, 80, 3, 2))
    _c2f("b6", 384, 384, 4, 40, L)
    L.append(ConvLayer("b7", 384, 576, 40, 3, 2))
    _c2f("b8", 576, 576, 2, 20, L)
    L.append(ConvLayer("b9.cv1", 576, 288, 20, 1, 1))  # SPPF
    L.append(ConvLayer("b9.cv2", 1152, 576, 20, 1, 1))
    _c2f("n12", 576 + 384, 384, 2, 40, L)  # upsampled b9 ++ b6
    _c2f("n15", 384 + 192, 192, 2, 80, L)  # upsampled n12 ++ b4
    L.append(ConvLayer("n16", 192, 192, 80, 3, 2))
    _c2f("n18", 192 + 384, 384, 2, 40, L)  # n16 ++ n12
    L.append(ConvLayer("n19", 384, 384, 40, 3, 2))
    _c2f("n21", 384 + 576, 576, 2, 20, L)  # n19 ++ b9
    return L


HEAD_SCALES = ((80, 192), (40, 384), (20, 576))  # (spatial, input channels) for strides 8/16/32


def literal_head_layers() -> List[ConvLayer]:
    """Detect head read literally: per scale, box C->64->64 and cls C->80->80, all 3x3 Conv+BN+SiLU."""
    L: List[ConvLayer] = []
    for h, c in HEAD_SCALES:
        L.append(ConvLayer(f"h{h}.box0", c, 64, h, 3, 1))
        L.append(ConvLayer(f"h{h}.box1", 64, 64, h, 3, 1))
        L.append(ConvLayer(f"h{h}.cls0", c, 80, h, 3, 1))
        L.append(ConvLayer(f"h{h}.cls1", 80, 80, h, 3, 1))
    return L


def faithful_head_param_tensors():
    """Architecture-faithful decoupled head (class hidden width 192): returns a list of
    (conv layer, has_bn, has_bias).  Used only to reproduce the paper's parameter counts."""
    out = []
    reg_hidden = max(16, HEAD_SCALES[0][1] // 4, 16 * 4)  # 64
    cls_hidden = max(HEAD_SCALES[0][1], min(80, 100))  # 192
    for h, c in HEAD_SCALES:
        out.append((ConvLayer(f"h{h}.box0", c, reg_hidden, h, 3, 1), True, False))
        out.append((ConvLayer(f"h{h}.box1", reg_hidden, reg_hidden, h, 3, 1), True, False))
        out.append((ConvLayer(f"h{h}.box2", reg_hidden, 64, h, 1, 1), False, True))
        out.append((ConvLayer(f"h{h}.cls0", c, cls_hidden, h, 3, 1), True, False))
        out.append((ConvLayer(f"h{h}.cls1", cls_hidden, cls_hidden, h, 3, 1), True, False))
        out.append((ConvLayer(f"h{h}.cls2", cls_hidden, 80, h, 1, 1), False, True))
    return out


@dataclass(frozen=True)
class Workload:
    index: int  # 1-based configuration number
    name: str
    n: int
    layers: List[ConvLayer] = field(default_factory=list)
    mode: str = "set"  # "set": independent layers; "chain": real dataflow
    x_dist: str = "normal"  # "normal" N(0,1) or "uniform01"
    g_std: float = 1.0
    eps: float = 1e-3

    def gemm_flops(self) -> float:
        """fwd + dgrad + wgrad FLOPs over all layers."""
        return 3.0 * sum(l.gemm_flops(self.n) for l in self.layers)


def workload(index: int, n: Optional[int] = None) -> Workload:
    """Configurations 1..5 (single block, stem, C2f at P3, backbone+neck, + literal head)."""
    if index == 1:
        return Workload(1, "single 3x3 block 16->32 @32x32", n or 2,
                        [ConvLayer("blk", 16, 32, 32, 3, 1)], mode="chain")
    if index == 2:
        return Workload(2, "stem 3->48 s2 @640, 48->96 s2 @320", n or 16,
                        [ConvLayer("b0", 3, 48, 640, 3, 2), ConvLayer("b1", 48, 96, 320, 3, 2)],
                        mode="chain", x_dist="uniform01")
    if index == 3:
        L: List[ConvLayer] = []
        _c2f("c2f", 192, 192, 2, 80, L)
        return Workload(3, "C2f 192->192 n=2 residual @80x80", n or 16, L, mode="chain")
    if index == 4:
        return Workload(4, "YOLOv8m backbone+neck conv set", n or 16, backbone_neck_layers())
    if index == 5:
        return Workload(5, "YOLOv8m backbone+neck+literal head conv set", n or 32,
                        backbone_neck_layers() + literal_head_layers(), g_std=0.1)
    raise ValueError(f"no configuration {index}")
