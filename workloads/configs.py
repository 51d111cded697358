"""Layer shapes and sparsity settings of the synthetic workloads.

Weight tensors follow the paper's notation (Section 3): a CONV layer holds
W in R^{A x B x C x D} -- A filters, B channels per filter (per conv group),
C x D kernel taps.  The shapes below are those of the networks the paper
evaluates on (AlexNet/CaffeNet conv1-5 in Tables 1-2, ResNet-50 in Table 3)
plus a CIFAR-sized layer; only their shapes are used, never trained values.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

# Constraint-set kinds of Section 3 (filter-, channel-, filter-shape-wise and
# non-structured sparsity).  The integer values are the C-ABI enum values.
FILTER, CHANNEL, SHAPE, ELEMENT = 0, 1, 2, 3
KIND_NAMES = {FILTER: "filter", CHANNEL: "channel", SHAPE: "shape", ELEMENT: "element"}


@dataclass(frozen=True)
class ConvLayer:
    """One CONV layer: weight [A, B, C, D], conv groups, input spatial size."""
    name: str
    A: int
    B: int
    C: int
    D: int
    H: int
    W: int
    stride: int = 1
    pad: int = 0
    groups: int = 1

    @property
    def n(self) -> int:
        return self.A * self.B * self.C * self.D

    @property
    def K(self) -> int:
        """Columns of the GEMM weight matrix [A, B*C*D] (Section 3)."""
        return self.B * self.C * self.D

    @property
    def in_channels(self) -> int:
        return self.groups * self.B

    @property
    def P(self) -> int:
        return (self.H + 2 * self.pad - self.C) // self.stride + 1

    @property
    def Q(self) -> int:
        return (self.W + 2 * self.pad - self.D) // self.stride + 1

    def n_groups(self, kind: int) -> int:
        if kind == FILTER:
            return self.A
        if kind == CHANNEL:
            return self.B
        if kind == SHAPE:
            return self.K
        if kind == ELEMENT:
            return self.n
        raise ValueError(f"unknown kind {kind}")

    def dense_flops(self, batch: int) -> int:
        return 2 * batch * self.P * self.Q * self.A * self.K


def kept_count(percent: float, n_groups: int) -> int:
    """Kept-group count from a percentage: floor((p*G + 50) / 100), i.e.
    round half up, evaluated in integers (p is given in whole percent)."""
    p = int(round(percent))
    if abs(p - percent) > 1e-12:
        raise ValueError("percent must be a whole number")
    return (p * n_groups + 50) // 100


def alexnet_layers() -> List[ConvLayer]:
    """AlexNet/CaffeNet conv1-5 (227x227 input; conv2, conv4, conv5 have two groups)."""
    return [
        ConvLayer("conv1", 96, 3, 11, 11, 227, 227, stride=4, pad=0, groups=1),
        ConvLayer("conv2", 256, 48, 5, 5, 27, 27, stride=1, pad=2, groups=2),
        ConvLayer("conv3", 384, 256, 3, 3, 13, 13, stride=1, pad=1, groups=1),
        ConvLayer("conv4", 384, 192, 3, 3, 13, 13, stride=1, pad=1, groups=2),
        ConvLayer("conv5", 256, 192, 3, 3, 13, 13, stride=1, pad=1, groups=2),
    ]


def resnet50_layers() -> List[ConvLayer]:
    """All 53 convolutions of ResNet-50 v1.5 (stride on the 3x3 of each
    stage's first block) at 224x224 input."""
    L: List[ConvLayer] = [ConvLayer("conv1", 64, 3, 7, 7, 224, 224, stride=2, pad=3)]
    cin, hw = 64, 56  # after the stem's 3x3/2 max-pool
    for si, (w, blocks) in enumerate([(64, 3), (128, 4), (256, 6), (512, 3)]):
        for bi in range(blocks):
            s = 2 if (bi == 0 and si > 0) else 1
            pre = f"layer{si + 1}.{bi}"
            L.append(ConvLayer(f"{pre}.conv1", w, cin, 1, 1, hw, hw))
            L.append(ConvLayer(f"{pre}.conv2", w, w, 3, 3, hw, hw, stride=s, pad=1))
            hw_out = (hw + 2 - 3) // s + 1
            L.append(ConvLayer(f"{pre}.conv3", 4 * w, w, 1, 1, hw_out, hw_out))
            if bi == 0:
                L.append(ConvLayer(f"{pre}.downsample", 4 * w, cin, 1, 1, hw, hw, stride=s))
            cin, hw = 4 * w, hw_out
    return L


@dataclass(frozen=True)
class Workload:
    """A set of layers with weight laws and a sparsity setting.

    ``variants`` lists (kind, percent) pairs; each layer is projected with
    every variant.  ``chain`` marks the filter+channel chain in which layer
    L's input-channel support is layer L-1's kept-filter mask.
    ``w_sigma`` of None means He initialisation, sigma^2 = 2 / fan_in.
    """
    name: str
    wid: int
    batch: int
    layers: Tuple[ConvLayer, ...]
    variants: Tuple[Tuple[int, int], ...]
    w_sigma: Optional[float]
    u_sigma: float
    rho: float
    chain: bool = False
    explicit_k: Optional[Tuple[int, ...]] = None
    description: str = ""
    extra_percents: Tuple[int, ...] = field(default_factory=tuple)

    def sigma_w(self, layer: ConvLayer) -> float:
        if self.w_sigma is not None:
            return self.w_sigma
        return (2.0 / layer.K) ** 0.5

    def k_for(self, li: int, kind: int, percent: int) -> int:
        if self.explicit_k is not None:
            return self.explicit_k[li]
        return kept_count(percent, self.layers[li].n_groups(kind))


WORKLOADS = {
    "cifar_conv64": Workload(
        "cifar_conv64", 1, 8,
        (ConvLayer("conv", 64, 64, 3, 3, 32, 32, stride=1, pad=1),),
        ((FILTER, 50),), w_sigma=0.05, u_sigma=0.0, rho=1e-3, explicit_k=(32,),
        description="CIFAR-style 3x3 conv [64,64,3,3] on [8,64,32,32], filter-wise keep 32"),
    "alexnet_shape30": Workload(
        "alexnet_shape30", 2, 128, tuple(alexnet_layers()),
        ((SHAPE, 30),), w_sigma=0.01, u_sigma=1e-4, rho=1.5e-3,
        description="AlexNet conv1-5, batch 128, filter-shape-wise keep 30% of (c,kh,kw) columns"),
    "alexnet_chain_f50c50": Workload(
        "alexnet_chain_f50c50", 3, 128, tuple(alexnet_layers()),
        ((FILTER, 50),), w_sigma=0.01, u_sigma=1e-4, rho=1.5e-3, chain=True,
        description="AlexNet conv1-5, batch 128, filter-wise keep 50% with each layer's input "
                    "channels restricted to the previous layer's kept filters"),
    "resnet50_filter60": Workload(
        "resnet50_filter60", 4, 64, tuple(resnet50_layers()),
        ((FILTER, 60),), w_sigma=None, u_sigma=0.0, rho=1.5e-3,
        description="ResNet-50 v1.5, all 53 convs, 224x224, batch 64, filter-wise keep 60%"),
    "resnet50_s3_sweep": Workload(
        "resnet50_s3_sweep", 5, 256,
        (ConvLayer("layer3.conv2", 256, 256, 3, 3, 14, 14, stride=1, pad=1),),
        tuple((k, p) for k in (FILTER, SHAPE, ELEMENT) for p in (10, 25, 50)),
        w_sigma=None, u_sigma=0.0, rho=1.5e-3, extra_percents=(75, 90),
        description="ResNet-50 stage-3 3x3 conv [256,256,3,3] on 14x14, batch 256: element-wise "
                    "vs filter/shape-wise at 10/25/50% density"),
}


# Per-layer row (filter) and column (filter-shape) sparsity, in percent, of the
# pruned AlexNet models whose batch-1 CONV speedups Tables 1 and 2 report
# (Table 1: column pruning at 0% accuracy loss; Table 2: row and column pruning
# at 0.7% and 2.0% loss, with the same row sparsities in both).  Only these
# counts are taken; the masks are drawn by projecting synthetic weights.
PAPER_TABLE_SPARSITY = {
    "table1": {"conv1": (0.0, 0.0), "conv2": (0.0, 70.0), "conv3": (0.0, 77.0), "conv4": (0.0, 85.0),
               "conv5": (0.0, 81.0)},
    "table2_loss0.7": {"conv1": (9.4, 0.0), "conv2": (12.9, 63.9), "conv3": (40.6, 78.1), "conv4": (46.9, 87.0),
                       "conv5": (0.0, 84.9)},
    "table2_loss2.0": {"conv1": (9.4, 0.0), "conv2": (12.9, 87.5), "conv3": (40.6, 90.0), "conv4": (46.9, 90.5),
                       "conv5": (0.0, 90.7)},
}


# Per-layer non-structured (element-wise) sparsity, in percent, of the pruned
# AlexNet CONV layers of Table 4 (no accuracy loss: 16.1x on conv2-5) and of
# Table 5's 1.95%-loss row (40.5x on conv2-5), whose GPU speed Section 5
# discusses.  conv1 is left dense in both.
PAPER_ELEMENT_SPARSITY = {
    "table4_16.1x": {"conv1": 0.0, "conv2": 93.0, "conv3": 94.3, "conv4": 93.6, "conv5": 93.5},
    "table5_40.5x": {"conv1": 0.0, "conv2": 97.0, "conv3": 98.0, "conv4": 97.5, "conv5": 97.0},
}


def kept_from_sparsity(sparsity_percent: float, n_groups: int) -> int:
    """Groups kept when sparsity_percent of n_groups are pruned (pruned count
    rounded half up)."""
    pruned = int(sparsity_percent * n_groups / 100.0 + 0.5)
    return n_groups - pruned


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]
