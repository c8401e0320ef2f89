"""Flat-buffer parameter layouts for the CNN shapes the AGS step is run on.

A model's parameter tensors are laid end to end in one fp32 buffer (weights
``w`` and momentum ``m`` share the layout; each gradient replica uses it too).
Each tensor becomes one *layer* ``[offset, offset + numel)`` of that buffer,
and every offset is rounded up to ``PAD_ELEMS`` elements so that vector loads
of 16 bytes never straddle two layers.  The AGS state (``gradscale``) and the
segmented statistics are kept per layer, i.e. per parameter tensor, which is
how the per-parameter scale of the Adaptive Gradient Scaling algorithm
(Algorithm 1, ``UpdateGradScale``) is read here.

Only shapes live here: this module holds no part of the method's arithmetic.
The tensor lists follow the public architecture definitions (ResNet: He et
al. 2016; VGG: Simonyan & Zisserman 2015), in the order a PyTorch module
lists its parameters.  The paper evaluates its method on CNNs of these
families (Sec. IV-B, experimental setup).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np

#: Layer offsets are multiples of this many elements (64 fp32 = 256 bytes).
PAD_ELEMS = 64

#: Bit flags of a layer, identical in value to the C-ABI's flags.
LAYER_SCALE = 1  # the layer takes part in AGS / LARS scaling
LAYER_DECAY = 2  # the layer receives weight decay


@dataclass(frozen=True)
class Tensor:
    name: str
    shape: Tuple[int, ...]
    kind: str        # "conv", "fc", "bias", "bn_weight", "bn_bias"
    fan_in: int      # fan-in of the owning conv / fc (for init), 0 for BN

    @property
    def numel(self) -> int:
        return int(np.prod(self.shape))


@dataclass
class Layout:
    """A flat layout: tensors, their offsets and per-layer flags."""
    name: str
    tensors: List[Tensor]
    offsets: np.ndarray            # int64 [L]
    numels: np.ndarray             # int64 [L]
    flags: np.ndarray              # uint32 [L]
    n_flat: int                    # padded length of the flat buffer
    meta: dict = field(default_factory=dict)

    @property
    def n_layers(self) -> int:
        return len(self.tensors)

    @property
    def n_params(self) -> int:
        return int(self.numels.sum())

    def table(self):
        """(offset, numel, flags) per layer, as the C-ABI's layer table wants."""
        return [(int(o), int(n), int(f)) for o, n, f in
                zip(self.offsets, self.numels, self.flags)]


def round_up(x: int, a: int) -> int:
    return (x + a - 1) // a * a


#: Gap, in elements, left between consecutive replica rows of a gradient
#: stack.  The K replica streams of a step are read at the same offset at the
#: same time; staggering their start addresses spreads them over more HBM
#: channels (measured on MI355X: 2.5% faster ResNet-50 K=16 steps, no change
#: for the fp32 layouts).
REPLICA_GAP = 2048


def replica_stride(layout: "Layout") -> int:
    """Row stride (elements) of a [K, stride] replica-gradient stack."""
    return round_up(layout.n_flat, 8) + REPLICA_GAP


def _flags_for(t: Tensor, policy: str) -> int:
    if policy == "all":
        return LAYER_SCALE | LAYER_DECAY
    if policy == "exclude_1d":
        # One-dimensional tensors (biases, BN gamma/beta) are neither scaled
        # nor decayed.
        return 0 if len(t.shape) == 1 else (LAYER_SCALE | LAYER_DECAY)
    raise ValueError(f"unknown flag policy {policy!r}")


def make_layout(name: str, tensors: List[Tensor], policy: str,
                pad: int = PAD_ELEMS) -> Layout:
    offs, nums, flg = [], [], []
    pos = 0
    for t in tensors:
        pos = round_up(pos, pad)
        offs.append(pos)
        nums.append(t.numel)
        flg.append(_flags_for(t, policy))
        pos += t.numel
    n_flat = round_up(pos, pad)
    return Layout(name, tensors, np.array(offs, np.int64),
                  np.array(nums, np.int64), np.array(flg, np.uint32), n_flat,
                  meta={"policy": policy, "pad": pad})


# --------------------------------------------------------------------------
# architectures


def _conv(name, cin, cout, k, bias):
    out = [Tensor(name + ".weight", (cout, cin, k, k), "conv", cin * k * k)]
    if bias:
        out.append(Tensor(name + ".bias", (cout,), "bias", cin * k * k))
    return out


def _fc(name, fin, fout):
    return [Tensor(name + ".weight", (fout, fin), "fc", fin),
            Tensor(name + ".bias", (fout,), "bias", fin)]


def _bn(name, c):
    return [Tensor(name + ".weight", (c,), "bn_weight", 0),
            Tensor(name + ".bias", (c,), "bn_bias", 0)]


def tiny_cnn_tensors() -> List[Tensor]:
    """conv3x3 3->16, 16->32, 32->64 and fc 64->10, each with a bias."""
    t = []
    t += _conv("conv1", 3, 16, 3, True)
    t += _conv("conv2", 16, 32, 3, True)
    t += _conv("conv3", 32, 64, 3, True)
    t += _fc("fc", 64, 10)
    return t


def resnet18_cifar_tensors(num_classes: int = 10) -> List[Tensor]:
    """ResNet-18 for 32x32 inputs: 3x3 stem, four stages of two basic blocks,
    1x1 projection shortcuts where the shape changes, fc 512->classes."""
    t = []
    t += _conv("conv1", 3, 64, 3, False)
    t += _bn("bn1", 64)
    cin = 64
    for si, (cout, stride) in enumerate([(64, 1), (128, 2), (256, 2), (512, 2)]):
        for bi in range(2):
            s = stride if bi == 0 else 1
            p = f"layer{si + 1}.{bi}"
            t += _conv(p + ".conv1", cin, cout, 3, False)
            t += _bn(p + ".bn1", cout)
            t += _conv(p + ".conv2", cout, cout, 3, False)
            t += _bn(p + ".bn2", cout)
            if s != 1 or cin != cout:
                t += _conv(p + ".shortcut.0", cin, cout, 1, False)
                t += _bn(p + ".shortcut.1", cout)
            cin = cout
    t += _fc("linear", 512, num_classes)
    return t


def resnet50_tensors(num_classes: int = 1000) -> List[Tensor]:
    """ResNet-50 for ImageNet: 7x7 stem, bottleneck stages [3, 4, 6, 3],
    1x1 projection on the first block of every stage, fc 2048->classes."""
    t = []
    t += _conv("conv1", 3, 64, 7, False)
    t += _bn("bn1", 64)
    cin = 64
    for si, (width, blocks) in enumerate([(64, 3), (128, 4), (256, 6), (512, 3)]):
        cout = width * 4
        for bi in range(blocks):
            p = f"layer{si + 1}.{bi}"
            t += _conv(p + ".conv1", cin, width, 1, False)
            t += _bn(p + ".bn1", width)
            t += _conv(p + ".conv2", width, width, 3, False)
            t += _bn(p + ".bn2", width)
            t += _conv(p + ".conv3", width, cout, 1, False)
            t += _bn(p + ".bn3", cout)
            if bi == 0:
                t += _conv(p + ".downsample.0", cin, cout, 1, False)
                t += _bn(p + ".downsample.1", cout)
            cin = cout
    t += _fc("fc", 2048, num_classes)
    return t


def vgg16_tensors(num_classes: int = 1000) -> List[Tensor]:
    """VGG-16 (configuration D) without batch norm, 224x224 inputs."""
    cfg = [64, 64, "M", 128, 128, "M", 256, 256, 256, "M",
           512, 512, 512, "M", 512, 512, 512, "M"]
    t = []
    cin, i = 3, 0
    for v in cfg:
        if v == "M":
            i += 1
            continue
        t += _conv(f"features.{i}", cin, v, 3, True)
        cin = v
        i += 2
    t += _fc("classifier.0", 512 * 7 * 7, 4096)
    t += _fc("classifier.3", 4096, 4096)
    t += _fc("classifier.6", 4096, num_classes)
    return t


#: Named layouts.  ``policy`` says which layers are scaled and decayed.
LAYOUTS = {
    "tiny_cnn": (tiny_cnn_tensors, "all"),
    "resnet18_cifar": (resnet18_cifar_tensors, "exclude_1d"),
    "resnet50": (resnet50_tensors, "exclude_1d"),
    "vgg16": (vgg16_tensors, "exclude_1d"),
}


def get_layout(name: str, policy: str | None = None) -> Layout:
    fn, default_policy = LAYOUTS[name]
    return make_layout(name, fn(), policy or default_policy)


def custom_layout(numels, flags=None, pad: int = 8, name: str = "custom") -> Layout:
    """A layout from a plain list of layer sizes (tests and edge cases).

    ``flags`` defaults to scale+decay on every layer; ``pad`` is the offset
    alignment in elements (the C-ABI requires a multiple of 8).
    """
    numels = [int(n) for n in numels]
    if flags is None:
        flags = [LAYER_SCALE | LAYER_DECAY] * len(numels)
    tensors = [Tensor(f"t{i}", (n,), "fc", max(n, 1)) for i, n in enumerate(numels)]
    offs, pos = [], 0
    for n in numels:
        pos = round_up(pos, pad)
        offs.append(pos)
        pos += n
    return Layout(name, tensors, np.array(offs, np.int64),
                  np.array(numels, np.int64), np.array(flags, np.uint32),
                  round_up(max(pos, 1), pad), meta={"policy": "custom", "pad": pad})
