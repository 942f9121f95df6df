"""The five synthetic workloads of the reconcile path and their tensor layouts.

Shapes stand in for the models the paper trains (ResNet-50 on CIFAR-100 and
TinyImageNet, ViT-S on CIFAR-100; Sec. 5.2); no weights or datasets are used.
The flat parameter buffer packs each model's parameter tensors in network
order; the layout only fixes P and the tensor boundaries (which the parity
tests sample), every coordinate is drawn from the same distribution.
"""
from __future__ import annotations

from dataclasses import dataclass, field


def resnet50_tensors(num_classes: int) -> list[tuple[str, int]]:
    """Parameter tensors of ResNet-50 (7x7 stem, bottleneck layers 3/4/6/3 of
    widths 64/128/256/512 with 4x expansion, a 1x1 projection shortcut in the
    first block of every stage, BatchNorm weight+bias after every conv, and a
    2048 x num_classes classifier), in network order."""
    out = [("conv1.weight", 64 * 3 * 7 * 7), ("bn1.weight", 64), ("bn1.bias", 64)]
    inplanes = 64
    for stage, (blocks, planes) in enumerate(zip((3, 4, 6, 3), (64, 128, 256, 512)), 1):
        for b in range(blocks):
            pre = f"layer{stage}.{b}."
            out += [(pre + "conv1.weight", planes * inplanes),
                    (pre + "bn1.weight", planes), (pre + "bn1.bias", planes),
                    (pre + "conv2.weight", planes * planes * 9),
                    (pre + "bn2.weight", planes), (pre + "bn2.bias", planes),
                    (pre + "conv3.weight", planes * 4 * planes),
                    (pre + "bn3.weight", planes * 4), (pre + "bn3.bias", planes * 4)]
            if b == 0:
                out += [(pre + "downsample.0.weight", planes * 4 * inplanes),
                        (pre + "downsample.1.weight", planes * 4),
                        (pre + "downsample.1.bias", planes * 4)]
            inplanes = planes * 4
    out += [("fc.weight", 2048 * num_classes), ("fc.bias", num_classes)]
    return out


def vit_s_tensors(num_classes: int = 100, depth: int = 12,
                  dim: int = 384) -> list[tuple[str, int]]:
    """Transformer-block and head tensors of ViT-S (dim 384, MLP ratio 4)."""
    out = []
    for b in range(depth):
        pre = f"blocks.{b}."
        out += [(pre + "norm1.weight", dim), (pre + "norm1.bias", dim),
                (pre + "attn.qkv.weight", dim * 3 * dim), (pre + "attn.qkv.bias", 3 * dim),
                (pre + "attn.proj.weight", dim * dim), (pre + "attn.proj.bias", dim),
                (pre + "norm2.weight", dim), (pre + "norm2.bias", dim),
                (pre + "mlp.fc1.weight", dim * 4 * dim), (pre + "mlp.fc1.bias", 4 * dim),
                (pre + "mlp.fc2.weight", 4 * dim * dim), (pre + "mlp.fc2.bias", dim)]
    out += [("head.weight", dim * num_classes), ("head.bias", num_classes)]
    return out


def round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


@dataclass(frozen=True)
class Workload:
    name: str
    W: int
    P: int
    K: int
    lr: float
    mu: float
    beta: float
    alpha: float
    periods: int
    param_dt: str = "f32"          # "f32" or "bf16"
    grad_dt: str = "f32"           # gradient storage, "f32" or "bf16"
    mom_dt: str = "f32"            # momentum storage, "f32" or "bf16"
    theta_sigma: float = 0.02
    grad_sigma: float = 1e-3
    outlier_rate: float = 0.0
    outlier_scale: float = 100.0
    tensors: tuple = field(default=(), repr=False)
    row_align_bytes: int = 1 << 20  # replica rows rounded up to a multiple of this

    @property
    def ld(self) -> int:
        return round_up(self.P, self.row_align_bytes // self.param_bytes())

    @property
    def steps(self) -> int:
        return self.periods * self.K

    def boundaries(self) -> list[int]:
        """Start offset of every tensor in the flat buffer."""
        offs, o = [], 0
        for _, n in self.tensors:
            offs.append(o)
            o += n
        return offs

    def param_bytes(self) -> int:
        return 2 if self.param_dt == "bf16" else 4

    def grad_bytes(self) -> int:
        return 2 if self.grad_dt == "bf16" else 4

    def mom_bytes(self) -> int:
        return 2 if self.mom_dt == "bf16" else 4

    def _replica_bytes(self, adamw: bool) -> int:
        """Per replica-coordinate bytes every step moves: the gradient read,
        the optimizer state read and written (momentum, plus AdamW's fp32
        second moment), the parameter read and written."""
        return (self.grad_bytes() + 2 * self.mom_bytes() + (8 if adamw else 0)
                + 2 * self.param_bytes())

    def reconcile_bytes(self, adamw: bool = False) -> int:
        """Algorithmic HBM bytes of one reconcile: every state tensor read
        once, every updated one written once, plus u and anchor read and
        written (optimizer state, u and anchor are fp32)."""
        return self.P * (self.W * self._replica_bytes(adamw) + 16)

    def sync_bytes(self, method: str = "cpdp", adamw: bool = False) -> int:
        """Algorithmic HBM bytes of one synchronisation step of a strategy:
        cpdp = the reconcile; localsgd = the per-replica traffic plus the
        averaged model written once; ddp = the per-replica traffic only."""
        if method == "cpdp":
            return self.reconcile_bytes(adamw)
        if method == "localsgd":
            return self.P * (self.W * self._replica_bytes(adamw) + 4)
        if method == "ddp":
            return self.local_step_bytes(adamw)
        raise ValueError(method)

    def local_step_bytes(self, adamw: bool = False) -> int:
        return self.P * self.W * self._replica_bytes(adamw)


def _make() -> dict[str, Workload]:
    r100 = tuple(resnet50_tensors(100))
    r200 = tuple(resnet50_tensors(200))
    vit = tuple(vit_s_tensors(100))
    n = lambda t: sum(s for _, s in t)  # noqa: E731
    return {
        "tiny": Workload("tiny", W=4, P=262_144, K=2, lr=0.1, mu=0.9, beta=0.5,
                         alpha=1.0, periods=10, tensors=(("flat", 262_144),)),
        "r50_100": Workload("r50_100", W=8, P=n(r100), K=4, lr=0.1, mu=0.9,
                            beta=0.5, alpha=1.0, periods=5, tensors=r100),
        "vit_s": Workload("vit_s", W=8, P=n(vit), K=4, lr=0.05, mu=0.9,
                          beta=0.7, alpha=1.0, periods=5, tensors=vit),
        "r50_200": Workload("r50_200", W=16, P=n(r200), K=8, lr=0.1, mu=0.9,
                            beta=0.6, alpha=1.0, periods=4, outlier_rate=0.01,
                            tensors=r200),
        "stress": Workload("stress", W=32, P=100_000_000, K=4, lr=0.1, mu=0.9,
                           beta=0.5, alpha=1.0, periods=3, param_dt="bf16",
                           tensors=(("flat", 100_000_000),)),
    }


WORKLOADS = _make()
