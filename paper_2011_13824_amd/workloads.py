"""Seeded synthetic workloads: networks, input boxes, specifications and split masks.

This module only draws random numbers and lays out shapes.  It performs none of the bound
computation, so the GPU path and the CPU oracle can both take their inputs from it.

The paper evaluates on CIFAR-10 properties of three robustly trained convolutional networks
(Base, Wide and Deep, App. B) which are not available here.  The stand-ins below take those
networks' shapes exactly and use He-initialised random weights:

* ``tiny``  -- FC 4-32-32-2, x0 ~ U[0,1]^4, eps = 0.1, spec e0 - e1, 64 sub-domains with
  0-6 splits each (a small correctness case).
* ``base``  -- Conv(3->8,k4,s2,p1), Conv(8->16,k4,s2,p1), FC 1024->100, FC 100->10;
  x0 ~ U[0,1]^{3x32x32}, eps = 2/255, 9 margin specs, 400 sub-domains, 0-10 splits.
* ``wide``  -- Conv(3->16), Conv(16->32) (k4,s2,p1), FC 2048->100, FC 100->10; 1024
  sub-domains, 0-16 splits.
* ``deep``  -- Conv(3->8,k4,s2,p1), 2x Conv(8->8,k3,s1,p1), Conv(8->8,k4,s2,p1), FC 512->100,
  FC 100->10; 1024 sub-domains, 0-16 splits.
* ``wide_opt`` -- the ``wide`` network and box with 2048 sub-domains and 20 Adam steps on alpha.

Weights are N(0, 2/fan_in) (fan_in = C_in*k*k for a convolution), biases N(0, 0.1^2), all fp32.
Margin specifications are the rows e_y - e_j, j != y, in increasing j (the margin property of
App. B, Eq. 10); the synthetic image has no true class, so y is drawn from the seed.  Split
masks hold -1 (h < 0 enforced), 0 (free) or +1 (h >= 0 enforced) per ReLU neuron, the ReLU
layers concatenated in layer order; the split neurons of a sub-domain are drawn without
replacement from a caller-supplied candidate set (normally the neurons that are unstable at
the root, as branch and bound only splits unstable neurons) with equiprobable directions.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

FC, CONV = 0, 1


def fc(n_in: int, n_out: int) -> dict:
    return dict(kind=FC, in_c=n_in, in_h=1, in_w=1, out_c=n_out, out_h=1, out_w=1,
                k=0, stride=1, pad=0)


def conv(in_c: int, in_hw: int, out_c: int, k: int, stride: int, pad: int) -> dict:
    out_hw = (in_hw + 2 * pad - k) // stride + 1
    return dict(kind=CONV, in_c=in_c, in_h=in_hw, in_w=in_hw, out_c=out_c, out_h=out_hw,
                out_w=out_hw, k=k, stride=stride, pad=pad)


ARCHS = {
    "tiny": [fc(4, 32), fc(32, 32), fc(32, 2)],
    "base": [conv(3, 32, 8, 4, 2, 1), conv(8, 16, 16, 4, 2, 1), fc(1024, 100), fc(100, 10)],
    "wide": [conv(3, 32, 16, 4, 2, 1), conv(16, 16, 32, 4, 2, 1), fc(2048, 100), fc(100, 10)],
    "deep": [conv(3, 32, 8, 4, 2, 1), conv(8, 16, 8, 3, 1, 1), conv(8, 16, 8, 3, 1, 1),
             conv(8, 16, 8, 4, 2, 1), fc(512, 100), fc(100, 10)],
}


def n_in(layer: dict) -> int:
    return layer["in_c"] * layer["in_h"] * layer["in_w"]


def n_out(layer: dict) -> int:
    return layer["out_c"] * layer["out_h"] * layer["out_w"]


def relu_sizes(layers: list[dict]) -> list[int]:
    """Sizes of the ReLU layers (every layer but the last)."""
    return [n_out(t) for t in layers[:-1]]


def num_relu(layers: list[dict]) -> int:
    return int(sum(relu_sizes(layers)))


def weight_shape(layer: dict) -> tuple:
    if layer["kind"] == FC:
        return (layer["out_c"], layer["in_c"])
    return (layer["out_c"], layer["in_c"], layer["k"], layer["k"])


def make_layers(arch: list[dict], seed: int) -> list[dict]:
    """He-initialised fp32 weights and N(0, 0.1^2) biases, drawn layer by layer."""
    rng = np.random.default_rng(seed)
    layers = []
    for spec in arch:
        shape = weight_shape(spec)
        fan_in = int(np.prod(shape[1:]))
        W = rng.normal(0.0, np.sqrt(2.0 / fan_in), size=shape).astype(np.float32)
        b = rng.normal(0.0, 0.1, size=spec["out_c"]).astype(np.float32)
        layers.append(dict(spec, W=np.ascontiguousarray(W), b=b))
    return layers


def margin_spec(n_classes: int, y: int) -> np.ndarray:
    """Rows e_y - e_j for every j != y, increasing j."""
    rows = []
    for j in range(n_classes):
        if j == y:
            continue
        c = np.zeros(n_classes, dtype=np.float32)
        c[y], c[j] = 1.0, -1.0
        rows.append(c)
    return np.stack(rows)


def make_splits(B: int, n_relu: int, max_splits: int, seed: int,
                candidates: np.ndarray | None = None) -> np.ndarray:
    """int8 [B, n_relu] masks; sub-domain b splits k_b ~ U{0..max_splits} distinct candidates."""
    rng = np.random.default_rng([seed, 0x5_9117])
    cand = np.arange(n_relu) if candidates is None else np.asarray(candidates, dtype=np.int64)
    split = np.zeros((B, n_relu), dtype=np.int8)
    for b in range(B):
        k = int(rng.integers(0, max_splits + 1))
        k = min(k, cand.size)
        if k == 0:
            continue
        idx = rng.choice(cand, size=k, replace=False)
        split[b, idx] = rng.choice(np.array([-1, 1], dtype=np.int8), size=k)
    return split


@dataclass
class Workload:
    name: str
    layers: list
    x0: np.ndarray
    eps: float
    C: np.ndarray
    B: int
    max_splits: int
    mask_seed: int
    steps: int = 0
    lr: float = 0.1
    extra: dict = field(default_factory=dict)

    @property
    def S(self) -> int:
        return self.C.shape[0]

    @property
    def n_relu(self) -> int:
        return num_relu(self.layers)

    def splits(self, candidates: np.ndarray | None = None, B: int | None = None) -> np.ndarray:
        return make_splits(self.B if B is None else B, self.n_relu, self.max_splits,
                           self.mask_seed, candidates)


EPS_CIFAR = float(np.float32(2.0 / 255.0))


def _image_workload(name, arch, seed, B, max_splits, mask_seed, steps=0):
    layers = make_layers(ARCHS[arch], seed)
    rng = np.random.default_rng([seed, 0x1_3A6E])
    x0 = rng.uniform(0.0, 1.0, size=n_in(layers[0])).astype(np.float32)
    y = int(rng.integers(0, layers[-1]["out_c"]))
    C = margin_spec(layers[-1]["out_c"], y)
    return Workload(name, layers, x0, EPS_CIFAR, C, B, max_splits, mask_seed, steps=steps,
                    extra=dict(label=y, arch=arch))


def tiny() -> Workload:
    layers = make_layers(ARCHS["tiny"], 0)
    rng = np.random.default_rng([0, 0x1_3A6E])
    x0 = rng.uniform(0.0, 1.0, size=4).astype(np.float32)
    C = np.array([[1.0, -1.0]], dtype=np.float32)
    return Workload("tiny", layers, x0, float(np.float32(0.1)), C, 64, 6, 0,
                    extra=dict(arch="tiny"))


def base() -> Workload:
    return _image_workload("base", "base", 1, 400, 10, 1)


def wide() -> Workload:
    return _image_workload("wide", "wide", 2, 1024, 16, 2)


def deep() -> Workload:
    return _image_workload("deep", "deep", 3, 1024, 16, 3)


def wide_opt() -> Workload:
    return _image_workload("wide_opt", "wide", 2, 2048, 16, 4, steps=20)


WORKLOADS = dict(tiny=tiny, base=base, wide=wide, deep=deep, wide_opt=wide_opt)


def get(name: str) -> Workload:
    return WORKLOADS[name]()


def random_net(arch: list[dict], seed: int) -> list[dict]:
    """Random network of any shape (small test cases)."""
    return make_layers(arch, seed)
