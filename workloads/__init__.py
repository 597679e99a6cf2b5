"""Seeded synthetic workloads: parameter-tree shapes and random arrays.

This module serves both sides of every parity check (the HIP path and the CPU
oracle) and the benchmark.  It holds no arithmetic of the method: it only
draws numbers and describes shapes.

The five trees follow the paper's workloads by shape only (MAML-style
networks, ResNet parameter trees of Appendix D, Table 2, and two synthetic
stress shapes); no dataset or trained weight is involved.

Value recipe (all fp32, seeded):
  params       p0 ~ N(0, 0.05^2)
  gradients    g_k ~ N(0, sigma_g^2), sigma_g per workload
  moments      zero (fresh inner loop, count0 = 0), or |N(0, (1e-4)^2)| with
               count0 = 100 for the flat 1B case
  cotangents   ~ N(0, 1) (the outer-loss gradient on p_K; interior-step
               cotangents of m and v for the flat 1B case)
N(0, s^2) names the standard deviation s.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Sequence, Tuple

import numpy as np

BASE_SEED = 20221112  # the paper's arXiv identifier date; any fixed value works

HYPER = dict(lr=1e-3, b1=0.9, b2=0.999, eps=1e-8)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    description: str
    shapes: Tuple[Tuple[int, ...], ...]
    K: int
    grad_std: float
    eps_root: float
    count0: int
    nonzero_moments: bool
    interior_cotangents: bool
    tasks: int = 1

    @property
    def numels(self) -> List[int]:
        return [int(np.prod(s, dtype=np.int64)) if len(s) else 1 for s in self.shapes]

    @property
    def n(self) -> int:
        return int(sum(self.numels))

    @property
    def nseg(self) -> int:
        return len(self.shapes)


def tiny_mlp_shapes() -> List[Tuple[int, ...]]:
    """1 -> 40 -> 40 -> 1 MLP: [40x1, 40, 40x40, 40, 1x40, 1] = 1,761 params."""
    return [(40, 1), (40,), (40, 40), (40,), (1, 40), (1,)]


def convnet_shapes(in_ch: int = 1, width: int = 64, ways: int = 5) -> List[Tuple[int, ...]]:
    """Four [conv3x3 + bias, BN scale, BN shift] blocks, then a linear head:
    18 tensors, 112,261 params for a 1-channel input and a 5-way head."""
    shapes: List[Tuple[int, ...]] = []
    c = in_ch
    for _ in range(4):
        shapes += [(width, c, 3, 3), (width,), (width,), (width,)]
        c = width
    shapes += [(ways, width), (ways,)]
    return shapes


def resnet18_shapes(classes: int = 1000) -> List[Tuple[int, ...]]:
    """Trainable tensors of ResNet-18 (convs without bias, BN weight/bias, fc):
    62 tensors, 11,689,512 params.  Running BN statistics are buffers, not
    parameters, and are not part of the tree."""
    shapes: List[Tuple[int, ...]] = [(64, 3, 7, 7), (64,), (64,)]
    cin = 64
    for cout, stride in ((64, 1), (128, 2), (256, 2), (512, 2)):
        for blk in range(2):
            s = stride if blk == 0 else 1
            shapes += [(cout, cin, 3, 3), (cout,), (cout,), (cout, cout, 3, 3), (cout,), (cout,)]
            if s != 1 or cin != cout:
                shapes += [(cout, cin, 1, 1), (cout,), (cout,)]
            cin = cout
    shapes += [(classes, 512), (classes,)]
    return shapes


def many_small_sizes(count: int = 20000, max_size: int = 65536, seed: int = 0) -> List[int]:
    """Sizes log-uniform on [1, max_size]: exp(U(0, ln max_size)) rounded to the
    nearest integer and clipped to [1, max_size]."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([BASE_SEED, 4, seed])))
    x = np.exp(rng.uniform(0.0, math.log(max_size), size=count))
    return [int(v) for v in np.clip(np.rint(x), 1, max_size).astype(np.int64)]


def _mk(name, desc, shapes, **kw) -> Workload:
    return Workload(name=name, description=desc, shapes=tuple(tuple(s) for s in shapes), **kw)


def tiny_mlp() -> Workload:
    return _mk("tiny_mlp", "tiny MLP tree, 6 tensors, 1,761 fp32 params, K=5",
               tiny_mlp_shapes(), K=5, grad_std=0.01, eps_root=0.0, count0=0,
               nonzero_moments=False, interior_cotangents=False)


def convnet32() -> Workload:
    one = convnet_shapes()
    return _mk("convnet32", "conv-net tree x 32 task copies, 576 tensors, 3,592,352 fp32 params, K=5",
               one * 32, K=5, grad_std=0.01, eps_root=0.0, count0=0,
               nonzero_moments=False, interior_cotangents=False, tasks=32)


def resnet18(K: int = 10) -> Workload:
    return _mk("resnet18_k%d" % K,
               "ResNet-18 parameter tree, 62 tensors, 11,689,512 fp32 params, K=%d" % K,
               resnet18_shapes(), K=K, grad_std=1e-3, eps_root=1e-8, count0=0,
               nonzero_moments=False, interior_cotangents=False)


def flat_1b(n: int = 1_000_000_000) -> Workload:
    return _mk("flat_1b", "flat fp32 buffer, one segment, n=%d, one step at count 100" % n,
               [(n,)], K=1, grad_std=1e-3, eps_root=0.0, count0=100,
               nonzero_moments=True, interior_cotangents=True)


def many_small(count: int = 20000, max_size: int = 65536, seed: int = 0, K: int = 3) -> Workload:
    sizes = many_small_sizes(count, max_size, seed)
    return _mk("many_small",
               "many-small-tensor tree, %d fp32 tensors, log-uniform sizes in [1, %d], "
               "n=%d, pack -> K=%d unrolled Adam fwd+bwd -> unpack" % (count, max_size, sum(sizes), K),
               [(s,) for s in sizes], K=K, grad_std=0.01, eps_root=0.0, count0=0,
               nonzero_moments=False, interior_cotangents=False)


WORKLOADS = {
    "tiny_mlp": tiny_mlp,
    "convnet32": convnet32,
    "resnet18_k1": lambda: resnet18(1),
    "resnet18_k10": lambda: resnet18(10),
    "flat_1b": flat_1b,
    "many_small": many_small,
}


# --------------------------------------------------------------------------
# Random arrays.  Streams are keyed by (workload tag, array tag, index) through
# numpy's SeedSequence, so any one array can be regenerated on its own.

ARRAY_TAGS = {"p0": 1, "grad": 2, "mu": 3, "nu": 4, "cot_p": 5, "cot_m": 6, "cot_v": 7, "misc": 8}


def _rng(wtag: str, atag: str, index: int = 0) -> np.random.Generator:
    wkey = [ord(c) for c in wtag]
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([BASE_SEED, ARRAY_TAGS[atag], index, *wkey])))


def normal(n: int, std: float, wtag: str, atag: str, index: int = 0) -> np.ndarray:
    """fp32 draw of N(0, std^2) (drawn in fp64, rounded once to fp32)."""
    return (_rng(wtag, atag, index).standard_normal(n) * std).astype(np.float32)


def abs_normal(n: int, std: float, wtag: str, atag: str, index: int = 0) -> np.ndarray:
    return np.abs(normal(n, std, wtag, atag, index))


def torch_normal(n: int, std: float, seed: int, device) -> "torch.Tensor":  # noqa: F821
    """fp32 N(0, std^2) drawn directly on a device with torch's seeded generator;
    used for arrays too large to draw on the host in reasonable time."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(BASE_SEED * 1000 + seed)
    out = torch.empty(n, dtype=torch.float32, device=device)
    out.normal_(0.0, std, generator=gen)
    return out


@dataclasses.dataclass
class StepInputs:
    """Host arrays for one unrolled run on a flat buffer (fp32)."""
    p0: np.ndarray
    grads: np.ndarray  # [K, n]
    m0: np.ndarray
    v0: np.ndarray
    cot_p: np.ndarray
    cot_m: np.ndarray  # zeros unless interior cotangents
    cot_v: np.ndarray
    count0: int
    K: int
    hyper: dict


def host_inputs(w: Workload, n: int | None = None) -> StepInputs:
    """Seeded host arrays for workload w (optionally truncated to n elements)."""
    n = w.n if n is None else n
    tag = w.name
    p0 = normal(n, 0.05, tag, "p0")
    grads = np.stack([normal(n, w.grad_std, tag, "grad", k) for k in range(w.K)]) if w.K else \
        np.zeros((0, n), np.float32)
    if w.nonzero_moments:
        m0 = abs_normal(n, 1e-4, tag, "mu")
        v0 = abs_normal(n, 1e-4, tag, "nu")
    else:
        m0 = np.zeros(n, np.float32)
        v0 = np.zeros(n, np.float32)
    cot_p = normal(n, 1.0, tag, "cot_p")
    if w.interior_cotangents:
        cot_m = normal(n, 1.0, tag, "cot_m")
        cot_v = normal(n, 1.0, tag, "cot_v")
    else:
        cot_m = np.zeros(n, np.float32)
        cot_v = np.zeros(n, np.float32)
    hyper = dict(HYPER, eps_root=w.eps_root)
    return StepInputs(p0, grads, m0, v0, cot_p, cot_m, cot_v, w.count0, w.K, hyper)


def random_shapes(count: int, max_numel: int, seed: int, allow_empty: bool = True) -> List[Tuple[int, ...]]:
    """Assorted leaf shapes for pack/unpack tests: empty, size-1, ragged, multi-d."""
    rng = _rng("shapes", "misc", seed)
    shapes: List[Tuple[int, ...]] = []
    for i in range(count):
        r = rng.uniform()
        if allow_empty and r < 0.05:
            shapes.append((0,))
        elif r < 0.15:
            shapes.append((1,))
        elif r < 0.5:
            shapes.append((int(rng.integers(2, 64)),))
        elif r < 0.8:
            a = int(rng.integers(1, 40))
            b = int(rng.integers(1, 40))
            shapes.append((a, b))
        else:
            shapes.append((int(rng.integers(1, max(2, max_numel))),))
    return shapes


def random_bits(n: int, dtype, seed: int) -> np.ndarray:
    """Uniformly random bit patterns of the given dtype (all NaN payloads,
    infinities, signed zeros and subnormals appear for float types)."""
    dtype = np.dtype(dtype)
    rng = _rng("bits", "misc", seed)
    raw = rng.integers(0, 256, size=n * dtype.itemsize, dtype=np.uint8)
    return raw.view(dtype)


def special_f32() -> np.ndarray:
    """A fixed set of fp32 bit patterns that must survive a copy unchanged."""
    bits = np.array([0x00000000, 0x80000000, 0x7F800000, 0xFF800000, 0x7FC00000,
                     0x7FA00001, 0xFFC12345, 0x7F800001, 0x00000001, 0x807FFFFF,
                     0x00800000, 0x3F800000, 0xBF800000, 0x7F7FFFFF], dtype=np.uint32)
    return bits.view(np.float32)
