"""The synthetic workloads C0..C6: flat fp32 parameter vectors shaped like
the generator/discriminator pairs of GAN training, split into segments (one
per layer or per group of layers), with the compressor each uses.  C0..C4
follow the five benchmark shapes; C5 and C6 repeat the shapes of C2 and C3
with the paper's own experimental compressor (8-bit sign-magnitude codes of
Appendix A with the infinity-norm scale).

Segment sizes of the two largest workloads are drawn log-uniformly (ratio up
to 1000 between segments), rounded down to a multiple of 64 elements (at least
64); the remainder of a region goes to its last segment.
"""
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np


def round_up(x, m):
    return (x + m - 1) // m * m


@dataclass
class Workload:
    index: int
    name: str
    d: int
    M: int
    kind: str                 # 'sign' | 'qsgd' | 'topk'
    norm: str                 # 'l1' | 'l2' | 'linf'
    levels: int               # s of the s-level quantizer (0 if unused)
    k: int                    # top-k budget (0 if unused)
    eta: float
    T: int
    seg_offsets: List[int]    # compressor segments: 0 = o_0 < ... < o_S = d
    groups: List[Tuple[int, int]]   # gradient groups (start, end), each with its own scale
    group_scale: List[float]  # per-group gradient scale (std or Laplace b)
    law: str                  # 'normal' | 'laplace'
    ld: int = 0
    base_seed: Optional[int] = None

    def __post_init__(self):
        if not self.ld:
            self.ld = round_up(self.d, 1024)

    @property
    def seed(self):
        """Gradient seed S: the workload index unless given explicitly."""
        return self.index if self.base_seed is None else self.base_seed

    @property
    def quant_seed(self):
        """Key of the stochastic-rounding generator."""
        return self.seed | (2 << 32)

    @property
    def init_seed(self):
        return self.seed | (3 << 32)

    @property
    def n_seg(self):
        return len(self.seg_offsets) - 1

    def as_dict(self):
        return {"d": self.d, "ld": self.ld, "M": self.M, "seg_offsets": list(self.seg_offsets),
                "kind": self.kind, "norm": self.norm, "levels": self.levels, "k": self.k,
                "seed": self.quant_seed}


def _log_uniform(rng, lo, hi, n):
    return np.exp(rng.uniform(np.log(lo), np.log(hi), size=n))


def _drawn_sizes(rng, total, count):
    """Log-uniform segment weights exp(U(0, ln 1000)); sizes rounded down to a
    multiple of 64 (minimum 64); the remainder goes to the last segment."""
    w = np.exp(rng.uniform(0.0, np.log(1000.0), size=count))
    raw = total * w / w.sum()
    sizes = [max(64, int(x) // 64 * 64) for x in raw[:-1]]
    last = total - sum(sizes)
    if last < 64:
        raise ValueError("segment draw left no room for the last segment")
    return sizes + [last]


def _offsets(sizes):
    o = [0]
    for s in sizes:
        o.append(o[-1] + s)
    return o


def _build(index):
    S = index
    if index == 0:
        d = 65536
        return Workload(0, "tiny", d, 4, "sign", "l1", 0, 0, 1e-3, 10, [0, d], [(0, d)], [1.0], "normal")
    if index == 1:
        # 2 -> 512 -> 512 -> 512 -> 1 MLP for each of G and D: layer parameter
        # counts 2*512+512, 512*512+512, 512*512+512, 512+1.
        per_net = [1536, 262656, 262656, 513]
        layers = per_net + per_net
        d = sum(layers)
        rng = np.random.default_rng(100 + S)
        sig = list(_log_uniform(rng, 1e-4, 1e-1, len(layers)))
        off = _offsets(layers)
        groups = [(off[j], off[j + 1]) for j in range(len(layers))]
        half = sum(per_net)
        return Workload(1, "mlp-gan", d, 8, "sign", "l1", 0, 0, 2e-4, 100, [0, half, d], groups, sig, "normal")
    if index == 2:
        # DCGAN 64x64: G (deconv + BN) and D (conv + BN) per-layer counts.
        G = [820224, 2097664, 524544, 131200, 3072]
        D = [3072, 131328, 524800, 2098176, 8192]
        layers = G + D
        d = sum(layers)
        rng = np.random.default_rng(100 + S)
        sig = list(_log_uniform(rng, 1e-4, 1e-1, len(layers)))
        off = _offsets(layers)
        groups = [(off[j], off[j + 1]) for j in range(len(layers))]
        return Workload(2, "dcgan", d, 16, "qsgd", "l2", 255, 0, 2e-4, 50, off, groups, sig, "normal")
    if index == 3:
        dG, dD = 24_000_000, 9_554_432
        rng = np.random.default_rng(200 + S)
        sizes = _drawn_sizes(rng, dG, 48) + _drawn_sizes(rng, dD, 16)
        off = _offsets(sizes)
        d = off[-1]
        rng2 = np.random.default_rng(100 + S)
        b = list(_log_uniform(rng2, 1e-5, 1e-1, len(sizes)))
        groups = [(off[j], off[j + 1]) for j in range(len(sizes))]
        return Workload(3, "resnet-wgan-gp", d, 32, "qsgd", "l2", 15, 0, 1e-4, 20, off, groups, b, "laplace")
    if index == 4:
        d = 100_000_000
        rng = np.random.default_rng(200 + S)
        sizes = _drawn_sizes(rng, d, 256)
        off = _offsets(sizes)
        rng2 = np.random.default_rng(100 + S)
        sig = list(_log_uniform(rng2, 1e-4, 1e-1, len(sizes)))
        groups = [(off[j], off[j + 1]) for j in range(len(sizes))]
        return Workload(4, "large-generator", d, 64, "topk", "none", 0, d // 100, 1e-4, 5, off, groups, sig, "normal")
    if index == 5:
        # the paper's experimental setting: DCGAN with 8-bit codes and Hou et
        # al.'s infinity-norm scale (Appendix A quantizer)
        w = _build(2)
        return Workload(5, "dcgan-hou8", w.d, w.M, "mbit", "linf", 8, 0, w.eta, w.T, w.seg_offsets, w.groups,
                        w.group_scale, w.law)
    if index == 6:
        w = _build(3)
        return Workload(6, "resnet-wgan-gp-hou8", w.d, w.M, "mbit", "linf", 8, 0, w.eta, w.T, w.seg_offsets,
                        w.groups, w.group_scale, w.law)
    raise KeyError(index)


CONFIGS = {i: None for i in range(7)}


def get(index) -> Workload:
    if CONFIGS[index] is None:
        CONFIGS[index] = _build(index)
    return CONFIGS[index]


def custom(d, M, kind, seg_offsets=None, norm=None, levels=0, k=0, eta=1e-3, seed=0, law="normal",
           group_scale=None, ld=None, index=99):
    """A small ad-hoc workload (tests: ragged sizes, tiny segments, ...)."""
    if seg_offsets is None:
        seg_offsets = [0, d]
    if norm is None:
        norm = "l1" if kind == "sign" else "l2"
    groups = [(seg_offsets[j], seg_offsets[j + 1]) for j in range(len(seg_offsets) - 1)]
    if group_scale is None:
        group_scale = [1.0] * len(groups)
    return Workload(index, "custom", d, M, kind, norm, levels, k, eta, 1, list(seg_offsets), groups,
                    list(group_scale), law, ld or 0, seed)
