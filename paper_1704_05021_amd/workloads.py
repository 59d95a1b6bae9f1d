"""Seeded synthetic gradient workloads shaped like the paper's two tasks.

This module only draws random numbers.  It holds none of the method's
arithmetic (no residual add, no threshold, no compaction) and is the one
piece of code that the CPU oracle and the HIP path share: both are fed the
same bytes from here.

The paper trains an MNIST multi-layer perceptron and an attentional NMT
encoder-decoder (Section 5).  Neither dataset nor any trained weight is
available, so every workload is a seeded stand-in with the structure the
paper describes (Section 1): gradients skewed towards zero, MNIST touching
every parameter on every batch, NMT dominated by three vocabulary-sized
embedding matrices of which only the rows of words seen in the batch carry a
gradient, and tensors on different scales (Sections 1 and 4).

Every stream is ``numpy.random.Generator(PCG64(SeedSequence(key)))`` with
``key = [seed, step, tensor]`` (or a tagged key for per-tensor constants);
values are drawn in float64 and rounded once to float32.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "Layout",
    "mlp_layout",
    "nmt_layout",
    "rng_for",
    "grad_mlp_normal",
    "grad_mlp_student_t",
    "grad_nmt",
    "server_shard",
    "Workload",
    "WORKLOADS",
    "workload",
]

# Tag mixed into the seed key for constants drawn once per tensor (not per step).
_TAG_TENSOR_CONST = 1_000_003
# Tag for the server-shard streams.
_TAG_SHARD = 2_000_003


def rng_for(*key: int) -> np.random.Generator:
    """A PCG64 generator seeded from ``SeedSequence(list(key))``."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


@dataclass(frozen=True)
class Layout:
    """Flat concatenation of named tensors; ``offsets`` has ``T + 1`` entries."""

    names: Tuple[str, ...]
    shapes: Tuple[Tuple[int, ...], ...]

    @property
    def sizes(self) -> List[int]:
        return [int(np.prod(s)) for s in self.shapes]

    @property
    def offsets(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.sizes)]).astype(np.uint64)

    @property
    def numel(self) -> int:
        return int(sum(self.sizes))

    @property
    def num_tensors(self) -> int:
        return len(self.names)

    @property
    def columns(self) -> List[int]:
        """Columns of each tensor read as a row-major matrix (a vector is one row)."""
        return [int(s[-1]) if len(s) else 1 for s in self.shapes]


def mlp_layout(widths: Sequence[int]) -> Layout:
    """Weights and biases of a fully connected net, interleaved W1, b1, W2, b2, ...

    ``widths = (784, 512, 512, 10)`` gives the six tensors of a 784-512-512-10
    MLP; each weight is stored ``fan_in x fan_out``.
    """
    names, shapes = [], []
    for i in range(len(widths) - 1):
        names += [f"W{i + 1}", f"b{i + 1}"]
        shapes += [(widths[i], widths[i + 1]), (widths[i + 1],)]
    return Layout(tuple(names), tuple(shapes))


def nmt_layout(vocab: int = 85000, emb: int = 500, hidden: int = 1024, blocks: int = 6) -> Layout:
    """Three vocabulary x embedding matrices, then ``blocks`` recurrent blocks.

    Order: source input embedding, target input embedding, target output
    embedding, then per block j: input weight ``hidden x emb`` and its bias,
    recurrent weight ``hidden x hidden`` and its bias (GRU-shaped dense tensors).
    """
    names = ["E_src", "E_tgt", "E_out"]
    shapes: List[Tuple[int, ...]] = [(vocab, emb)] * 3
    for j in range(blocks):
        names += [f"W{j}", f"bW{j}", f"U{j}", f"bU{j}"]
        shapes += [(hidden, emb), (hidden,), (hidden, hidden), (hidden,)]
    return Layout(tuple(names), tuple(shapes))


def grad_mlp_normal(layout: Layout, seed: int, step: int, sigma: float = 1e-2) -> np.ndarray:
    """Every tensor drawn i.i.d. normal with standard deviation ``sigma``."""
    out = np.empty(layout.numel, dtype=np.float32)
    off = layout.offsets
    for t, n in enumerate(layout.sizes):
        out[off[t]:off[t + 1]] = rng_for(seed, step, t).normal(0.0, sigma, n).astype(np.float32)
    return out


def tensor_scales_loguniform(layout: Layout, seed: int, lo_exp: float = -4.0, hi_exp: float = -2.0) -> np.ndarray:
    """One scale per tensor, ``10 ** U(lo_exp, hi_exp)``, fixed for all steps."""
    return np.array(
        [10.0 ** rng_for(seed, _TAG_TENSOR_CONST, t).uniform(lo_exp, hi_exp) for t in range(layout.num_tensors)]
    )


def grad_mlp_student_t(layout: Layout, seed: int, step: int, nu: float = 3.0) -> np.ndarray:
    """Heavy-tailed gradients: ``c_t * StudentT(nu)`` with a per-tensor scale ``c_t``."""
    scales = tensor_scales_loguniform(layout, seed)
    out = np.empty(layout.numel, dtype=np.float32)
    off = layout.offsets
    for t, n in enumerate(layout.sizes):
        out[off[t]:off[t + 1]] = (scales[t] * rng_for(seed, step, t).standard_t(nu, n)).astype(np.float32)
    return out


def zipf_cdf(vocab: int, s: float) -> np.ndarray:
    """Cumulative distribution of a Zipf law truncated to ranks ``1..vocab``."""
    w = np.arange(1, vocab + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(w)
    return c / c[-1]


def grad_nmt(
    layout: Layout,
    seed: int,
    step: int,
    tokens: int = 3000,
    zipf_s: float = 1.1,
    sigma: float = 1e-3,
    n_embeddings: int = 3,
) -> np.ndarray:
    """NMT-shaped gradient set.

    For each embedding matrix, ``tokens`` word ranks are drawn i.i.d. from a
    truncated Zipf law over the vocabulary; the distinct rows hit get
    ``N(0, sigma)`` in every column and every other row is exactly zero.
    Dense and bias tensors are ``N(0, sigma)``.
    """
    out = np.zeros(layout.numel, dtype=np.float32)
    off = layout.offsets
    for t, (shape, n) in enumerate(zip(layout.shapes, layout.sizes)):
        rng = rng_for(seed, step, t)
        if t < n_embeddings:
            vocab, width = shape
            cdf = zipf_cdf(vocab, zipf_s)
            ranks = np.searchsorted(cdf, rng.random(tokens), side="right")  # 0-based row
            rows = np.unique(np.minimum(ranks, vocab - 1))
            vals = rng.normal(0.0, sigma, (rows.size, width)).astype(np.float32)
            view = out[off[t]:off[t + 1]].reshape(vocab, width)
            view[rows] = vals
        else:
            out[off[t]:off[t + 1]] = rng.normal(0.0, sigma, n).astype(np.float32)
    return out


@dataclass
class ShardPushes:
    params: np.ndarray  # float32 [n]
    idx: List[np.ndarray]  # uint32, ascending, unique per client
    val: List[np.ndarray]  # float32


def server_shard(
    n: int,
    clients: int,
    nnz: int,
    dup_frac: float,
    seed: int,
    p_sigma: float = 0.1,
    v_scale: float = 1e-3,
    nu: float = 3.0,
) -> ShardPushes:
    """A parameter shard and sparse pushes from ``clients`` simulated clients.

    Client 0 draws ``nnz`` distinct indices uniformly.  Client c > 0 draws
    ``round(dup_frac * nnz)`` indices from the union of earlier clients'
    indices and the rest fresh (outside that union), all distinct.  Values are
    ``v_scale * StudentT(nu)``; parameters are ``N(0, p_sigma)``.
    """
    params = rng_for(seed, _TAG_SHARD, 0).normal(0.0, p_sigma, n).astype(np.float32)
    idx_lists: List[np.ndarray] = []
    val_lists: List[np.ndarray] = []
    union = np.zeros(0, dtype=np.int64)
    for c in range(clients):
        rng = rng_for(seed, _TAG_SHARD, 1 + c)
        n_dup = int(round(dup_frac * nnz)) if c > 0 else 0
        n_dup = min(n_dup, union.size)
        dup = rng.choice(union, size=n_dup, replace=False) if n_dup else np.zeros(0, np.int64)
        need = nnz - n_dup
        if need > n - union.size:
            raise ValueError(f"client {c} needs {need} fresh indices but only {n - union.size} of {n} are left")
        fresh = np.zeros(0, dtype=np.int64)
        while fresh.size < need:
            cand = rng.integers(0, n, size=2 * (need - fresh.size) + 16, dtype=np.int64)
            cand = np.setdiff1d(np.unique(cand), union, assume_unique=False)
            cand = np.setdiff1d(cand, fresh, assume_unique=True)
            if cand.size > need - fresh.size:
                cand = rng.choice(cand, size=need - fresh.size, replace=False)
            fresh = np.concatenate([fresh, cand])
        ix = np.sort(np.concatenate([dup, fresh]))
        idx_lists.append(ix.astype(np.uint32))
        val_lists.append((v_scale * rng.standard_t(nu, ix.size)).astype(np.float32))
        union = np.union1d(union, ix)
    return ShardPushes(params, idx_lists, val_lists)


@dataclass
class Workload:
    """A named configuration: layout, generator, drop ratio, threshold mode, steps."""

    name: str
    layout: Layout
    kind: str  # "mlp_normal" | "mlp_student_t" | "nmt" | "shard"
    seed: int
    steps: int
    drop: float = 0.99
    per_tensor: bool = False
    quant: bool = False
    extra: Dict[str, float] = field(default_factory=dict)

    def grad(self, step: int) -> np.ndarray:
        if self.kind == "mlp_normal":
            return grad_mlp_normal(self.layout, self.seed, step, **self.extra)
        if self.kind == "mlp_student_t":
            return grad_mlp_student_t(self.layout, self.seed, step, **self.extra)
        if self.kind == "nmt":
            return grad_nmt(self.layout, self.seed, step, **self.extra)
        raise ValueError(f"workload {self.name} has no gradient stream")


def _nmt_extra(tokens: int) -> Dict[str, float]:
    return {"tokens": tokens}


# Full-size workloads.  Names describe the shapes; "scaled" variants keep the
# structure at a size a CPU finishes in well under a second.
WORKLOADS: Dict[str, Workload] = {
    "mnist_mlp_784_512_512_10": Workload(
        "mnist_mlp_784_512_512_10", mlp_layout((784, 512, 512, 10)), "mlp_normal", seed=0, steps=1),
    "mlp_784_4096_4096_10_t3": Workload(
        "mlp_784_4096_4096_10_t3", mlp_layout((784, 4096, 4096, 10)), "mlp_student_t", seed=2, steps=20),
    "nmt_85k_per_tensor": Workload(
        "nmt_85k_per_tensor", nmt_layout(), "nmt", seed=3, steps=10, per_tensor=True, extra=_nmt_extra(3000)),
    "nmt_85k_global_signmean": Workload(
        "nmt_85k_global_signmean", nmt_layout(), "nmt", seed=3, steps=10, quant=True, extra=_nmt_extra(3000)),
    # scaled stand-ins with the same structure, for fast parity runs
    "mlp_784_256_256_10_t3_small": Workload(
        "mlp_784_256_256_10_t3_small", mlp_layout((784, 256, 256, 10)), "mlp_student_t", seed=2, steps=4),
    "nmt_small_per_tensor": Workload(
        "nmt_small_per_tensor", nmt_layout(vocab=4000, emb=96, hidden=128, blocks=2), "nmt", seed=3, steps=4,
        per_tensor=True, extra=_nmt_extra(140)),
    "nmt_small_global_signmean": Workload(
        "nmt_small_global_signmean", nmt_layout(vocab=4000, emb=96, hidden=128, blocks=2), "nmt", seed=3, steps=4,
        quant=True, extra=_nmt_extra(140)),
}

# Server shard: 37,000,000 fp32 parameters, 4 clients x 370,000 pushes, ~5% overlap.
SHARD_FULL = dict(n=37_000_000, clients=4, nnz=370_000, dup_frac=0.05, seed=5)
SHARD_SMALL = dict(n=600_000, clients=4, nnz=6_000, dup_frac=0.05, seed=5)


def workload(name: str) -> Workload:
    return WORKLOADS[name]
