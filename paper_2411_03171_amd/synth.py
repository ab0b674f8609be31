"""Seeded synthetic inputs for the fixed fan-in sparse layer.

This module holds the workload shapes and the input generators only; it does
none of the method's arithmetic, so that both the HIP path and the CPU oracle
can be fed the very same bits.  The paper's datasets are not available; the
generators reproduce the shapes and the statistics that matter for the sparse
layer (label-space size, fan-in, batch size, number of positives per sample,
long-tailed label frequencies):

  X        N(0,1) rows, then either L2-normalised (fp32 workload) or
           LayerNorm-ed without affine (eps 1e-5) and rounded to bf16 -- a
           stand-in for a BERT [CLS] embedding, d = 768 (Sec. 3.1 encoders).
  W        U(-1/sqrt(k), 1/sqrt(k)), stored in the workload's value type.
  I        k distinct uniform columns per row, ascending.
  targets  1 + Poisson(mean-1) positives per sample, labels drawn i.i.d. from
           a Zipf(s) law truncated to [0, L) (rank r -> label r-1), repeats
           within a sample redrawn -- a stand-in for the long-tailed label
           distributions of the XMC datasets (Sec. 3.1, Table 1).

All randomness flows from one root seed through numpy SeedSequence.spawn.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int                 # batch size
    d: int                 # input width of the sparse layer
    L: int                 # number of labels
    k: int                 # fan-in
    value: str             # "f32" or "bf16" for X and W
    mean_pos: float        # mean positives per sample
    zipf_s: float          # Zipf exponent of label frequencies
    set_frac: float        # SET prune/regrow fraction
    set_every: int         # SET interval (steps)
    steps: int = 1         # training steps of the workload
    x_norm: str = "layernorm"   # "l2" or "layernorm"
    din: int = 0           # dense intermediate layer input width (0: none)
    aux_clusters: int = 0  # auxiliary head over label clusters (0: none)

    @property
    def slots(self) -> int:
        return self.L * self.k


# The five workloads: fp32 correctness case; LF-AmazonTitles-131K-like;
# intermediate layer + sparse head; Amazon-3M-like (the largest label space);
# auxiliary cluster head + sparse head.
WORKLOADS = {
    "c1_fp32_L4096": Workload("c1_fp32_L4096", B=32, d=128, L=4096, k=16, value="f32",
                              mean_pos=4.0, zipf_s=1.1, set_frac=0.3, set_every=1,
                              steps=1, x_norm="l2"),
    "c2_bf16_L131072": Workload("c2_bf16_L131072", B=128, d=768, L=131072, k=32, value="bf16",
                                mean_pos=5.0, zipf_s=1.1, set_frac=0.1, set_every=20,
                                steps=100),
    "c3_inter2048_L1M": Workload("c3_inter2048_L1M", B=128, d=2048, L=1048576, k=64,
                                 value="bf16", mean_pos=5.0, zipf_s=1.0, set_frac=0.1,
                                 set_every=100, steps=1, din=768),
    "c4_bf16_L3M": Workload("c4_bf16_L3M", B=64, d=768, L=3145728, k=32, value="bf16",
                            mean_pos=4.0, zipf_s=1.1, set_frac=0.1, set_every=1000, steps=1),
    "c5_aux8192_L1M": Workload("c5_aux8192_L1M", B=128, d=768, L=1048576, k=32, value="bf16",
                               mean_pos=5.0, zipf_s=1.1, set_frac=0.1, set_every=100, steps=1,
                               aux_clusters=8192),
}


def scaled(w: Workload, L: Optional[int] = None, B: Optional[int] = None,
           d: Optional[int] = None, k: Optional[int] = None, name: Optional[str] = None) -> Workload:
    """A smaller copy of a workload (same distributions), for oracle-sized tests."""
    return dataclasses.replace(w, L=L or w.L, B=B or w.B, d=d or w.d, k=k or w.k,
                               name=name or (w.name + "_scaled"))


# --------------------------------------------------------------------------
# bf16 bit patterns

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (ties to even); returns uint16 bit patterns."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    u = x32.view(np.uint32)
    # for every non-NaN pattern u + 0x8000 stays below 2^32, so uint32 is exact
    r = (u >> 16) & np.uint32(1)
    r += u
    r += np.uint32(0x7FFF)
    r >>= np.uint32(16)
    out = r.astype(np.uint16)
    nan = np.isnan(x32)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# generators

class Streams:
    """Independent numpy Generators derived from one root seed."""

    NAMES = ("x", "w", "i", "targets", "dense", "aux", "batches")

    def __init__(self, seed: int):
        ss = np.random.SeedSequence(seed)
        children = ss.spawn(len(self.NAMES))
        self.g = {n: np.random.Generator(np.random.PCG64(c)) for n, c in zip(self.NAMES, children)}

    def __getitem__(self, name):
        return self.g[name]


def gen_x(rng: np.random.Generator, B: int, d: int, norm: str, value: str) -> np.ndarray:
    """Returns float32 values (value == 'f32') or bf16 bit patterns (uint16)."""
    x = rng.standard_normal((B, d))
    if norm == "l2":
        x = x / np.linalg.norm(x, axis=1, keepdims=True)
    else:
        mu = x.mean(axis=1, keepdims=True)
        var = ((x - mu) ** 2).mean(axis=1, keepdims=True)
        x = (x - mu) / np.sqrt(var + 1e-5)
    x32 = x.astype(np.float32)
    return x32 if value == "f32" else f32_to_bf16_bits(x32)


def gen_w(rng: np.random.Generator, L: int, k: int, value: str, chunk: int = 1 << 18) -> np.ndarray:
    """U(-1/sqrt(k), 1/sqrt(k)) weights, drawn in float32 chunk by chunk."""
    a = np.float32(1.0 / np.sqrt(k))
    out = np.empty((L, k), dtype=np.float32 if value == "f32" else np.uint16)
    for s in range(0, L, chunk):
        e = min(L, s + chunk)
        w32 = rng.random((e - s, k), dtype=np.float32)
        w32 *= 2 * a
        w32 -= a
        out[s:e] = w32 if value == "f32" else f32_to_bf16_bits(w32)
    return out


def gen_indices(rng: np.random.Generator, L: int, k: int, d: int, chunk: int = 1 << 20) -> np.ndarray:
    """k distinct uniform columns in [0, d) per row, sorted ascending (int32)."""
    if k > d:
        raise ValueError("fan-in k cannot exceed the input width d")
    out = np.empty((L, k), dtype=np.int32)
    for s in range(0, L, chunk):
        e = min(L, s + chunk)
        rows = rng.integers(0, d, size=(e - s, k), dtype=np.int32)
        while True:
            rows.sort(axis=1)
            dup = np.zeros(rows.shape, dtype=bool)
            dup[:, 1:] = rows[:, 1:] == rows[:, :-1]
            n = int(dup.sum())
            if n == 0:
                break
            rows[dup] = rng.integers(0, d, size=n, dtype=np.int32)
        out[s:e] = rows
    return out


def zipf_cdf(L: int, s: float) -> np.ndarray:
    r = np.arange(1, L + 1, dtype=np.float64)
    w = r ** (-s)
    c = np.cumsum(w)
    return c / c[-1]


def gen_targets(rng: np.random.Generator, B: int, L: int, mean_pos: float, s: float,
                cdf: Optional[np.ndarray] = None):
    """CSR multi-hot targets: (offsets int64 [B+1], labels int32 [nnz])."""
    if cdf is None:
        cdf = zipf_cdf(L, s)
    npos = 1 + rng.poisson(max(mean_pos - 1.0, 0.0), size=B)
    npos = np.minimum(npos, L)
    labs = []
    for b in range(B):
        chosen = []
        seen = set()
        while len(chosen) < npos[b]:
            u = rng.random(int(npos[b]) - len(chosen))
            cand = np.minimum(np.searchsorted(cdf, u, side="right"), L - 1)
            for c in cand.tolist():
                if c not in seen:
                    seen.add(c)
                    chosen.append(c)
        labs.append(np.array(chosen, dtype=np.int32))
    off = np.zeros(B + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(a) for a in labs])
    lab = np.concatenate(labs) if labs else np.zeros(0, dtype=np.int32)
    return off, lab.astype(np.int32)


@dataclasses.dataclass
class LayerInputs:
    X: np.ndarray          # float32 [B,d] or uint16 bf16 bits
    W: np.ndarray          # float32 [L,k] or uint16 bf16 bits
    I: np.ndarray          # int32 [L,k]
    off: np.ndarray        # int64 [B+1]
    lab: np.ndarray        # int32 [nnz]
    bias: np.ndarray       # float32 [L] (zeros)


def make_layer_inputs(w: Workload, seed: int = 0) -> LayerInputs:
    st = Streams(seed)
    din = w.din if w.din else w.d
    X = gen_x(st["x"], w.B, din, "l2" if w.x_norm == "l2" else "layernorm", w.value)
    W = gen_w(st["w"], w.L, w.k, w.value)
    I = gen_indices(st["i"], w.L, w.k, w.d)
    off, lab = gen_targets(st["targets"], w.B, w.L, w.mean_pos, w.zipf_s)
    bias = np.zeros(w.L, dtype=np.float32)
    return LayerInputs(X=X, W=W, I=I, off=off, lab=lab, bias=bias)


def make_batches(w: Workload, n: int, seed: int = 0):
    """n fresh (X, off, lab) batches for multi-step runs."""
    st = Streams(seed)
    rng = st["batches"]
    cdf = zipf_cdf(w.L, w.zipf_s)
    din = w.din if w.din else w.d
    out = []
    for _ in range(n):
        X = gen_x(rng, w.B, din, "l2" if w.x_norm == "l2" else "layernorm", w.value)
        off, lab = gen_targets(rng, w.B, w.L, w.mean_pos, w.zipf_s, cdf=cdf)
        out.append((X, off, lab))
    return out


def make_dense(rng: np.random.Generator, din: int, dout: int) -> np.ndarray:
    """A dense bf16 weight [din, dout] ~ U(-1/sqrt(din), 1/sqrt(din)) (bit patterns)."""
    a = 1.0 / np.sqrt(din)
    return f32_to_bf16_bits(rng.uniform(-a, a, size=(din, dout)).astype(np.float32))


def make_intermediate(w: Workload, seed: int = 0) -> np.ndarray:
    return make_dense(Streams(seed)["dense"], w.din, w.d)


def make_aux(w: Workload, seed: int = 0) -> np.ndarray:
    return make_dense(Streams(seed)["aux"], w.d, w.aux_clusters)
