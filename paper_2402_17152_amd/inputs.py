"""Seeded synthetic inputs for the HSTU jagged-attention path.

This module holds none of the method's arithmetic: it only draws the
random arrays (lengths, timestamps, Q/K/V/U, bias tables, upstream
gradient) that both the GPU path and the CPU oracle consume, and the
round-to-nearest-even cast of fp32 to bfloat16 used to store them.

The five workloads stand in for the paper's (its industrial data and the
public datasets are not used):

  tiny      fp32, B=4, L ~ U[16,128], h=2, d=32, N=128            (seed 0)
  medium    bf16 fwd, B=32, L ~ Zipf(1.2) clipped to [8,1024], h=4, d=64,
            N=1024                                                 (seed 1)
  training  bf16 fwd+bwd + LN*U epilogue, B=64, truncated power law on
            [64,4096] (mean ~1000), h=8, d=64, N=4096              (seed 2)
  long      bf16 fwd+bwd, B=8, L ~ U[4096,8192], h=4, d=128, N=8192 (seed 3)
  target    bf16 fwd, target-aware mask, B=16 x (2048 history + 1024
            candidates), h=4, d=128, N=3072                         (seed 4)

The skewed length mixes follow the paper's remark that user-history
lengths are skewed (Sec. 3.2, "Leveraging and algorithmically increasing
sparsity"); the 8192-long shape is its headline length (Sec. 4.2,
encoder efficiency); the target-aware shape is the M-FALCON inference
setting (Appendix on M-FALCON, Algorithm 1).

Draw order (one PCG64 stream per workload, seed = workload index):
lengths, timestamp gaps, Q, K, V, U, rab_pos, rab_time, dO.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

CONFIG_NAMES = ("tiny", "medium", "training", "long", "target")

# Exponent of the truncated power law for the training-shape lengths; it
# makes the mean of a density proportional to x**-a on [64, 4096] equal 1000.
_POWER_LAW_A = 0.9727141
TIME_ORIGIN = 1_700_000_000
GAP_MEAN_S = 600.0
RAB_STD = 0.02


@dataclasses.dataclass(frozen=True)
class Workload:
    index: int
    name: str
    dtype: str            # "f32" or "bf16": storage type of Q/K/V/U/dO
    num_heads: int
    d_qk: int
    d_v: int
    max_seq_len: int      # N: normalizer and rab_pos half-width
    num_time_buckets: int
    backward: bool
    epilogue: bool
    target_aware: bool


WORKLOADS = (
    Workload(0, "tiny", "f32", 2, 32, 32, 128, 128, True, True, False),
    Workload(1, "medium", "bf16", 4, 64, 64, 1024, 128, False, False, False),
    Workload(2, "training", "bf16", 8, 64, 64, 4096, 128, True, True, False),
    Workload(3, "long", "bf16", 4, 128, 128, 8192, 128, True, False, False),
    Workload(4, "target", "bf16", 4, 128, 128, 3072, 128, False, False, True),
)


def workload(name_or_index) -> Workload:
    if isinstance(name_or_index, int):
        return WORKLOADS[name_or_index]
    for w in WORKLOADS:
        if w.name == name_or_index:
            return w
    raise KeyError(name_or_index)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit pattern (uint16), round to nearest, ties to even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    """Widen a bf16 bit pattern (uint16) exactly to float64."""
    u = (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16)
    return u.view(np.float32).astype(np.float64)


@dataclasses.dataclass
class Batch:
    """One jagged batch. Float tensors are kept both as the stored values
    (``*_store``: float32 arrays or bf16 bit patterns as uint16) and as the
    same values widened exactly to float64 (for the oracle)."""
    spec: Workload
    lengths: np.ndarray          # int64 [B]
    seq_offsets: np.ndarray      # int64 [B+1]
    timestamps: np.ndarray       # int64 [T]
    num_targets: Optional[np.ndarray]  # int64 [B] or None
    rab_pos: np.ndarray          # float32 [2N-1]
    rab_time: np.ndarray         # float32 [B_t]
    store: dict                  # name -> stored array [T, h, d] (float32 or uint16)

    @property
    def total_tokens(self) -> int:
        return int(self.seq_offsets[-1])

    def f64(self, name: str) -> np.ndarray:
        a = self.store[name]
        if a.dtype == np.uint16:
            return bf16_bits_to_f64(a)
        return a.astype(np.float64)


def _lengths(spec: Workload, rng: np.random.Generator) -> np.ndarray:
    i = spec.index
    if i == 0:
        return rng.integers(16, 128, size=4, endpoint=True).astype(np.int64)
    if i == 1:
        return np.clip(rng.zipf(1.2, size=32), 8, 1024).astype(np.int64)
    if i == 2:
        a = _POWER_LAW_A
        u = rng.random(64)
        lo, hi = 64.0 ** (1 - a), 4096.0 ** (1 - a)
        x = np.floor((lo + u * (hi - lo)) ** (1.0 / (1 - a)))
        return np.clip(x, 64, 4096).astype(np.int64)
    if i == 3:
        return rng.integers(4096, 8192, size=8, endpoint=True).astype(np.int64)
    if i == 4:
        return np.full(16, 3072, dtype=np.int64)
    raise ValueError(i)


def _silu_normal(rng: np.random.Generator, shape) -> np.ndarray:
    # Q/K/V/U are drawn as the output of the SiLU projection of Eq. 1:
    # z ~ N(0,1), value = z * sigmoid(z). This is the input distribution only.
    z = rng.standard_normal(shape)
    return z / (1.0 + np.exp(-z))


def _store(x64: np.ndarray, dtype: str) -> np.ndarray:
    x32 = x64.astype(np.float32)
    if dtype == "f32":
        return x32
    return f32_to_bf16_bits(x32)


def make_batch(spec, seed: Optional[int] = None, lengths=None,
               num_targets=None, num_heads=None, d_qk=None, d_v=None,
               max_seq_len=None, dtype=None, num_time_buckets=None,
               timestamps=None) -> Batch:
    """Draw one batch. ``spec`` is a Workload, its name or index. Any of the
    shape arguments overrides the workload's (used by tests for small or
    edge-case shapes); the draw order stays the same."""
    if not isinstance(spec, Workload):
        spec = workload(spec)
    over = {}
    for k, v in (("num_heads", num_heads), ("d_qk", d_qk), ("d_v", d_v),
                 ("max_seq_len", max_seq_len), ("dtype", dtype),
                 ("num_time_buckets", num_time_buckets)):
        if v is not None:
            over[k] = v
    if over:
        spec = dataclasses.replace(spec, **over)
    rng = np.random.default_rng(spec.index if seed is None else seed)

    if lengths is None:
        lens = _lengths(WORKLOADS[spec.index], rng)
    else:
        lens = np.asarray(lengths, dtype=np.int64)
    B = len(lens)
    offs = np.zeros(B + 1, dtype=np.int64)
    offs[1:] = np.cumsum(lens)
    T = int(offs[-1])

    if num_targets is None and spec.target_aware and lengths is None:
        nt = np.full(B, 1024, dtype=np.int64)
    elif num_targets is not None:
        nt = np.broadcast_to(np.asarray(num_targets, dtype=np.int64), (B,)).copy()
    else:
        nt = None

    gaps = np.floor(rng.exponential(GAP_MEAN_S, size=T)).astype(np.int64)
    if timestamps is None:
        ts = np.empty(T, dtype=np.int64)
        for b in range(B):
            s, e = offs[b], offs[b + 1]
            ts[s:e] = TIME_ORIGIN + np.cumsum(gaps[s:e])
    else:
        ts = np.asarray(timestamps, dtype=np.int64).copy()

    h, dqk, dv = spec.num_heads, spec.d_qk, spec.d_v
    store = {}
    store["q"] = _store(_silu_normal(rng, (T, h, dqk)), spec.dtype)
    store["k"] = _store(_silu_normal(rng, (T, h, dqk)), spec.dtype)
    store["v"] = _store(_silu_normal(rng, (T, h, dv)), spec.dtype)
    store["u"] = _store(_silu_normal(rng, (T, h, dv)), spec.dtype)
    N = spec.max_seq_len
    rab_pos = (RAB_STD * rng.standard_normal(2 * N - 1)).astype(np.float32)
    rab_time = (RAB_STD * rng.standard_normal(spec.num_time_buckets)).astype(np.float32)
    store["do"] = _store(rng.standard_normal((T, h, dv)), spec.dtype)
    return Batch(spec, lens, offs, ts, nt, rab_pos, rab_time, store)


def causal_pairs(batch: Batch) -> int:
    """Number of (query, key) pairs the mask keeps, per head."""
    total = 0
    for b, L in enumerate(batch.lengths):
        L = int(L)
        nt = 0 if batch.num_targets is None else int(batch.num_targets[b])
        nh = L - nt
        total += nh * (nh + 1) // 2 + nt * (nh + 1)
    return total


def flops(batch: Batch):
    """Algorithmic MFMA work of one forward and one backward pass: two
    contractions of width d per kept pair and head forward (Q K^T, A V),
    five backward (recomputed Q K^T, dO V^T, A^T dO, dS K, dS^T Q)."""
    s = batch.spec
    p = causal_pairs(batch) * s.num_heads
    return 2 * p * (s.d_qk + s.d_v), 2 * p * (3 * s.d_qk + 2 * s.d_v)


def sub_batch(batch: Batch, seqs) -> Batch:
    """The sequences ``seqs`` of a batch as a batch of their own (same N,
    tables and values)."""
    offs = batch.seq_offsets
    seqs = [int(b) for b in seqs]
    rows = (np.concatenate([np.arange(offs[b], offs[b + 1]) for b in seqs])
            if seqs else np.zeros(0, np.int64))
    lens = np.array([offs[b + 1] - offs[b] for b in seqs], dtype=np.int64)
    new_offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    store = {k: v[rows] for k, v in batch.store.items()}
    nt = None if batch.num_targets is None else batch.num_targets[seqs]
    return Batch(batch.spec, lens, new_offs, batch.timestamps[rows], nt, batch.rab_pos,
                 batch.rab_time, store)


def make_proj(num_tokens, d_model, num_heads, d_qk, d_v, dtype="bf16", seed=0) -> dict:
    """Seeded inputs of the layer's linear maps (Eq. 1 and Eq. 3's f_2):
    x [T, D], w1 [F, D], w2 [D, h d_v] with N(0, 1/fan_in) entries; b1 [F],
    b2 [D] ~ N(0, 0.1^2) (kept fp32); g [T, h d_v] (the gated layer-norm
    output), dz [T, F] and dy [T, D] ~ N(0, 1).  Matrices are stored in
    ``dtype`` (bf16 bit patterns or fp32)."""
    rng = np.random.default_rng(seed)
    T, D = int(num_tokens), int(d_model)
    hv = num_heads * d_v
    F = 2 * num_heads * (d_qk + d_v)
    out = {
        "x": _store(rng.standard_normal((T, D)), dtype),
        "w1": _store(rng.standard_normal((F, D)) / np.sqrt(D), dtype),
        "b1": (0.1 * rng.standard_normal(F)).astype(np.float32),
        "w2": _store(rng.standard_normal((D, hv)) / np.sqrt(hv), dtype),
        "b2": (0.1 * rng.standard_normal(D)).astype(np.float32),
        "g": _store(rng.standard_normal((T, hv)), dtype),
        "dz": _store(rng.standard_normal((T, F)), dtype),
        "dy": _store(rng.standard_normal((T, D)), dtype),
    }
    return out


def make_sl_draws(num_seqs, num_tokens, seed=0):
    """The random draws Stochastic Length consumes: u_keep [B] ~ U[0, 1)
    (keep-whole decision of Eq. 4) and e_rand [T] ~ Exp(1) (selection keys)."""
    rng = np.random.default_rng(seed)
    return rng.random(int(num_seqs)), rng.exponential(size=int(num_tokens))


def stored_f64(a: np.ndarray) -> np.ndarray:
    """The exact values of a stored array (bf16 bit patterns or fp32) in fp64."""
    return bf16_bits_to_f64(a) if a.dtype == np.uint16 else a.astype(np.float64)


def array_to_device(a: np.ndarray, device="cuda"):
    """One stored array as a torch tensor (bf16 bit patterns reinterpreted)."""
    import torch
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def to_device(batch: Batch, device="cuda") -> dict:
    """Copies a batch to device memory as torch tensors (bf16 bit patterns
    are reinterpreted, not converted)."""
    import torch

    def t(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(device)
        return torch.from_numpy(np.ascontiguousarray(a)).to(device)

    d = {n: t(a) for n, a in batch.store.items()}
    d["seq_offsets"] = t(batch.seq_offsets)
    d["timestamps"] = t(batch.timestamps)
    d["rab_pos"] = t(batch.rab_pos)
    d["rab_time"] = t(batch.rab_time)
    d["num_targets"] = None if batch.num_targets is None else t(batch.num_targets)
    return d
