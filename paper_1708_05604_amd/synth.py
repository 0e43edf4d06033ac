"""Seeded synthetic workloads standing in for the paper's handwriting data.

The paper trains on a private online-handwriting corpus (Sec. IV.A) that is not
available, so every input here is synthetic, with the shapes of the six
workloads this library is measured on:

  tiny      1-layer LSTM, D=4,  H=32,  C=20, n=64,    lengths U[10,100],        B=16,  fp32
  lstm2     2-layer LSTM, D=8,  H=128, C=80, n=4096,  lognormal(300,0.6)[20,1500], B=64, fp32
  bilstm3   3-layer bidirectional LSTM, D=8, H=256, C=80, n=16384,
            lognormal(400,0.7)[20,2500], B=64, bf16 GEMM operands / fp32 accumulate
  longtail  2-layer LSTM, D=16, H=512, C=100, n=8192, Pareto(1.5, x_m=50)[50,4000],
            B=128, bf16 GEMM operands
  gru2      2-layer GRU,  D=8,  H=384, C=80, n=16384, lognormal(300,0.6)[20,1500], B=96, fp32
  lstm2p    lstm2 with the peephole LSTM cell

This module is shared by the oracle and by the GPU path; it only draws random
numbers and holds none of the method's arithmetic (no bucketing, no batching,
no recurrence).  Draw order for ``make_workload``:
  1. lengths (n values) from the workload's length law,
  2. features X = standard_normal((sum(lengths), D)) as float32, rows in
     sequence order (sequence s occupies rows offsets[s]:offsets[s+1]),
  3. labels   Y = integers(0, C, sum(lengths)) as int32, same row order,
  4. parameters (when a count is given) = uniform(-0.1, 0.1, count) as float32.
Shuffle keys for an epoch come from a separate generator seeded by
(seed, epoch) so that any epoch can be regenerated on its own.

Label strings for the CTC loss (``ctc_targets``) come from their own generator
seeded by (seed, 0xC7C), so the per-frame draws above do not change: sequence
s, in index order, gets max(1, L_s // FRAMES_PER_LABEL) labels uniform over
classes 1..C-1 (class 0 is the blank).  Eight frames per label keeps every
string alignable (L_s >= 2 U_s covers a blank between every pair of equal
neighbours).
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

LSTM = 0
GRU = 1
LSTM_PEEPHOLE = 2
FP32 = 0
BF16 = 1


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    cell: int            # LSTM, GRU or LSTM_PEEPHOLE
    num_layers: int
    bidirectional: int   # 0 or 1
    input_dim: int
    hidden: int
    num_classes: int
    n: int               # number of sequences
    batch: int           # mini-batch size B
    gemm_dtype: int      # FP32 or BF16 GEMM operands
    k_list: tuple        # bucket counts measured (1 = unbucketed baseline)
    law: str             # length law
    law_args: tuple


WORKLOADS = {
    "tiny": Workload("tiny", LSTM, 1, 0, 4, 32, 20, 64, 16, FP32, (1, 2),
                     "uniform", (10, 100)),
    "lstm2": Workload("lstm2", LSTM, 2, 0, 8, 128, 80, 4096, 64, FP32, (1, 8),
                      "lognormal", (300.0, 0.6, 20, 1500)),
    "bilstm3": Workload("bilstm3", LSTM, 3, 1, 8, 256, 80, 16384, 64, BF16, (1, 16),
                        "lognormal", (400.0, 0.7, 20, 2500)),
    "longtail": Workload("longtail", LSTM, 2, 0, 16, 512, 100, 8192, 128, BF16,
                         (1, 4, 16, 32), "pareto", (1.5, 50, 4000)),
    "gru2": Workload("gru2", GRU, 2, 0, 8, 384, 80, 16384, 96, FP32, (1, 8),
                     "lognormal", (300.0, 0.6, 20, 1500)),
    "lstm2p": Workload("lstm2p", LSTM_PEEPHOLE, 2, 0, 8, 128, 80, 4096, 64, FP32, (1, 8),
                       "lognormal", (300.0, 0.6, 20, 1500)),
}


def draw_lengths(rng: np.random.Generator, law: str, args: tuple, n: int) -> np.ndarray:
    """Sequence lengths (int32, all >= 1) drawn from one of the length laws."""
    if law == "uniform":
        lo, hi = args
        out = rng.integers(lo, hi + 1, n)
    elif law == "lognormal":
        median, sigma, lo, hi = args
        out = np.clip(np.rint(rng.lognormal(np.log(median), sigma, n)), lo, hi)
    elif law == "pareto":
        alpha, xm, hi = args
        # numpy's pareto() is the Lomax law; xm*(1+Lomax) is the classical Pareto.
        out = np.clip(np.floor(xm * (1.0 + rng.pareto(alpha, n))), xm, hi)
    else:
        raise ValueError(f"unknown length law {law!r}")
    return out.astype(np.int32)


@dataclasses.dataclass
class Data:
    lengths: np.ndarray   # int32 [n]
    offsets: np.ndarray   # int64 [n+1], row offsets of each sequence in X/Y
    X: np.ndarray         # float32 [sum(lengths), D]
    Y: np.ndarray         # int32 [sum(lengths)]
    params: Optional[np.ndarray]  # float32 [count] or None


def make_workload(w: Workload, seed: int = 0, param_count: Optional[int] = None,
                  n: Optional[int] = None) -> Data:
    """Draws the full synthetic data set of a workload (see module docstring)."""
    rng = np.random.default_rng(seed)
    nn = w.n if n is None else n
    lengths = draw_lengths(rng, w.law, w.law_args, nn)
    offsets = np.zeros(nn + 1, np.int64)
    np.cumsum(lengths, out=offsets[1:])
    U = int(offsets[-1])
    X = rng.standard_normal((U, w.input_dim), dtype=np.float32)
    Y = rng.integers(0, w.num_classes, U, dtype=np.int32)
    params = None
    if param_count is not None:
        params = rng.uniform(-0.1, 0.1, param_count).astype(np.float32)
    return Data(lengths, offsets, X, Y, params)


FRAMES_PER_LABEL = 8


def ctc_targets(lengths, C: int, seed: int = 0):
    """One label string per sequence (int32 arrays, classes 1..C-1)."""
    rng = np.random.default_rng([seed, 0xC7C])
    return [rng.integers(1, C, max(1, int(L) // FRAMES_PER_LABEL)).astype(np.int32)
            for L in lengths]


def shuffle_keys(seed: int, epoch: int, n: int) -> np.ndarray:
    """Per-sequence random keys (uint64) that order the sequences inside each
    bucket for one epoch (the paper reshuffles the data before every epoch)."""
    rng = np.random.default_rng([seed, 0x5EED, epoch])
    return rng.integers(0, np.iinfo(np.int64).max, n, dtype=np.int64).astype(np.uint64)


def random_lengths(seed: int, n: int, lo: int, hi: int) -> np.ndarray:
    """Uniform int32 lengths in [lo, hi] for planner tests."""
    return np.random.default_rng(seed).integers(lo, hi + 1, n).astype(np.int32)


def padded_batch(data: Data, order: np.ndarray, t_max: Optional[int] = None):
    """Gathers sequences ``order`` (already in the batch's row order) into the
    time-major padded layout X[T_max][B][D] (float32) and labels[T_max][B]
    (int32, -1 on pad frames).  Pad feature values are 0 unless the caller
    overwrites them; nothing here depends on the method."""
    lens = data.lengths[order]
    T = int(lens.max()) if t_max is None else t_max
    B = len(order)
    D = data.X.shape[1]
    x = np.zeros((T, B, D), np.float32)
    y = np.full((T, B), -1, np.int32)
    for b, s in enumerate(order):
        L = int(lens[b])
        o = int(data.offsets[s])
        x[:L, b, :] = data.X[o:o + L]
        y[:L, b] = data.Y[o:o + L]
    return x, y, lens.astype(np.int32)


def order_keys(seed: int, epoch: int, n: int) -> np.ndarray:
    """Random uint64 keys that rank buckets or batches for the randomised
    feeding orders (one stream per epoch, independent of the shuffle keys)."""
    rng = np.random.default_rng([seed, 0x0DE5, epoch])
    return rng.integers(0, np.iinfo(np.int64).max, n, dtype=np.int64).astype(np.uint64)
