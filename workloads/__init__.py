"""Seeded synthetic workloads for the pruned RNN-T loss.

This module only draws random arrays of the right shapes and distributions.
It holds none of the loss arithmetic, so both the CPU oracle's tests and the
GPU path's tests and benchmark can take their inputs from here without
sharing any computation.

The five workloads mirror the shapes the paper benchmarks on (LibriSpeech
test-clean utterances, a 500-token BPE vocabulary, Sec. 4.1), plus a larger
character vocabulary (the motivation in Sec. 1) and a long-utterance stress
case. The dataset itself is not used: lengths are drawn uniformly in the
stated ranges and every value is synthetic.

Draw order (fixed, so that a seed names one batch): t_len, u_len, the
"U close to T/3" override (stress only), symbols, am, lm, enc, dec, W.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = ["Workload", "WORKLOADS", "make_batch", "round_to_bf16", "Batch"]


@dataclass(frozen=True)
class Workload:
    name: str
    N: int
    T_range: tuple          # inclusive (lo, hi) for per-utterance frame counts
    U_range: tuple          # inclusive (lo, hi) for per-utterance token counts
    V: int
    S: int
    J: int
    joiner_dtype: str       # "f32" or "bf16" for enc, dec, W, bias
    symbols: str = "uniform"  # "uniform" on [1, V-1] or "zipf1.1"
    u_third_frac: float = 0.0  # fraction of utterances with U_n = floor(T_n/3)
    blank: int = 0
    seed: int = 0


WORKLOADS = {
    "tiny": Workload("tiny", N=2, T_range=(20, 20), U_range=(5, 5), V=16, S=4, J=32,
                     joiner_dtype="f32"),
    "bpe": Workload("bpe", N=16, T_range=(150, 250), U_range=(20, 60), V=500, S=5, J=512,
                    joiner_dtype="f32"),
    "long": Workload("long", N=32, T_range=(300, 500), U_range=(50, 100), V=500, S=5, J=512,
                     joiner_dtype="bf16"),
    "largev": Workload("largev", N=16, T_range=(200, 300), U_range=(40, 80), V=5000, S=5, J=512,
                       joiner_dtype="f32", symbols="zipf1.1"),
    "stress": Workload("stress", N=8, T_range=(800, 1000), U_range=(200, 300), V=8000, S=10, J=768,
                       joiner_dtype="bf16", u_third_frac=0.25),
}


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bfloat16 (ties to even); return fp32.

    NaN stays NaN. The result holds only bf16-representable values, so a
    later conversion to a bf16 tensor is exact.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    out = rounded.view(np.float32).copy()
    nan = np.isnan(x)
    out[nan] = np.nan
    return out


@dataclass
class Batch:
    """One synthetic batch. All arrays are host numpy arrays."""
    wl: Workload
    t_len: np.ndarray        # [N] int32
    u_len: np.ndarray        # [N] int32
    symbols: np.ndarray      # [N, U] int32, symbols[n, u] = y_{u+1}
    am: np.ndarray           # [N, T, V] float32
    lm: np.ndarray           # [N, U+1, V] float32
    enc: np.ndarray          # [N, T, J] float32 (bf16-representable if joiner_dtype == bf16)
    dec: np.ndarray          # [N, U+1, J]
    W: np.ndarray            # [J, V]
    bias: np.ndarray         # [V]
    extra: dict = field(default_factory=dict)

    @property
    def N(self):
        return self.am.shape[0]

    @property
    def T(self):
        return self.am.shape[1]

    @property
    def U(self):
        return self.lm.shape[1] - 1

    @property
    def V(self):
        return self.am.shape[2]

    @property
    def frames(self) -> int:
        return int(self.t_len.sum())


def _zipf_symbols(rng, V, size, s=1.1):
    k = np.arange(1, V, dtype=np.float64)
    p = k ** (-s)
    p /= p.sum()
    return rng.choice(np.arange(1, V), size=size, p=p).astype(np.int32)


def make_batch(wl: Workload | str, seed: Optional[int] = None, *, N: Optional[int] = None,
               T_range=None, U_range=None, V=None, J=None, S=None,
               with_joiner: bool = True) -> Batch:
    """Draw one batch for a workload (optionally overriding sizes for tests)."""
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    over = {}
    for k, v in (("N", N), ("T_range", T_range), ("U_range", U_range), ("V", V), ("J", J), ("S", S)):
        if v is not None:
            over[k] = v
    if over:
        wl = Workload(**{**wl.__dict__, **over})
    rng = np.random.default_rng(wl.seed if seed is None else seed)
    Nb = wl.N
    t_len = rng.integers(wl.T_range[0], wl.T_range[1], endpoint=True, size=Nb).astype(np.int32)
    u_len = rng.integers(wl.U_range[0], wl.U_range[1], endpoint=True, size=Nb).astype(np.int32)
    if wl.u_third_frac > 0:
        k = int(np.ceil(Nb * wl.u_third_frac))
        pick = rng.choice(Nb, size=k, replace=False)
        u_len[pick] = t_len[pick] // 3
    T = int(t_len.max())
    U = int(u_len.max())
    if wl.symbols == "zipf1.1":
        symbols = _zipf_symbols(rng, wl.V, (Nb, max(U, 1)))
    else:
        symbols = rng.integers(1, wl.V, size=(Nb, max(U, 1))).astype(np.int32)
    symbols = np.ascontiguousarray(symbols[:, :U]) if U > 0 else np.zeros((Nb, 0), np.int32)
    am = rng.standard_normal((Nb, T, wl.V), dtype=np.float32)
    lm = rng.standard_normal((Nb, U + 1, wl.V), dtype=np.float32)
    if with_joiner:
        enc = rng.standard_normal((Nb, T, wl.J), dtype=np.float32)
        dec = rng.standard_normal((Nb, U + 1, wl.J), dtype=np.float32)
        W = (rng.standard_normal((wl.J, wl.V), dtype=np.float32) / np.float32(np.sqrt(wl.J))).astype(np.float32)
    else:
        enc = np.zeros((Nb, T, wl.J), np.float32)
        dec = np.zeros((Nb, U + 1, wl.J), np.float32)
        W = np.zeros((wl.J, wl.V), np.float32)
    bias = np.zeros((wl.V,), np.float32)
    if wl.joiner_dtype == "bf16":
        enc, dec, W, bias = (round_to_bf16(a) for a in (enc, dec, W, bias))
    return Batch(wl=wl, t_len=t_len, u_len=u_len, symbols=symbols, am=am, lm=lm,
                 enc=enc, dec=dec, W=W, bias=bias)
