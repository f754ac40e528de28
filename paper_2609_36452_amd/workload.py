"""Seeded synthetic inputs for the RPD commit step.

This module draws the arrays the commit step consumes (unembedding matrix,
hidden states of the final K layers, canvas mask) and nothing else: it holds
none of the method's arithmetic. Both the fp64 oracle and the HIP path are
fed from it, so both sides read identical, already-rounded values.

The paper's workloads are LLaDA-8B-Instruct and Dream-v0-Instruct-7B in bf16 on
a 256-position canvas at batch 1 (Section 4 setup; Appendix A.2 and A.5); the
trained weights and the benchmark prompts are not available, so seeded random
stand-ins with the same shapes are drawn here:

* ``W_U[v][:] ~ N(0, 1/d)`` (row norms close to 1);
* per masked position a target token ``t ~ U{0..V-1}`` and a sharpness ``s``;
  the hidden state of layer ``l`` is ``s*sqrt(d)*W_U[t_l]/||W_U[t_l]|| + N(0, I_d)``
  so that the target logit is about ``s*sqrt(d)`` while the other logits are
  about ``N(0, s^2 + 1)``;
* a fixed fraction of positions is "unstable": its target switches to another
  token ``t' = (t + U{1..V-1}) mod V`` at the final layer only;
* unmasked hidden rows are filled with NaN so that any read of them shows.

A supplementary "calibrated" mode places the target logit near a chosen level
``g`` (``h = g*W_U[t]/||W_U[t]||^2 + noise`` with a per-layer jitter of ``g``),
which populates the intermediate-confidence band that the stability test
governs; the graded workloads use the scaled mode above.

Rounding to bf16 is round-to-nearest-even of the fp64 value, done on the
integer bit pattern; bf16 arrays are returned as ``uint16`` bit patterns.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np

__all__ = [
    "WorkloadConfig",
    "CONFIGS",
    "Workload",
    "make_workload",
    "round_bf16_bits",
    "bf16_bits_to_f32",
    "draw_unembedding",
]

_W_CHUNK_ROWS = 4096  # W_U rows per independent random stream (fixes the draw
                      # regardless of how many threads fill it)


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    B: int
    L: int
    K: int
    d: int
    V: int
    dtype: str                      # "bf16" or "f32"
    masked_frac: float | None = None  # fraction of L masked per sequence
    n_masked: int | None = None       # or an exact count per sequence
    sharp: tuple = ("uniform", 0.0, 8.0)  # ("uniform", lo, hi) | ("ushape", smax) | ("calibrated"[, lo, hi])
    unstable_frac: float = 0.4
    layer_jitter: float = 0.5       # calibrated mode only: std of per-layer level jitter

    def masked_per_seq(self) -> int:
        if self.n_masked is not None:
            return int(self.n_masked)
        return int(round(self.masked_frac * self.L))

    def with_(self, **kw) -> "WorkloadConfig":
        return replace(self, **kw)


# Shapes of the paper's two backbones: LLaDA-8B (d=4096, V=126464) and
# Dream-7B (d=3584, V=152064), canvas of 256 positions, final K=4 layers.
CONFIGS: dict[str, WorkloadConfig] = {
    # small case that the oracle finishes in well under a second
    "tiny": WorkloadConfig("tiny", B=1, L=64, K=3, d=256, V=4096, dtype="f32",
                           n_masked=40, sharp=("uniform", 0.0, 8.0), unstable_frac=0.4),
    # late decoding: few masked positions, W_U streaming dominates
    "llada_late": WorkloadConfig("llada_late", B=1, L=256, K=4, d=4096, V=126464, dtype="bf16",
                                 n_masked=8, sharp=("uniform", 0.0, 12.0), unstable_frac=0.4),
    "llada_100": WorkloadConfig("llada_100", B=1, L=256, K=4, d=4096, V=126464, dtype="bf16",
                                masked_frac=1.0, sharp=("ushape", 12.0), unstable_frac=0.3),
    "llada_50": WorkloadConfig("llada_50", B=1, L=256, K=4, d=4096, V=126464, dtype="bf16",
                               masked_frac=0.5, sharp=("ushape", 12.0), unstable_frac=0.3),
    "llada_25": WorkloadConfig("llada_25", B=1, L=256, K=4, d=4096, V=126464, dtype="bf16",
                               masked_frac=0.25, sharp=("ushape", 12.0), unstable_frac=0.3),
    "llada_10": WorkloadConfig("llada_10", B=1, L=256, K=4, d=4096, V=126464, dtype="bf16",
                               masked_frac=0.1, sharp=("ushape", 12.0), unstable_frac=0.3),
    "dream_100": WorkloadConfig("dream_100", B=1, L=256, K=4, d=3584, V=152064, dtype="bf16",
                                masked_frac=1.0, sharp=("uniform", 0.0, 10.0), unstable_frac=0.3),
    "dream_50": WorkloadConfig("dream_50", B=1, L=256, K=4, d=3584, V=152064, dtype="bf16",
                               masked_frac=0.5, sharp=("uniform", 0.0, 10.0), unstable_frac=0.3),
    # batched code-generation shape: 8 sequences x 512 positions, 75% masked
    "llada_batched": WorkloadConfig("llada_batched", B=8, L=512, K=4, d=4096, V=126464, dtype="bf16",
                                    masked_frac=0.75, sharp=("ushape", 12.0), unstable_frac=0.3),
    # same at 32 sequences (about 49k projected rows)
    "llada_batched32": WorkloadConfig("llada_batched32", B=32, L=512, K=4, d=4096, V=126464, dtype="bf16",
                                      masked_frac=0.75, sharp=("ushape", 12.0), unstable_frac=0.3),
}


@dataclass
class Workload:
    cfg: WorkloadConfig
    seed: int
    w_u: np.ndarray          # [V][d] uint16 (bf16 bits) or float32
    hidden: np.ndarray       # [K][B][L][d] same dtype as w_u
    mask: np.ndarray         # [B][L] uint8, 1 = masked
    targets: np.ndarray      # [B][L] int64, -1 unmasked (final-layer target)
    meta: dict = field(default_factory=dict)

    @property
    def n_masked(self) -> int:
        return int(self.mask.sum())


# ---------------------------------------------------------------- rounding --

def round_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 (nearest, ties to even); return uint16 bits.

    bf16 keeps 8 significant bits, so the fp64 significand is rounded at its
    bit 45; the rounded value is then exactly a float32 whose top half is the
    bf16 pattern. NaN inputs stay NaN (quiet, positive)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    nan = np.isnan(x)
    b = x.view(np.uint64)
    lsb = (b >> np.uint64(45)) & np.uint64(1)
    b = (b + (np.uint64((1 << 44) - 1) + lsb)) & np.uint64(~((1 << 45) - 1) & 0xFFFFFFFFFFFFFFFF)
    r = b.view(np.float64).astype(np.float32)
    out = (r.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _round(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_bf16_bits(x)
    if dtype == "f32":
        return x.astype(np.float32)
    raise ValueError(dtype)


def _as_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return bf16_bits_to_f32(a).astype(np.float64)
    return a.astype(np.float64)


# ------------------------------------------------------------------ drawing --

def _gen(*key) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


_W_CACHE: dict = {}


def draw_unembedding(V: int, d: int, dtype: str, seed: int, cache: bool = True) -> np.ndarray:
    """W_U[v][k] ~ N(0, 1/d), rounded to ``dtype``; rows drawn in fixed chunks
    from independent streams so the result does not depend on thread count."""
    key = (V, d, dtype, seed)
    if cache and key in _W_CACHE:
        return _W_CACHE[key]
    out = np.empty((V, d), dtype=np.uint16 if dtype == "bf16" else np.float32)
    scale = 1.0 / math.sqrt(d)
    nchunks = (V + _W_CHUNK_ROWS - 1) // _W_CHUNK_ROWS

    def fill(c: int) -> None:
        r0 = c * _W_CHUNK_ROWS
        r1 = min(V, r0 + _W_CHUNK_ROWS)
        z = _gen(seed, 1, c).standard_normal((r1 - r0, d), dtype=np.float32)
        out[r0:r1] = _round(z.astype(np.float64) * scale, dtype)

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fill, range(nchunks)))
    if cache:
        _W_CACHE.clear()  # keep at most one large matrix alive
        _W_CACHE[key] = out
    return out


def _sharpness(cfg: WorkloadConfig, g: np.random.Generator, pos: np.ndarray) -> np.ndarray:
    kind = cfg.sharp[0]
    if kind == "uniform":
        return g.uniform(cfg.sharp[1], cfg.sharp[2], size=pos.size)
    if kind == "ushape":
        # rising toward both canvas ends: s = smax * u^2 * xi, u in [-1, 1]
        u = 2.0 * pos / max(cfg.L - 1, 1) - 1.0
        return cfg.sharp[1] * u * u * g.uniform(0.5, 1.0, size=pos.size)
    if kind == "calibrated":
        # target-logit level spanning low to saturated confidence (by default
        # ln V - 3 to ln V + 6; ("calibrated", lo, hi) sets the offsets)
        lnv = math.log(cfg.V)
        lo, hi = (cfg.sharp[1], cfg.sharp[2]) if len(cfg.sharp) == 3 else (-3.0, 6.0)
        return g.uniform(lnv + lo, lnv + hi, size=pos.size)
    raise ValueError(kind)


def make_workload(cfg: WorkloadConfig | str, seed: int, w_u: np.ndarray | None = None) -> Workload:
    """Draw one seeded instance of ``cfg``.

    Draw order (each from its own stream keyed on ``seed``): W_U (stream 1);
    per sequence b the masked positions, targets, sharpness, unstable subset
    and switched targets (stream 2, b); per layer and sequence the noise
    (stream 3, l, b); calibrated mode's per-layer jitter (stream 4, b)."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    K, B, L, d, V = cfg.K, cfg.B, cfg.L, cfg.d, cfg.V
    nm = cfg.masked_per_seq()
    if not 0 <= nm <= L:
        raise ValueError("masked count out of range")
    if w_u is None:
        w_u = draw_unembedding(V, d, cfg.dtype, seed)
    mask = np.zeros((B, L), np.uint8)
    targets = np.full((B, L), -1, np.int64)
    hid_dtype = np.uint16 if cfg.dtype == "bf16" else np.float32
    hidden = np.empty((K, B, L, d), hid_dtype)
    hidden[...] = np.uint16(0x7FC0) if cfg.dtype == "bf16" else np.float32(np.nan)
    calibrated = cfg.sharp[0] == "calibrated"
    sqrt_d = math.sqrt(d)
    per_seq = []
    for b in range(B):
        g = _gen(seed, 2, b)
        pos = np.sort(g.choice(L, size=nm, replace=False)).astype(np.int64)
        t = g.integers(0, V, size=nm)
        s = _sharpness(cfg, g, pos)
        n_unst = int(round(cfg.unstable_frac * nm))
        unst = np.zeros(nm, bool)
        unst[g.choice(nm, size=n_unst, replace=False)] = True
        t_sw = (t + g.integers(1, V, size=nm)) % V
        jit = _gen(seed, 4, b).normal(0.0, cfg.layer_jitter, size=(K, nm)) if calibrated else None
        mask[b, pos] = 1
        t_final = np.where(unst, t_sw, t)
        targets[b, pos] = t_final
        per_seq.append((pos, t, t_sw, unst, s, jit))

    def fill(job):
        l, b = job
        pos, t, t_sw, unst, s, jit = per_seq[b]
        if pos.size == 0:
            return
        tl = np.where(unst, t_sw, t) if l == K - 1 else t
        wt = _as_f64(w_u[tl], cfg.dtype)                       # [n][d] rounded rows
        nrm2 = np.einsum("ij,ij->i", wt, wt)
        if calibrated:
            lvl = s + jit[l]
            dirn = wt * (lvl / nrm2)[:, None]
        else:
            dirn = wt * (s * sqrt_d / np.sqrt(nrm2))[:, None]
        noise = _gen(seed, 3, l, b).standard_normal((pos.size, d), dtype=np.float32)
        hidden[l, b, pos] = _round(dirn + noise.astype(np.float64), cfg.dtype)

    jobs = [(l, b) for l in range(K) for b in range(B)]
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fill, jobs))
    meta = {"unstable": [ps[3] for ps in per_seq], "sharpness": [ps[4] for ps in per_seq]}
    return Workload(cfg=cfg, seed=seed, w_u=w_u, hidden=hidden, mask=mask, targets=targets, meta=meta)
