"""Shared helpers of the GPU tests: move a seeded workload to the device, run
the HIP path through the C ABI, run the oracle on the same arrays."""
from __future__ import annotations

import dataclasses
import sys

import numpy as np
import torch

import oracle as O
from paper_2609_36452_amd import binding as rpd


def note(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(w, dev="cuda:0"):
    if w.cfg.dtype == "bf16":
        hidden = torch.from_numpy(w.hidden).view(torch.bfloat16).to(dev)
        w_u = torch.from_numpy(w.w_u).view(torch.bfloat16).to(dev)
    else:
        hidden = torch.from_numpy(w.hidden).to(dev)
        w_u = torch.from_numpy(w.w_u).to(dev)
    mask = torch.from_numpy(w.mask).to(dev)
    return hidden, w_u, mask


def gpu_params(P: O.Params) -> rpd.Params:
    return rpd.Params(**dataclasses.asdict(P))


def run_gpu(w, P: O.Params, layer_stats=True, max_masked="exact", tensors=None) -> dict:
    hidden, w_u, mask = tensors if tensors is not None else to_device(w)
    mm = w.n_masked if max_masked == "exact" else max_masked
    note(f"  gpu call: {w.cfg.name} K={w.cfg.K} B={w.cfg.B} L={w.cfg.L} d={w.cfg.d} V={w.cfg.V} "
         f"dtype={w.cfg.dtype} n={w.n_masked} seed={w.seed} max_masked={mm}")
    out = rpd.score_commit(hidden, w_u, mask, gpu_params(P), max_masked=mm, layer_stats=layer_stats)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


_LAYER_CACHE: dict = {}


def run_oracle(w, P: O.Params) -> dict:
    """Oracle outputs; the per-layer projection of a workload is computed once
    and reused across parameter sets."""
    key = id(w)
    if key not in _LAYER_CACHE or _LAYER_CACHE[key][0] is not w:
        _LAYER_CACHE.clear()
        _LAYER_CACHE[key] = (w, O.layer_stats_masked(w.hidden, w.w_u, w.mask, w.cfg.dtype))
    pos, layer = _LAYER_CACHE[key][1]
    return O.assemble(w.mask, pos, layer, P)
