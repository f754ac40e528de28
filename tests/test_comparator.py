"""The parity comparator itself, on the CPU: it accepts the oracle's own
outputs (in the GPU's output types) and rejects each kind of planted mistake;
an exact argmax tie is never excused, a near-tie below the accumulation bound
is. Also pins the oracle's near-tie diagnostics (top-2 gap and sum |W x|)
against brute force."""
import dataclasses
import math

import numpy as np
import pytest

import oracle as O
from paper_2609_36452_amd.workload import CONFIGS, make_workload
from tests.parity import F_CAND, F_FALLBACK, as_gpu_outputs, compare, gap_tol, near_tie


def _oracle(w, P):
    pos, layer = O.layer_stats_masked(w.hidden, w.w_u, w.mask, w.cfg.dtype, logit_scale=P.logit_scale)
    return O.assemble(w.mask, pos, layer, P)


@pytest.fixture(scope="module")
def case():
    w = make_workload(CONFIGS["tiny"].with_(sharp=("calibrated",), unstable_frac=0.3, B=2), 5)
    P = O.LLADA
    return w, P, _oracle(w, P)


@pytest.fixture(scope="module")
def fallback_case():
    # no candidate at all (theta_h above every confidence, beta = 0): every sequence falls back
    w = make_workload(CONFIGS["tiny"].with_(sharp=("calibrated", -3.0, 0.0), unstable_frac=0.3), 6)
    P = O.Params(theta_h=0.999999, theta_c=0.999998, beta=0.0)
    o = _oracle(w, P)
    assert all((o["flags"][b] & F_FALLBACK).any() for b in range(w.cfg.B))
    return w, P, o


def _run(w, P, o, g):
    return compare(g, o, w.mask, P, w.cfg.d)


def test_accepts_the_oracle_itself(case, fallback_case):
    for w, P, o in (case, fallback_case):
        rep = _run(w, P, o, as_gpu_outputs(o))
        assert rep.ok(), rep.summary()
        assert not rep.excused, rep.summary()


def _pick(w, o, pred):
    """First masked position (b, i) satisfying pred(b, i)."""
    for b, i in zip(*np.nonzero(w.mask)):
        if pred(int(b), int(i)):
            return int(b), int(i)
    raise AssertionError("no position fits")


def _clear(o, d):
    """Not a near-tie at any layer, confidence away from the thresholds."""
    tie = near_tie(o["layer_gap"], o["layer_absbound"], d).any(0)
    return lambda b, i: (not tie[b, i] and o["layer_gap"][:, b, i].min() > 1e-3
                         and min(abs(o["confidence"][b, i] - 0.9), abs(o["confidence"][b, i] - 0.6)) > 0.01)


PLANTS = ["token", "layer_argmax", "entropy", "confidence", "layer_entropy", "layer_conf", "persistence",
          "drop", "candidate_flag", "commit", "n_commit", "upstream_entropy", "sentinel", "committed_bit",
          "nan_entropy", "nan_layer_conf"]


@pytest.mark.parametrize("what", PLANTS)
def test_rejects_planted_mistake(case, what):
    w, P, o = case
    g = as_gpu_outputs(o)
    K = w.cfg.K
    b, i = _pick(w, o, _clear(o, w.cfg.d))
    if what == "token":
        g["token"][b, i] = (g["token"][b, i] + 1) % w.cfg.V
        g["layer_argmax"][K - 1, b, i] = g["token"][b, i]
    elif what == "layer_argmax":
        g["layer_argmax"][0, b, i] = (g["layer_argmax"][0, b, i] + 7) % w.cfg.V
    elif what == "entropy":
        g["entropy"][b, i] += 2.5e-3
    elif what == "confidence":
        g["confidence"][b, i] += 1.5e-3
    elif what == "layer_entropy":
        g["layer_entropy"][1, b, i] -= 2.5e-3
    elif what == "layer_conf":
        g["layer_conf"][0, b, i] -= 1.5e-3
    elif what == "persistence":
        g["persistence"][b, i] = g["persistence"][b, i] % K + 1
    elif what == "drop":
        g["drop"][b, i] += 0.05
    elif what == "candidate_flag":
        g["flags"][b, i] ^= F_CAND
    elif what == "commit":
        g["commit"][b, i] ^= 1
    elif what == "n_commit":
        g["n_commit"][b] += 1
    elif what == "upstream_entropy":
        bb, ii = _pick(w, o, lambda b_, i_: o["upstream_entropy"][b_, i_] > 0.1)
        g["upstream_entropy"][bb, ii] += 0.01
    elif what == "sentinel":
        bb, ii = map(int, np.argwhere(w.mask == 0)[0])
        g["token"][bb, ii] = 3
    elif what == "committed_bit":
        g["flags"][b, i] ^= 8
    elif what == "nan_entropy":
        g["entropy"][b, i] = np.nan
    elif what == "nan_layer_conf":
        g["layer_conf"][0, b, i] = np.nan
    rep = _run(w, P, o, g)
    assert not rep.ok(), f"{what} planted at {(b, i)} was accepted: {rep.summary()}"


def test_rejects_moved_fallback(fallback_case):
    w, P, o = fallback_case
    g = as_gpu_outputs(o)
    b = 0
    idx = np.nonzero(w.mask[b])[0]
    fo = int(np.nonzero(o["flags"][b, idx] & F_FALLBACK)[0][0])
    win = idx[:P.window]
    c = o["confidence"][b, win]
    # the least confident position of the window, clearly below the chosen one
    q = int(np.argmin(c))
    assert c[fo] - c[q] > 0.01
    g["commit"][b, idx[fo]] = 0
    g["flags"][b, idx[fo]] &= ~np.uint8(F_FALLBACK | 8)
    g["commit"][b, idx[q]] = 1
    g["flags"][b, idx[q]] |= np.uint8(F_FALLBACK | 8)
    rep = _run(w, P, o, g)
    assert not rep.ok(), rep.summary()


def test_rejects_fallback_on_one_side_only(fallback_case):
    # the GPU commits a non-fallback position in a sequence where the oracle falls back
    w, P, o = fallback_case
    g = as_gpu_outputs(o)
    b = 0
    idx = np.nonzero(w.mask[b])[0]
    fo = int(np.nonzero(o["flags"][b, idx] & F_FALLBACK)[0][0])
    g["flags"][b, idx[fo]] &= ~np.uint8(F_FALLBACK)
    rep = _run(w, P, o, g)
    assert not rep.ok(), rep.summary()


# -------------------------------------------------------------- argmax ties --

def _two_row_case(delta: float):
    """One masked position, K = 2, f32: x = e_0 and W_U rows 3 and 5 whose
    first entries differ by ``delta`` (relative); every other row far below."""
    K, B, L, d, V = 2, 1, 2, 8, 16
    w_u = np.zeros((V, d), np.float32)
    w_u[:, 1] = np.linspace(-1.0, -0.5, V, dtype=np.float32)
    w_u[5, 0] = 4.0
    w_u[3, 0] = np.float32(4.0 * (1.0 - delta))
    hidden = np.full((K, B, L, d), np.nan, np.float32)
    hidden[:, 0, 0] = 0.0
    hidden[:, 0, 0, 0] = 1.0
    mask = np.array([[1, 0]], np.uint8)
    return hidden, w_u, mask


def test_exact_tie_is_never_excused():
    # rows 3 and 5 identical: the oracle's argmax is the lower index with a gap of exactly 0 at every
    # layer; a GPU reporting the higher index is wrong, not excused
    hidden, w_u, mask = _two_row_case(0.0)
    P = O.Params(theta_s=1.0, w=1.0)
    o = O.score_commit(hidden, w_u, mask, "f32", P)
    assert o["token"][0, 0] == 3 and (o["layer_gap"][:, 0, 0] == 0.0).all()
    g = as_gpu_outputs(o)
    assert compare(g, o, mask, P, 8).ok()
    g["token"][0, 0] = 5
    g["layer_argmax"][:, 0, 0] = 5
    rep = compare(g, o, mask, P, 8)
    assert not rep.ok() and not rep.excused, rep.summary()


def test_near_tie_below_the_bound_is_excused():
    # rows 3 and 5 one float32 ulp apart: a positive gap below 4 (d+1) 2^-24 max|W x|
    hidden, w_u, mask = _two_row_case(2.0 ** -23)
    P = O.Params(theta_s=1.0, w=1.0)
    o = O.score_commit(hidden, w_u, mask, "f32", P)
    gap = o["layer_gap"][:, 0, 0]
    assert o["token"][0, 0] == 5 and (gap > 0).all() and (gap < gap_tol(8, o["layer_absbound"][:, 0, 0])).all()
    g = as_gpu_outputs(o)
    g["token"][0, 0] = 3
    g["layer_argmax"][:, 0, 0] = 3
    rep = compare(g, o, mask, P, 8)
    assert rep.ok(), rep.summary()
    assert rep.excused["argmax_tie"] == 2 and rep.excused["token_tie"] == 1


def test_intermediate_tie_does_not_excuse_a_token_mismatch():
    # a near-tie at an intermediate layer only: the final-layer token must still match exactly
    hidden, w_u, mask = _two_row_case(2.0 ** -23)
    hidden[1, 0, 0, 0] = 1.0
    hidden[1, 0, 0, 2] = 1.0
    w_u[3, 2] = 1.0          # at the final layer row 3 now wins clearly
    P = O.Params(theta_s=1.0, w=1.0)
    o = O.score_commit(hidden, w_u, mask, "f32", P)
    tie = near_tie(o["layer_gap"], o["layer_absbound"], 8)[:, 0, 0]
    assert tie[0] and not tie[1] and o["token"][0, 0] == 3
    g = as_gpu_outputs(o)
    g["token"][0, 0] = 5
    g["layer_argmax"][1, 0, 0] = 5
    assert not compare(g, o, mask, P, 8).ok()


def _nan_row_case():
    # the tie case's position with one NaN hidden element at every layer: every logit is NaN
    hidden, w_u, mask = _two_row_case(0.5)
    hidden[:, 0, 0, 3] = np.nan
    P = O.Params(theta_s=1.0, w=1.0)
    return O.score_commit(hidden, w_u, mask, "f32", P), mask, P


def test_nan_row_has_no_argmax_to_compare():
    o, mask, P = _nan_row_case()
    assert np.isnan(o["layer_entropy"][:, 0, 0]).all() and np.isnan(o["entropy"][0, 0])
    g = as_gpu_outputs(o)
    g["layer_argmax"][:, 0, 0] = -1       # the GPU finds no ordered maximum in such a row
    g["token"][0, 0] = -1
    rep = compare(g, o, mask, P, 8)
    assert rep.ok(), rep.summary()


def test_nan_row_must_stay_nan_and_not_a_candidate():
    o, mask, P = _nan_row_case()
    g = as_gpu_outputs(o)
    g["layer_entropy"][0, 0, 0] = 0.5
    assert not compare(g, o, mask, P, 8).ok()
    g = as_gpu_outputs(o)
    g["flags"][0, 0] |= F_CAND
    assert not compare(g, o, mask, P, 8).ok()


# ------------------------------------------------- near-tie diagnostics pin --

def test_gap_and_absbound_against_brute_force():
    w = make_workload(CONFIGS["tiny"].with_(V=97, d=16, L=6, n_masked=3, K=2), 11)
    pos = O.masked_positions(w.mask)
    st = O.project_layer_stats(w.hidden, w.w_u, w.cfg.dtype, pos)
    W = w.w_u.astype(np.float64)
    for a, (b, i) in enumerate(pos):
        for l in range(w.cfg.K):
            x = w.hidden[l, b, i].astype(np.float64)
            z = [math.fsum(W[v, k] * x[k] for k in range(w.cfg.d)) for v in range(w.cfg.V)]
            order = sorted(range(w.cfg.V), key=lambda v: (-z[v], v))
            top, second = order[0], order[1]
            A = [math.fsum(abs(W[v, k] * x[k]) for k in range(w.cfg.d)) for v in (top, second)]
            assert st["argmax"][a, l] == top
            assert st["gap"][a, l] == pytest.approx(z[top] - z[second], rel=1e-12, abs=1e-12)
            assert st["absbound"][a, l] == pytest.approx(max(A), rel=1e-12)
