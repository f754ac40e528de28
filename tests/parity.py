"""Element-by-element comparison of the HIP path with the fp64 oracle.

Contract (floating point): per masked position and per layer, entropy within
2e-3 nats and top probability within 1e-3 (bf16 inputs, fp32 accumulation).
Integer results (argmax, token, persistence, candidacy, commit, fallback
choice, counts) must be bit-exact, except where the exact answer is decided
by a margin smaller than the arithmetic can resolve; such differences are
counted by class and not treated as mismatches:

1. argmax near-tie: oracle top-2 logit gap g with 0 < g < 4 (d+1) u max(A_1, A_2),
   ``A_v = sum_k |W_U[v,k] x_k|``, u = 2^-24 -- twice the worst-case bound of
   fp32 accumulation in any order, leaving room for the matrix cores'
   internal rounding. An exact tie (g = 0, e.g. duplicated W_U rows) is
   never excused: the lowest vocabulary index must win, as in the oracle. A
   token (final-layer argmax) difference is excused only by a final-layer
   near-tie; persistence only by a near-tie at some layer;
2. threshold near-tie: oracle confidence within 1e-3 of theta_h or theta_c;
3. stability near-tie: oracle S_i within w * 2e-3 of theta_s (r_i is a
   difference of two probabilities, each within 1e-3);
4. budget near-tie: oracle prefix N_i within 1e-4 + fp32 scan rounding + the
   sum of the entropy errors over the earlier masked non-candidates (+ the
   entropy of earlier positions whose candidacy was itself excused) of beta;
5. cascade: a commit difference at or after a position whose candidacy
   differs under classes 1-3;
6. fallback near-tie: both sides fell back and the GPU's choice has an oracle
   confidence within 2e-3 of the oracle's choice (each side within 1e-3);
   a fallback on one side only is excused only as the consequence of
   excused differences in the budget decisions before it.

Independently of the oracle, the GPU's commitment must be exactly the
commitment rule applied (in float64, by the oracle's own scan) to the GPU's
own candidate flags, entropies and confidences -- the "conditioned oracle";
only a decision within fp32 scan rounding of beta may differ there. Its
candidate flags must follow exactly from its own confidence and stability in
float32, its persistence from its own per-layer argmaxes.
"""
from __future__ import annotations

from collections import Counter

import numpy as np

import oracle as O

ENTROPY_TOL = 2e-3
CONF_TOL = 1e-3
U = 2.0 ** -24

F_CAND, F_HIGH, F_STAB, F_COMMIT, F_FALLBACK = 1, 2, 4, 8, 16


def gap_tol(d: int, absbound):
    return 4.0 * (d + 1) * U * np.asarray(absbound)


def near_tie(gap, absbound, d: int):
    """Argmax near-tie: a positive oracle gap below the accumulation bound. A
    gap of exactly 0 is an exact tie, which the lowest-index rule decides."""
    gap = np.asarray(gap)
    with np.errstate(invalid="ignore"):
        return np.nan_to_num((gap > 0.0) & (gap < gap_tol(d, absbound)), nan=False).astype(bool)


class Report:
    def __init__(self):
        self.fail: list[str] = []
        self.excused = Counter()
        self.checked = Counter()

    def bad(self, msg: str):
        if len(self.fail) < 40:
            self.fail.append(msg)
        elif self.fail[-1] != "...":
            self.fail.append("...")

    def ok(self) -> bool:
        return not self.fail

    def summary(self) -> str:
        return f"checked={dict(self.checked)} excused={dict(self.excused)} failures={self.fail[:20]}"


def _flags_f32(c, s, P) -> np.ndarray:
    """Eq. 5 route bits evaluated in float32 on the GPU's own values."""
    c = np.asarray(c, np.float32)
    s = np.asarray(s, np.float32)
    th, tc, ts = np.float32(P.theta_h), np.float32(P.theta_c), np.float32(P.theta_s)
    with np.errstate(invalid="ignore"):
        high = c >= th
        stab = (c >= tc) & (c < th) & (s >= ts)
    return ((high | stab) * F_CAND | high * F_HIGH | stab * F_STAB).astype(np.uint8)


def _persistence_from_layers(ya: np.ndarray) -> int:
    """Eq. 2 on the GPU's own per-layer argmaxes (unprojected layers hold -1)."""
    return O.persistence(list(ya))


def conditioned(idx: np.ndarray, H: np.ndarray, cand: np.ndarray, c: np.ndarray, P) -> dict:
    """The oracle's commitment (Section 3.2, or RPD-block) run in float64 on
    given candidate flags, entropies and confidences of one sequence."""
    H = np.asarray(H, np.float64)
    c = np.asarray(c, np.float64)
    cand = np.asarray(cand, bool)
    if getattr(P, "block", 0) > 0:
        r = O.commit_block(idx, H, cand, c, P.block)
        r["N"] = np.zeros(len(H))
        return r
    r = O.commit_scan(H, cand, c, P)
    r["N"] = O.commit_closed_form(H, cand, P)["N"]
    return r


def compare(g: dict, o: dict, mask: np.ndarray, P, d: int, layer: bool = True) -> Report:
    """g: GPU outputs as numpy; o: oracle outputs (oracle.score_commit or
    score_commit_lazy, with the per-layer diagnostics)."""
    rep = Report()
    B, L = mask.shape
    K = o["layer_argmax"].shape[0]
    m = mask != 0
    block = getattr(P, "block", 0)
    # unmasked sentinels
    for name, val in (("commit", 0), ("token", -1), ("persistence", 0), ("flags", 0), ("entropy", 0.0),
                      ("confidence", 0.0), ("drop", 0.0), ("stability", 0.0), ("upstream_entropy", 0.0)):
        if np.any(g[name][~m] != val):
            rep.bad(f"unmasked sentinel {name}")
    tie = near_tie(o["layer_gap"], o["layer_absbound"], d) & m[None]    # [K][B][L]
    tie_final = tie[K - 1]
    tie_any = tie.any(0)
    # lazy projection: which intermediate layers exist depends on band membership (confidence next to
    # theta_c / theta_h) and on each layer's agreement (argmax near-ties); such positions are excused
    # from the per-layer and persistence comparisons
    lazy = bool(getattr(P, "lazy", False))
    lazy_all = bool(getattr(P, "lazy_all", False))
    lazy_excuse = np.zeros((B, L), bool)
    if lazy:
        c_o = o["confidence"]
        near_band = (np.abs(c_o - P.theta_c) <= CONF_TOL) | (np.abs(c_o - P.theta_h) <= CONF_TOL)
        lazy_excuse = m & ((near_band & (not lazy_all)) | tie_any)
    # per-layer statistics
    if layer:
        for l in range(K):
            gy, oy = g["layer_argmax"][l], o["layer_argmax"][l]
            gc, oc = g["layer_conf"][l], o["layer_conf"][l]
            gh, oh = g["layer_entropy"][l], o["layer_entropy"][l]
            for b, i in zip(*np.nonzero(m)):
                rep.checked["layer"] += 1
                issues = []
                nan_row = bool(np.isnan(oh[b, i]))
                if nan_row:
                    # a distribution with undefined entries: both statistics NaN, no argmax to compare
                    if not (np.isnan(gh[b, i]) and np.isnan(gc[b, i])):
                        issues.append(f"NaN row not NaN on GPU at l={l} b={b} i={i}")
                else:
                    if not abs(gh[b, i] - oh[b, i]) <= ENTROPY_TOL:
                        issues.append(f"entropy l={l} b={b} i={i}: gpu {gh[b, i]:.6g} oracle {oh[b, i]:.6g}")
                    if not abs(gc[b, i] - oc[b, i]) <= CONF_TOL:
                        issues.append(f"conf l={l} b={b} i={i}: gpu {gc[b, i]:.6g} oracle {oc[b, i]:.6g}")
                argmax_differs = (not nan_row) and gy[b, i] != oy[b, i]
                if not issues and not argmax_differs:
                    continue
                if lazy_excuse[b, i] and l < K - 1:
                    # which intermediate layers a lazy walk reaches depends on a near-tie here
                    rep.excused["lazy_layer"] += 1
                    continue
                for msg in issues:
                    rep.bad(msg)
                if argmax_differs:
                    if tie[l, b, i]:
                        rep.excused["argmax_tie"] += 1
                    else:
                        rep.bad(f"argmax l={l} b={b} i={i}: gpu {gy[b, i]} oracle {oy[b, i]} "
                                f"gap {o['layer_gap'][l][b, i]:.3g}")
    nan_pos = np.isnan(o["entropy"]) & m
    # per-position scoring
    cand_excused = np.zeros((B, L), bool)
    gflags_expect = _flags_f32(g["confidence"], g["stability"], P)
    for b, i in zip(*np.nonzero(m)):
        rep.checked["position"] += 1
        if nan_pos[b, i]:
            if g["flags"][b, i] & F_CAND:
                rep.bad(f"NaN position b={b} i={i} became a candidate")
            continue
        for name, tol in (("entropy", ENTROPY_TOL), ("confidence", CONF_TOL)):
            if not abs(g[name][b, i] - o[name][b, i]) <= tol:     # a NaN on the GPU side fails too
                rep.bad(f"{name} b={b} i={i}: gpu {g[name][b, i]:.6g} oracle {o[name][b, i]:.6g}")
        if g["token"][b, i] != o["token"][b, i]:
            if tie_final[b, i]:
                rep.excused["token_tie"] += 1
            else:
                rep.bad(f"token b={b} i={i}: gpu {g['token'][b, i]} oracle {o['token'][b, i]}")
        if layer and g["persistence"][b, i] >= 0 and \
                g["persistence"][b, i] != _persistence_from_layers(g["layer_argmax"][:, b, i]):
            rep.bad(f"persistence b={b} i={i}: gpu {g['persistence'][b, i]} disagrees with its own layer argmaxes")
        same_k = g["persistence"][b, i] == o["persistence"][b, i]
        if not same_k:
            if lazy_excuse[b, i]:
                rep.excused["lazy_band"] += 1
            elif tie_any[b, i]:
                rep.excused["persistence_tie"] += 1
            else:
                rep.bad(f"persistence b={b} i={i}: gpu {g['persistence'][b, i]} oracle {o['persistence'][b, i]}")
        elif g["persistence"][b, i] >= 0 and (
                abs(g["drop"][b, i] - o["drop"][b, i]) > 2 * CONF_TOL or
                abs(g["stability"][b, i] - o["stability"][b, i]) > P.w * 2 * CONF_TOL + 1e-6):
            rep.bad(f"drop/stability b={b} i={i}: gpu {g['drop'][b, i]:.6g}/{g['stability'][b, i]:.6g} "
                    f"oracle {o['drop'][b, i]:.6g}/{o['stability'][b, i]:.6g}")
        gf, of = int(g["flags"][b, i]) & 7, int(o["flags"][b, i]) & 7
        if gf != int(gflags_expect[b, i]):
            rep.bad(f"route flags b={b} i={i}: gpu {gf} do not follow from its own c/S ({gflags_expect[b, i]})")
        if gf != of:
            c = o["confidence"][b, i]
            if tie_any[b, i] or (lazy_excuse[b, i] and not same_k):
                why = "cand_argmax_tie"
            elif abs(c - P.theta_h) <= CONF_TOL or abs(c - P.theta_c) <= CONF_TOL:
                why = "threshold_tie"
            elif abs(o["stability"][b, i] - P.theta_s) <= P.w * 2 * CONF_TOL:
                why = "stability_tie"
            else:
                why = None
            if why is None:
                rep.bad(f"route flags b={b} i={i}: gpu {gf} oracle {of} c={c:.6g} S={o['stability'][b, i]:.6g}")
            else:
                rep.excused[why] += 1
                if (gf ^ of) & F_CAND:
                    cand_excused[b, i] = True
    # commitment per sequence
    for b in range(B):
        idx = np.nonzero(m[b])[0]
        n = idx.size
        if n == 0:
            if g["n_commit"][b] != 0:
                rep.bad(f"n_commit b={b} with no masked position")
            continue
        rep.checked["commit"] += n
        gcm = g["commit"][b, idx] != 0
        ocm = o["commit"][b, idx] != 0
        gfb = (g["flags"][b, idx] & F_FALLBACK) > 0
        ofb = (o["flags"][b, idx] & F_FALLBACK) > 0
        if np.any(((g["flags"][b, idx] & F_COMMIT) > 0) != gcm):
            rep.bad(f"committed flag bit b={b} differs from the commit mask")
        if g["n_commit"][b] != gcm.sum():
            rep.bad(f"n_commit b={b}: gpu {g['n_commit'][b]} but {gcm.sum()} committed")
        # (a) the conditioned oracle: the commitment rule on the GPU's own inputs, in float64
        gcand = (g["flags"][b, idx] & F_CAND) > 0
        Hg = g["entropy"][b, idx].astype(np.float64)
        cg = g["confidence"][b, idx].astype(np.float64)
        cond = conditioned(idx, Hg, gcand, cg, P)
        ccm = np.asarray(cond["commit"], bool)
        cfb = np.zeros(n, bool)
        if cond["fallback"] >= 0:
            cfb[cond["fallback"]] = True
        rounding = n * U * np.abs(np.nan_to_num(cond["N"])) + 1e-7
        cond_tie = (np.abs(cond["N"] - P.beta) <= rounding) if block == 0 else np.zeros(n, bool)
        pre_g, pre_c = gcm & ~gfb, ccm & ~cfb
        for q in np.nonzero(pre_g != pre_c)[0]:
            if cond_tie[q]:
                rep.excused["gpu_scan_rounding"] += 1
            else:
                rep.bad(f"commit b={b} i={idx[q]}: gpu {pre_g[q]} but the rule on its own candidates and "
                        f"entropies gives {pre_c[q]} (N={cond['N'][q]:.6g}, beta={P.beta})")
        if np.array_equal(pre_g, pre_c):
            if not np.array_equal(gfb, cfb) or not np.array_equal(gcm, ccm):
                rep.bad(f"fallback b={b}: gpu {idx[gfb]} but the rule on its own confidences gives {idx[cfb]}")
            Ec = np.asarray(cond["E"], np.float64)
            Eg = g["upstream_entropy"][b, idx].astype(np.float64)
            fin = np.isfinite(Ec)
            bad = fin & (np.abs(Eg - Ec) > n * U * np.abs(np.nan_to_num(Ec)) + 1e-6)
            if bad.any():
                q = int(np.argmax(bad))
                rep.bad(f"upstream_entropy b={b} i={idx[q]}: gpu {Eg[q]:.7g}, the rule on its own entropies "
                        f"{Ec[q]:.7g}")
        # (b) parity with the oracle: budget decisions before the fallback, then the fallback
        ocand = (o["flags"][b, idx] & F_CAND) > 0
        dH = np.abs(np.nan_to_num(g["entropy"][b, idx] - o["entropy"][b, idx]))
        N = o["budget_prefix"][b, idx]
        slack = 1e-4 + n * U * np.abs(np.nan_to_num(N)) + np.concatenate([[0.0], np.cumsum(np.where(ocand, 0.0, dH))[:-1]])
        slack = slack + np.concatenate([[0.0], np.cumsum(np.where(cand_excused[b, idx],
                                                                  np.nan_to_num(o["entropy"][b, idx]), 0.0))[:-1]])
        # RPD-block has no budget: no commit decision sits near beta
        budget_tie = np.zeros(n, bool) if block > 0 else np.abs(N - P.beta) <= slack
        flipped_before = np.cumsum(cand_excused[b, idx]) > 0     # an excused candidacy flip at or before q
        pre_go, pre_o = gcm & ~gfb, ocm & ~ofb
        pre_excused = False
        for q in np.nonzero(pre_go != pre_o)[0]:
            if flipped_before[q]:
                rep.excused["commit_cascade"] += 1
            elif budget_tie[q]:
                rep.excused["budget_tie"] += 1
            else:
                rep.bad(f"commit b={b} i={idx[q]}: gpu {pre_go[q]} oracle {pre_o[q]} N={N[q]:.6g} beta={P.beta}")
                continue
            pre_excused = True
        if gfb.any() and ofb.any():
            fg, fo = int(np.nonzero(gfb)[0][0]), int(np.nonzero(ofb)[0][0])
            if fg != fo:
                co = np.nan_to_num(o["confidence"][b, idx], nan=-np.inf)
                if co[fg] >= co[fo] - 2 * CONF_TOL:
                    rep.excused["fallback_tie"] += 1
                else:
                    rep.bad(f"fallback b={b}: gpu {idx[fg]} (oracle c {co[fg]:.6g}) oracle {idx[fo]} "
                            f"(c {co[fo]:.6g})")
        elif gfb.any() != ofb.any():
            if pre_excused:
                rep.excused["fallback_follows"] += 1
            else:
                rep.bad(f"fallback b={b}: gpu {idx[gfb]} oracle {idx[ofb]} with the same budget decisions")
        if np.array_equal(gcm, ocm) and np.array_equal(gfb, ofb):
            dE = np.abs(g["upstream_entropy"][b, idx] - o["upstream_entropy"][b, idx])
            tolE = 1e-4 + np.concatenate([[0.0], np.cumsum(dH)[:-1]]) + \
                (n * U + 1e-6) * np.abs(np.nan_to_num(o["upstream_entropy"][b, idx]))
            fin = np.isfinite(o["upstream_entropy"][b, idx])
            if np.any((dE > tolE) & fin):
                q = int(np.argmax((dE > tolE) & fin))
                rep.bad(f"upstream_entropy b={b} i={idx[q]}: gpu {g['upstream_entropy'][b, idx[q]]:.6g} "
                        f"oracle {o['upstream_entropy'][b, idx[q]]:.6g}")
    return rep


def as_gpu_outputs(o: dict) -> dict:
    """The oracle's outputs in the types the GPU returns them (float32, int32,
    uint8): what a GPU that reproduced the oracle exactly would report. Used
    to show on the CPU that the comparator accepts a correct result and
    rejects planted mistakes."""
    g = {}
    for k in ("commit", "flags"):
        g[k] = np.asarray(o[k]).astype(np.uint8)
    for k in ("token", "persistence", "n_commit"):
        g[k] = np.asarray(o[k]).astype(np.int32)
    for k in ("entropy", "confidence", "drop", "stability", "upstream_entropy"):
        g[k] = np.asarray(o[k]).astype(np.float32)
    g["layer_argmax"] = np.asarray(o["layer_argmax"]).astype(np.int32)
    g["layer_conf"] = np.asarray(o["layer_conf"]).astype(np.float32)
    g["layer_entropy"] = np.asarray(o["layer_entropy"]).astype(np.float32)
    return g
