"""fp64 reference of the Reliable Parallel Decoding (RPD) commit step.

TEST INFRASTRUCTURE ONLY. This module is the plain, slow, obviously correct
CPU statement of what the commit step computes. Only the test suite, the
package smoke check and the CPU-baseline leg of the benchmark may import it;
the product path never does, and it shares no code with the HIP library.

Every function follows a passage of the paper (He, Liu, Xiong, Zhang,
"Reliable Parallel Decoding in Masked Diffusion Language Models"):

* projection of hidden states through the unembedding ("logit lens") --
  Section 2.2 and Appendix A.2 "Intermediate-layer readout", Appendix A.6
  "Layerwise projection";
* the model's final normalization applied to intermediate states before the
  output head, with the final layer's native (already normalized) state
  used as is -- Appendix A.2 "Intermediate-layer readout", Appendix A.6
  "Layerwise projection";
* entropy ``H(p) = -sum_v p(v) log p(v)`` in nats -- Eq. (1), Section 2.1;
* prediction persistence ``K_i`` -- Eq. (2), Section 2.2 and Appendix A.2;
* confidence drop ``r_i`` -- Eq. (3), Section 2.2 and Appendix A.2;
* stability score ``S_i = min(K_i, K_max) - w r_i`` -- Eq. (4), Section 3.1;
* candidate set -- Eq. (5), Section 3.1;
* sequential cumulative-entropy commitment and the progress fallback --
  Section 3.2 (definitions of ``E_i`` and ``A_t``), hyperparameters in
  Table 4 (Appendix A.6);
* the RPD-block commitment -- Section 3.2 "Variants" and Appendix A.6
  "RPD-block": the candidates of the active 32-position block, no budget,
  fallback to the block's most confident masked position;
* lazy layerwise projection -- Appendix A.6 "Layerwise projection": a
  position's intermediate layers are projected from the final one down and
  no further than its agreement suffix needs (the first disagreeing layer);
* the end of an iteration (fill A_t with its predictions, keep the rest
  masked) and a loop of iterations until the canvas is filled -- Section 3.2.

Readings where the paper is silent (stated once here, used throughout):
the supplied hidden states are already normalised (the projection is a plain
product with W_U); the scoring softmax uses temperature 1; argmax ties go to
the lowest vocabulary index; the layer window is the K layers supplied, with
layer K-1 the final one; ``p^(l)(y_i)`` in the drop is the probability of the
final-layer token; sequences of a batch are independent; "the first W masked
positions" are the first W entries of the masked list in canvas order; the
fallback ignores NaN confidences and picks the lowest index among equals.
For RPD-block: blocks are consecutive runs of ``block`` canvas positions
starting at position 0 of each sequence; the active block is the first one
that still holds a masked position; ``E_i`` is still reported, as the
entropy over earlier masked positions outside the commitment set.

Arithmetic is float64 on the exact values of the bf16 / fp32 inputs.
The final normalization is RMS normalization with a gain vector g,
``g * x / sqrt(mean(x^2) + eps)``, evaluated in float64 and rounded (round
to nearest, ties to even) to the input type, since the model's
normalization hands the output head a state of that type. An optional
logit scale (an inverse temperature, 1 by default, the paper's reading)
multiplies every logit before the softmax statistics.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

# flag bits of the per-position record (same meaning on every side)
FLAG_CANDIDATE = 1
FLAG_HIGH_CONF = 2
FLAG_STABLE = 4
FLAG_COMMITTED = 8
FLAG_FALLBACK = 16


@dataclass(frozen=True)
class Params:
    """Hyperparameters of the commit rule (Table 4, Appendix A.6)."""
    theta_h: float = 0.9     # high-confidence threshold, bypasses stability
    theta_c: float = 0.6     # minimum confidence for stability admission
    theta_s: float = 3.5     # stability threshold
    w: float = 15.0          # weight of the confidence-drop penalty
    k_max: int = 6           # cap on persistence
    beta: float = 4.0        # cumulative entropy budget, nats
    window: int = 32         # fallback window W
    block: int = 0           # 0: full RPD; > 0: RPD-block with blocks of this many positions
    logit_scale: float = 1.0  # multiplies every logit before the softmax statistics (1 / temperature)
    lazy: bool = False        # lazy layerwise projection (score_commit_lazy); the rule itself is unchanged
    lazy_all: bool = False    # lazy: every masked position walks its layers (else only the band theta_c <= c < theta_h)
    monotone: bool = False    # report-only reading of the agreement rule: see monotone_agreement (oracle only)


LLADA = Params(theta_s=3.5, w=15.0)
DREAM = Params(theta_s=2.5, w=20.0)


def strict(K: int, beta: float = 1.0) -> Params:
    """The rule "argmax agrees across all K layers and its probability does
    not drop at the final layer" expressed in Eq. (4): with w = 1, K_max >= K
    and theta_s = K, S_i >= theta_s holds exactly when K_i = K and r_i = 0."""
    return Params(theta_h=0.9, theta_c=0.6, theta_s=float(K), w=1.0,
                  k_max=max(K, 6), beta=beta, window=32)


# ------------------------------------------------------------- inputs ----

def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of bf16 bit patterns (uint16) or fp32 values."""
    if dtype == "bf16":
        return (np.asarray(a).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def round_to_bf16(v: np.ndarray) -> np.ndarray:
    """float64 -> the nearest bfloat16 value (8 significant bits, ties to
    even), returned as float64. Normal range: v = m 2^e with 0.5 <= |m| < 1,
    kept to m rounded at 2^-8; below 2^-126 the grid is 2^-133."""
    v = np.asarray(v, np.float64)
    m, e = np.frexp(v)
    normal = np.round(m * 256.0) * np.exp2(e.astype(np.float64) - 8.0)   # np.round: ties to even
    sub = np.round(v * 2.0 ** 133) * 2.0 ** -133
    return np.where(np.abs(v) < 2.0 ** -126, sub, normal)


def final_norm(x: np.ndarray, g: np.ndarray, eps: float, dtype: str) -> np.ndarray:
    """The model's final normalization applied to a state before the output
    head (Appendix A.2 "Intermediate-layer readout"): RMS normalization
    ``g * x / sqrt(mean(x^2) + eps)`` in float64, rounded to the input type.
    ``x`` and ``g`` are exact float64 values of the inputs."""
    x = np.asarray(x, np.float64)
    n = np.asarray(g, np.float64) * x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return round_to_bf16(n) if dtype == "bf16" else n.astype(np.float32).astype(np.float64)


# ------------------------------------------------- distribution statistics --

def distribution_stats(z: np.ndarray) -> dict:
    """Softmax statistics of logit rows ``z[..., V]`` (temperature 1).

    argmax: lowest index of the maximum logit; conf: largest probability;
    entropy: Eq. (1), ``-sum p log p`` with ``0 log 0 = 0``, in nats."""
    z = np.asarray(z, dtype=np.float64)
    m = z.max(axis=-1, keepdims=True)
    y = z.argmax(axis=-1)                      # first maximum = lowest index
    e = np.exp(z - m)
    p = e / e.sum(axis=-1, keepdims=True)
    with np.errstate(divide="ignore", invalid="ignore"):
        plogp = np.where(p > 0.0, p * np.log(np.where(p > 0.0, p, 1.0)), 0.0)
    plogp = np.where(np.isnan(p), np.nan, plogp)
    return {
        "argmax": y.astype(np.int64),
        "conf": p.max(axis=-1),
        "entropy": -plogp.sum(axis=-1),
        "p": p,
    }


def _top2_gap(z: np.ndarray, y: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Gap between the top logit and the best other logit, and that runner-up."""
    zz = z.copy()
    np.put_along_axis(zz, y[..., None], -np.inf, axis=-1)
    second = zz.argmax(axis=-1)
    gap = np.take_along_axis(z, y[..., None], -1)[..., 0] - np.take_along_axis(z, second[..., None], -1)[..., 0]
    return gap, second


def project_layer_stats(hidden: np.ndarray, w_u: np.ndarray, dtype: str,
                        positions: list[tuple[int, int]], w_rows_per_chunk: int = 8192,
                        max_bytes: int = 1 << 30, norm: tuple | None = None,
                        logit_scale: float = 1.0) -> dict:
    """Per-layer statistics at the given canvas positions.

    For each position (b, i) and each supplied layer l the logits are
    ``z = logit_scale * W_U x`` with ``x = hidden[l][b][i]`` (Section 2.2:
    intermediate states read out through the output head; Appendix A.6: only
    masked positions are projected). With ``norm = (g, eps, norm_final)`` the
    states of layers 0 .. K-2 (and of layer K-1 too if ``norm_final``) first
    go through final_norm, ``g`` given like the hidden states (bf16 bit
    patterns or fp32). Returns arrays shaped [npos][K]:
    ``argmax, conf, entropy`` of each layer's distribution, ``p_final`` =
    probability at layer l of the final layer's argmax token, and two
    diagnostics for classifying near-ties: ``gap`` (top-1 minus top-2 logit)
    and ``absbound`` (max over the top two tokens v of sum_k |W_U[v,k] x_k|)."""
    K = hidden.shape[0]
    V, d = w_u.shape
    npos = len(positions)
    out = {k: np.zeros((npos, K), np.float64) for k in ("conf", "entropy", "p_final", "gap", "absbound")}
    out["argmax"] = np.zeros((npos, K), np.int64)
    if npos == 0:
        return out
    per_block = max(1, int(max_bytes // (K * V * 8)))
    for p0 in range(0, npos, per_block):
        blk = positions[p0:p0 + per_block]
        nb = len(blk)
        x = np.stack([to_f64(hidden[l, b, i], dtype) for (b, i) in blk for l in range(K)])  # [nb*K][d]
        if norm is not None:
            g, eps, norm_final = norm
            gf = to_f64(g, dtype)
            for a in range(nb):
                for l in range(K if norm_final else K - 1):
                    x[a * K + l] = final_norm(x[a * K + l], gf, eps, dtype)
        z = np.empty((nb * K, V), np.float64)
        for v0 in range(0, V, w_rows_per_chunk):
            wc = to_f64(w_u[v0:v0 + w_rows_per_chunk], dtype)
            z[:, v0:v0 + wc.shape[0]] = logit_scale * (x @ wc.T)
        z = z.reshape(nb, K, V)
        st = distribution_stats(z)
        y_final = st["argmax"][:, K - 1]
        gap, second = _top2_gap(z, st["argmax"])
        absb = np.zeros((nb, K))
        for a in range(nb):
            for l in range(K):
                xr = np.abs(x[a * K + l])
                rows = to_f64(w_u[[st["argmax"][a, l], second[a, l]]], dtype)
                absb[a, l] = abs(logit_scale) * (np.abs(rows) @ xr).max()
        sl = slice(p0, p0 + nb)
        out["argmax"][sl] = st["argmax"]
        out["conf"][sl] = st["conf"]
        out["entropy"][sl] = st["entropy"]
        out["p_final"][sl] = np.take_along_axis(st["p"], y_final[:, None, None].repeat(K, 1), -1)[..., 0]
        out["gap"][sl] = gap
        out["absbound"][sl] = absb
    return out


# ------------------------------------------------------ layerwise stability --

def persistence(layer_argmax: np.ndarray) -> int:
    """Eq. (2): number of consecutive layers, ending at the final one, whose
    argmax equals the final prediction; the count stops at the first
    disagreement (earlier agreeing layers are not counted)."""
    K = len(layer_argmax)
    y = layer_argmax[K - 1]
    k = 1
    while k < K and layer_argmax[K - 1 - k] == y:
        k += 1
    return k


def confidence_drop(p_final: np.ndarray, k_i: int) -> float:
    """Eq. (3): peak over the agreement suffix of the final token's
    probability, minus its final-layer probability."""
    K = len(p_final)
    return float(max(p_final[K - k_i:]) - p_final[K - 1])


def stability_score(k_i: int, r_i: float, p: Params) -> float:
    """Eq. (4)."""
    return float(min(k_i, p.k_max)) - p.w * r_i


def monotone_agreement(layer_argmax: np.ndarray, p_final: np.ndarray) -> bool:
    """The literal reading of the rule "argmax agreement across all K layers
    with non-decreasing top probability": every layer predicts the final
    token (K_i = K, Eq. 2) and that token's probability never falls from one
    layer to the next. The reading the commit step implements instead is
    Eq. 4 with w = 1, K_max >= K, theta_s = K (strict()): K_i = K and r_i <= 0
    (Eq. 3), i.e. only the final layer has to hold the peak. This one is
    evaluated by the oracle only, to report where the two readings part."""
    K = len(layer_argmax)
    if any(layer_argmax[l] != layer_argmax[K - 1] for l in range(K)):
        return False
    return all(p_final[l] <= p_final[l + 1] for l in range(K - 1))


def candidate_routes(c: float, s: float, p: Params) -> tuple[bool, bool]:
    """Eq. (5): (high-confidence route, stability route). NaN fails both."""
    high = bool(c >= p.theta_h)
    stab = bool(p.theta_c <= c < p.theta_h and s >= p.theta_s)
    return high, stab


# ------------------------------------------------------------ commitment --

def commit_scan(H: np.ndarray, cand: np.ndarray, c: np.ndarray, p: Params) -> dict:
    """Section 3.2 for one sequence, on its masked positions in canvas order.

    Literal left-to-right construction: when the scan reaches position i,
    ``E_i`` is the entropy summed over earlier masked positions not yet
    selected (non-candidates and rejected candidates alike); a candidate is
    selected when ``E_i <= beta``. If nothing is selected, the single most
    confident of the first W masked positions is committed (progress
    fallback). Returns ``commit`` (bool), ``E`` (E_i at every masked
    position, before the fallback) and ``fallback`` (index or -1)."""
    n = len(H)
    commit = np.zeros(n, bool)
    E = np.zeros(n, np.float64)
    acc = 0.0  # sum of H over earlier masked positions left out of A
    for i in range(n):
        E[i] = acc
        if cand[i] and acc <= p.beta:
            commit[i] = True
        else:
            acc = acc + H[i]
    fb = -1
    if n > 0 and not commit.any():
        win = c[:min(p.window, n)]
        best = -np.inf
        fb = 0
        for j, cj in enumerate(win):
            if not np.isnan(cj) and cj > best:
                best, fb = cj, j
        commit[fb] = True
    return {"commit": commit, "E": E, "fallback": fb}


def commit_block(idx: np.ndarray, H: np.ndarray, cand: np.ndarray, c: np.ndarray, block: int) -> dict:
    """RPD-block for one sequence (Section 3.2 "Variants"; Appendix A.6
    "RPD-block"), on its masked positions in canvas order at canvas indices
    ``idx``. The active block is the first run of ``block`` canvas positions
    (runs start at 0) that holds a masked position; every candidate inside it
    is committed and no entropy budget applies. If none is, the single most
    confident masked position of the active block is committed. ``E`` reports
    the entropy over earlier masked positions outside the commitment set
    (before the fallback), as in commit_scan."""
    n = len(H)
    commit = np.zeros(n, bool)
    E = np.zeros(n, np.float64)
    fb = -1
    if n == 0:
        return {"commit": commit, "E": E, "fallback": fb}
    lo = (int(idx[0]) // block) * block
    active = (idx >= lo) & (idx < lo + block)
    for q in range(n):
        commit[q] = bool(cand[q] and active[q])
    acc = 0.0
    for q in range(n):
        E[q] = acc
        if not commit[q]:
            acc = acc + H[q]
    if not commit.any():
        best = -np.inf
        for q in range(n):
            if active[q] and not np.isnan(c[q]) and (fb < 0 or c[q] > best):
                best, fb = c[q], q
        if fb < 0:   # every confidence in the block is NaN: the first masked position
            fb = 0
        commit[fb] = True
    return {"commit": commit, "E": E, "fallback": fb}


def commit_closed_form(H: np.ndarray, cand: np.ndarray, p: Params) -> dict:
    """Equivalent closed form of the budget test: with
    ``N_i = sum of H_j over earlier masked non-candidates``, the selected set
    is exactly ``{i : cand_i and N_i <= beta}`` (every earlier candidate of an
    accepted one is accepted, so ``E_i = N_i`` there; a rejected one has
    ``E_i >= N_i > beta``). Returned without the fallback."""
    n = len(H)
    N = np.zeros(n, np.float64)
    acc = 0.0
    for i in range(n):
        N[i] = acc
        if not cand[i]:
            acc = acc + H[i]
    return {"commit": np.asarray(cand, bool) & (N <= p.beta), "N": N}


# ------------------------------------------------------------- assembly --

def select(mask: np.ndarray, layer: dict, p: Params, positions: list[tuple[int, int]]) -> dict:
    """Scoring (Eq. 2-5) and commitment (Section 3.2) from per-layer
    statistics ``layer[name][npos][K]`` listed in ``positions`` order, which
    must hold every masked position of every sequence in canvas order."""
    B, L = mask.shape
    K = layer["argmax"].shape[1]
    o = {
        "commit": np.zeros((B, L), np.uint8),
        "token": np.full((B, L), -1, np.int32),
        "entropy": np.zeros((B, L)),
        "confidence": np.zeros((B, L)),
        "persistence": np.zeros((B, L), np.int32),
        "drop": np.zeros((B, L)),
        "stability": np.zeros((B, L)),
        "flags": np.zeros((B, L), np.uint8),
        "upstream_entropy": np.zeros((B, L)),
        "budget_prefix": np.zeros((B, L)),
        "n_commit": np.zeros(B, np.int32),
    }
    index = {bi: a for a, bi in enumerate(positions)}
    for b in range(B):
        masked = np.nonzero(mask[b])[0]
        n = len(masked)
        H = np.zeros(n)
        c = np.zeros(n)
        cand = np.zeros(n, bool)
        for q, i in enumerate(masked):
            a = index[(b, int(i))]
            am = layer["argmax"][a]
            pf = layer["p_final"][a]
            k_i = persistence(am)
            r_i = confidence_drop(pf, k_i)
            s_i = stability_score(k_i, r_i, p)
            c_i = layer["conf"][a, K - 1]
            h_i = layer["entropy"][a, K - 1]
            high, stab = candidate_routes(c_i, s_i, p)
            if p.monotone:   # the literal reading (report only): agreement with a non-decreasing probability
                stab = bool(p.theta_c <= c_i < p.theta_h and monotone_agreement(am, pf))
            H[q], c[q], cand[q] = h_i, c_i, high or stab
            o["token"][b, i] = am[K - 1]
            o["entropy"][b, i] = h_i
            o["confidence"][b, i] = c_i
            o["persistence"][b, i] = k_i
            o["drop"][b, i] = r_i
            o["stability"][b, i] = s_i
            o["flags"][b, i] = (FLAG_CANDIDATE * (high or stab)) | (FLAG_HIGH_CONF * high) | (FLAG_STABLE * stab)
        if p.block > 0:
            sc = commit_block(masked, H, cand, c, p.block)
            cf = {"N": np.zeros(n)}
        else:
            sc = commit_scan(H, cand, c, p)
            cf = commit_closed_form(H, cand, p)
        if p.block == 0 and not np.isnan(H).any():
            pre = sc["commit"].copy()
            if sc["fallback"] >= 0:
                pre[sc["fallback"]] = False
            assert np.array_equal(pre, cf["commit"]), "sequential scan and closed form disagree"
        for q, i in enumerate(masked):
            o["upstream_entropy"][b, i] = sc["E"][q]
            o["budget_prefix"][b, i] = cf["N"][q]
            if sc["commit"][q]:
                o["commit"][b, i] = 1
                o["flags"][b, i] |= FLAG_COMMITTED
        if sc["fallback"] >= 0:
            o["flags"][b, masked[sc["fallback"]]] |= FLAG_FALLBACK
        o["n_commit"][b] = int(sc["commit"].sum())
    return o


def lazy_layer_stats(hidden: np.ndarray, w_u: np.ndarray, mask: np.ndarray, dtype: str, p: Params,
                     norm: tuple | None = None):
    """Lazy layerwise projection (Appendix A.6 "Layerwise projection"): the
    final layer of every masked position is projected first; then a position
    projects its intermediate layers from K-2 downwards, stopping after the
    first layer whose argmax differs from the final token, which is where
    its agreement suffix is known. Its persistence and drop are then exactly
    those of the eager projection. With ``p.lazy_all`` every masked position
    with a finite final confidence walks (the procedure as the paper states
    it); otherwise only the positions whose candidacy the stability test
    can decide (theta_c <= c < theta_h, Eq. 5) do, a further saving of this
    implementation that leaves every decision unchanged. Unprojected layers
    hold argmax -1 and NaN statistics.
    Returns (positions, per-layer statistics, layers projected per position)."""
    pos = masked_positions(mask)
    K = hidden.shape[0]
    n = len(pos)
    layer = {k: np.full((n, K), np.nan) for k in ("conf", "entropy", "p_final", "gap", "absbound")}
    layer["argmax"] = np.full((n, K), -1, np.int64)
    projected = np.zeros(n, np.int64)

    def one(a: int, l: int) -> dict:
        # layer l of position a alone; normalized like the eager path (layer K-1 native unless norm_final)
        b, i = pos[a]
        hl = hidden[l:l + 1]
        nrm = None
        if norm is not None and (l < K - 1 or norm[2]):
            nrm = (norm[0], norm[1], True)
        st = project_layer_stats(hl, w_u, dtype, [(b, i)], norm=nrm, logit_scale=p.logit_scale)
        projected[a] += 1
        return {k: st[k][0, 0] for k in ("argmax", "conf", "entropy", "gap", "absbound")}

    for a in range(n):
        f = one(a, K - 1)
        for k in ("argmax", "conf", "entropy", "gap", "absbound"):
            layer[k][a, K - 1] = f[k]
        layer["p_final"][a, K - 1] = f["conf"]
        c = f["conf"]
        if not (_walks(c, p)):
            continue
        for l in range(K - 2, -1, -1):
            st = one(a, l)
            for k in ("argmax", "conf", "entropy", "gap", "absbound"):
                layer[k][a, l] = st[k]
            if st["argmax"] != f["argmax"]:
                break
            layer["p_final"][a, l] = st["conf"]   # the layer's argmax is the final token
    return pos, layer, projected


def _walks(c: float, p: Params) -> bool:
    """Whether a position with final confidence c walks its intermediate
    layers in the lazy projection."""
    if p.lazy_all:
        return not np.isnan(c)
    return bool(p.theta_c <= c < p.theta_h)


def score_commit_lazy(hidden: np.ndarray, w_u: np.ndarray, mask: np.ndarray, dtype: str, p: Params,
                      norm: tuple | None = None) -> dict:
    """The commit step with lazy layerwise projection: the same candidacy and
    commitment as score_commit (stability matters only inside the band
    theta_c <= c < theta_h, and every walking position reaches its first
    disagreement). Where a position does not walk (outside the band unless
    ``p.lazy_all``; a NaN confidence) stability is not evaluated: persistence
    -1, drop and stability NaN. ``layers_projected`` counts the projections
    per position."""
    pos, layer, projected = lazy_layer_stats(hidden, w_u, mask, dtype, p, norm)
    o = assemble(mask, pos, layer, p)
    for a, (b, i) in enumerate(pos):
        c = layer["conf"][a, -1]
        if not _walks(c, p):
            o["persistence"][b, i] = -1
            o["drop"][b, i] = np.nan
            o["stability"][b, i] = np.nan
    o["layers_projected"] = projected
    return o


def apply_commit(mask: np.ndarray, canvas: np.ndarray, commit: np.ndarray, token: np.ndarray) -> None:
    """End of an iteration (Section 3.2): every position of A_t is filled with
    its prediction y_i and leaves the mask; the rest stay masked. A_t is a
    subset of the masked positions, so a flag at a position that is no longer
    masked changes nothing (a filled token is never overwritten). In place."""
    sel = (mask != 0) & (commit != 0)
    canvas[sel] = token[sel]
    mask[sel] = 0


def decode_loop(hidden: np.ndarray, w_u: np.ndarray, mask: np.ndarray, dtype: str, p: Params,
                max_iter: int | None = None, norm: tuple | None = None) -> dict:
    """Iterations of the commit step until no position is masked, on fixed
    hidden states (a synthetic stand-in for the forward passes between
    iterations): returns the canvas (-1 where never filled), the number of
    iterations and each iteration's commit mask. The progress fallback
    commits at least one position per iteration, so at most n iterations run."""
    mask = mask.copy()
    canvas = np.full(mask.shape, -1, np.int64)
    commits = []
    n0 = int(mask.sum())
    limit = n0 if max_iter is None else max_iter
    while mask.any() and len(commits) < limit:
        o = (score_commit_lazy if p.lazy else score_commit)(hidden, w_u, mask, dtype, p, norm=norm)
        commits.append(o["commit"].copy())
        apply_commit(mask, canvas, o["commit"], o["token"])
    return {"canvas": canvas, "iterations": len(commits), "commits": commits, "mask": mask}


def masked_positions(mask: np.ndarray) -> list[tuple[int, int]]:
    B, L = mask.shape
    return [(b, int(i)) for b in range(B) for i in np.nonzero(mask[b])[0]]


def layer_stats_masked(hidden: np.ndarray, w_u: np.ndarray, mask: np.ndarray, dtype: str,
                       norm: tuple | None = None, logit_scale: float = 1.0):
    """Per-layer statistics of every masked position (canvas order)."""
    pos = masked_positions(mask)
    return pos, project_layer_stats(hidden, w_u, dtype, pos, norm=norm, logit_scale=logit_scale)


def assemble(mask: np.ndarray, pos: list, layer: dict, p: Params) -> dict:
    """Scoring and commitment plus the per-layer arrays in [K][B][L] layout."""
    o = select(mask, layer, p, pos)
    K = layer["argmax"].shape[1]
    B, L = mask.shape
    for name in ("argmax", "conf", "entropy", "p_final", "gap", "absbound"):
        arr = np.full((K, B, L), -1 if name == "argmax" else 0.0,
                      np.int64 if name == "argmax" else np.float64)
        for a, (b, i) in enumerate(pos):
            arr[:, b, i] = layer[name][a]
        o["layer_" + name] = arr
    return o


def score_commit(hidden: np.ndarray, w_u: np.ndarray, mask: np.ndarray, dtype: str, p: Params,
                 norm: tuple | None = None) -> dict:
    """The whole commit step for one decoding iteration: project every masked
    position at every supplied layer, score, select candidates and commit.
    ``hidden[K][B][L][d]``, ``w_u[V][d]``, ``mask[B][L]`` (1 = masked);
    ``norm = (g, eps, norm_final)`` normalizes the states first
    (project_layer_stats)."""
    pos, layer = layer_stats_masked(hidden, w_u, mask, dtype, norm=norm, logit_scale=p.logit_scale)
    return assemble(mask, pos, layer, p)
