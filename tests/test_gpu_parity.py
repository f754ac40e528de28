"""Parity of the HIP commit step with the fp64 oracle, through the C ABI.

Small and mid-size cases are compared element by element (every masked
position, every layer); they span several vocabulary and row tiles, ragged
vocabulary sizes and hidden sizes that are not multiples of the 64-wide
k-chunk, and every projection variant (the streaming family at <= 32 and
64 projected rows, and the 128-, 192- and 256-row MFMA tiles above, with row
tiles split across XCDs, and rows gathered through 32-bit buffer offsets or,
from a hidden tensor of more than 2^31 bytes, 64-bit addresses). The
full-size LLaDA-8B / Dream-7B shapes are compared at every masked position
and layer too (whole sequences of the batched shapes), and additionally on
sampled positions of the whole batches. Edge cases: vocabularies smaller
than one tile (down to V = 1), exact argmax ties from duplicated unembedding
rows, zero hidden rows (uniform distribution), empty
sequences inside a batch, NaN rows, budget and window extremes."""
import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_36452_amd import binding as rpd
from paper_2609_36452_amd.workload import CONFIGS, draw_unembedding, make_workload, round_bf16_bits
from tests.gpu_util import gpu_params, note, run_gpu, run_oracle, to_device
from tests.parity import compare, gap_tol, ENTROPY_TOL, CONF_TOL

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _check(w, P, layer=True, norm=None, **kw):
    g = run_gpu(w, P, layer_stats=layer, norm=norm, **kw)
    o = run_oracle(w, P, norm=norm)
    rep = compare(g, o, w.mask, P, w.cfg.d, layer=layer)
    note("  " + rep.summary()[:300])
    assert rep.ok(), rep.summary()
    masked = int(w.mask.sum())
    assert sum(rep.excused.values()) <= max(2, 0.05 * masked * (w.cfg.K + 3)), rep.summary()
    return g, o, rep


# -------------------------------------------------------------- tiny fp32 --

@pytest.mark.parametrize("seed", range(12))
def test_tiny_f32_strict(seed):
    w = make_workload("tiny", seed)
    _check(w, O.strict(3, 1.0))


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("pname", ["llada", "dream"])
def test_tiny_f32_calibrated(seed, pname):
    cfg = CONFIGS["tiny"].with_(sharp=("calibrated",), unstable_frac=0.3)
    w = make_workload(cfg, 100 + seed)
    _check(w, O.LLADA if pname == "llada" else O.DREAM)


# ------------------------------------------------- bf16, several variants --

BF16_CASES = [
    # name (the projection variant the case runs, then what it exercises), overrides, seed;
    # rows = K * masked. Hidden sizes: whole 64-wide chunks, odd chunk counts, ragged tails.
    ("bf16_s32", dict(B=1, L=64, K=4, d=264, V=5003, n_masked=8, masked_frac=None), 11),
    ("bf16_s64", dict(B=2, L=40, K=3, d=512, V=4099, n_masked=10, masked_frac=None), 12),
    ("bf16_big128_long_d", dict(B=1, L=40, K=4, d=4104, V=2500, n_masked=20, masked_frac=None), 15),
    ("bf16_big192_two_seqs", dict(B=2, L=40, K=4, d=520, V=7001, n_masked=20, masked_frac=None), 16),
    ("bf16_big_one_row_tile_odd_chunks", dict(B=1, L=80, K=3, d=200, V=6007, n_masked=80, masked_frac=None), 17),
    ("bf16_big_vocab_split", dict(B=3, L=100, K=4, d=520, V=7001, n_masked=None, masked_frac=0.5), 13),
    ("bf16_big192_row_split", dict(B=4, L=600, K=4, d=136, V=3001, n_masked=None, masked_frac=1.0), 14),
    ("bf16_big_row_split", dict(B=4, L=512, K=4, d=136, V=3001, n_masked=None, masked_frac=1.0), 22),
    ("bf16_big192_three_row_tiles", dict(B=2, L=100, K=4, d=264, V=3001, n_masked=72, masked_frac=None), 23),
    ("bf16_big128_short_d", dict(B=1, L=60, K=3, d=56, V=3001, n_masked=40, masked_frac=None), 26),
    ("bf16_big128_one_chunk", dict(B=1, L=60, K=4, d=64, V=2011, n_masked=30, masked_frac=None), 27),
    ("bf16_big128_ragged_vocab_two_seqs", dict(B=2, L=50, K=4, d=328, V=6999, n_masked=12, masked_frac=None), 28),
    ("bf16_big192_short_d", dict(B=1, L=60, K=3, d=56, V=3001, n_masked=48, masked_frac=None), 24),
    ("bf16_big192_one_chunk", dict(B=1, L=60, K=3, d=64, V=2011, n_masked=48, masked_frac=None), 25),
    # the 256 x 256 tile with no full 64-wide chunk (only the zero-filled tail) and with exactly one
    ("bf16_big_short_d", dict(B=1, L=80, K=3, d=56, V=3001, n_masked=80, masked_frac=None), 18),
    ("bf16_big_one_chunk", dict(B=1, L=80, K=3, d=64, V=2011, n_masked=80, masked_frac=None), 19),
    # 80 row tiles: 10 per XCD, swept in a group of 8 and a group of 2
    ("bf16_big_row_groups", dict(B=64, L=80, K=4, d=64, V=700, n_masked=None, masked_frac=1.0), 21),
]


@pytest.mark.parametrize("name,ov,seed", BF16_CASES, ids=[c[0] for c in BF16_CASES])
@pytest.mark.parametrize("sharp", ["scaled", "calibrated"])
def test_bf16_variants(name, ov, seed, sharp):
    base = CONFIGS["llada_late"].with_(name=name, **ov)
    if sharp == "calibrated":
        base = base.with_(sharp=("calibrated",), unstable_frac=0.3)
    w = make_workload(base, seed)
    variant = rpd.projection_variant(base.K, base.B, base.L, base.d, base.V, rpd.DTYPE_BF16, max_masked=w.n_masked)
    assert name.startswith(variant), (name, variant)
    for P in (O.strict(base.K, 1.0), O.LLADA, O.DREAM):
        _check(w, P)


# ------------------------------------------------------------ RPD-block --

@pytest.mark.parametrize("block", [32, 1, 7, 48])
def test_rpd_block_commitment(block):
    # Section 3.2 "Variants" / Appendix A.6 "RPD-block": candidates of the active block, no budget
    w = make_workload(CONFIGS["llada_late"].with_(name="blk", B=3, L=48, K=4, d=256, V=3001, n_masked=None,
                                                  masked_frac=0.6, sharp=("calibrated",), unstable_frac=0.3), 41)
    for P in (O.Params(theta_s=3.5, w=15.0, block=block), O.Params(theta_s=2.5, w=20.0, block=block, beta=0.0)):
        g, o, _ = _check(w, P)
        for b in range(w.cfg.B):
            m = np.nonzero(w.mask[b])[0]
            lo = m[0] // block * block
            com = np.nonzero(g["commit"][b])[0]
            assert len(com) >= 1 and ((com >= lo) & (com < lo + block)).all()


def test_rpd_block_at_late_decode_shape():
    # the headline shape with the paper's block size
    w = make_workload("llada_late", 3)
    _check(w, O.Params(theta_s=3.5, w=15.0, block=32))


# ------------------------------------------- final normalization, scale --

def _gain(w, seed):
    # the normalization gain, g ~ U(0.5, 2), in the workload's input encoding
    g = np.random.default_rng(seed).uniform(0.5, 2.0, w.cfg.d)
    return round_bf16_bits(g) if w.cfg.dtype == "bf16" else g.astype(np.float32)


NORM_CASES = [c for c in BF16_CASES if c[0] in ("bf16_s32", "bf16_big128_long_d", "bf16_big_one_row_tile_odd_chunks",
                                               "bf16_big_vocab_split")]


@pytest.mark.parametrize("name,ov,seed", NORM_CASES, ids=[c[0] for c in NORM_CASES])
@pytest.mark.parametrize("norm_final", [False, True])
def test_final_normalization_prologue(name, ov, seed, norm_final):
    # Appendix A.2 "Intermediate-layer readout": layers 0..K-2 through the final normalization,
    # the final layer native unless norm_final
    base = CONFIGS["llada_late"].with_(name=name, **ov).with_(sharp=("calibrated",), unstable_frac=0.3)
    w = make_workload(base, seed)
    norm = (_gain(w, seed + 100), 1e-5, norm_final)
    for P in (O.LLADA, O.strict(base.K, 1.0)):
        _check(w, P, norm=norm)


@pytest.mark.parametrize("scale", [0.5, 2.0])
@pytest.mark.parametrize("name", ["bf16_s32", "bf16_big128_long_d", "bf16_big_vocab_split"])
def test_logit_scale(name, scale):
    ov, seed = {c[0]: (c[1], c[2]) for c in BF16_CASES}[name]
    w = make_workload(CONFIGS["llada_late"].with_(name=name, **ov), seed)
    _check(w, dataclasses.replace(O.DREAM, logit_scale=scale))


def test_fp32_normalization_and_scale():
    w = make_workload("tiny", 7)
    norm = (_gain(w, 9), 1e-6, False)
    _check(w, dataclasses.replace(O.strict(3, 1.0), logit_scale=1.5), norm=norm)
    _check(w, O.LLADA, norm=(norm[0], 0.0, True))


# ------------------------------------------------------- lazy projection --

LAZY_CASES = [("bf16_s32", dict(B=1, L=64, K=4, d=264, V=5003, n_masked=8, masked_frac=None), 11),
              ("bf16_big128", dict(B=2, L=40, K=4, d=520, V=7001, n_masked=16, masked_frac=None), 16),
              ("bf16_big", dict(B=1, L=120, K=4, d=200, V=6007, n_masked=100, masked_frac=None), 17),
              # 200 positions: the final-layer pass lists 200 rows, which the 256 x 256 tile takes
              ("bf16_big_row_list", dict(B=1, L=240, K=4, d=136, V=3001, n_masked=200, masked_frac=None), 20),
              # most positions in the band: the passes after the first list 65-256 rows, launched once per
              # size class (<= 64, <= 128, above) with the count taken on the device
              ("bf16_size_classes", dict(B=1, L=256, K=5, d=136, V=3001, n_masked=250, masked_frac=None,
                                         sharp=("calibrated", 0.5, 2.5), unstable_frac=0.1), 21),
              # above 256 positions the second pass reads its count back, later ones run per size class
              ("bf16_readback", dict(B=2, L=160, K=5, d=136, V=3001, n_masked=150, masked_frac=None,
                                     sharp=("calibrated", 0.5, 2.5), unstable_frac=0.1), 22)]


@pytest.mark.parametrize("name,ov,seed", LAZY_CASES, ids=[c[0] for c in LAZY_CASES])
def test_lazy_projection(name, ov, seed):
    # Appendix A.6 "Layerwise projection": intermediate layers only inside the band theta_c <= c < theta_h,
    # down to the first disagreement; decisions are the eager ones
    base = CONFIGS["llada_late"].with_(name="lazy_" + name, sharp=("calibrated",), unstable_frac=0.4).with_(**ov)
    w = make_workload(base, seed)
    for P in (dataclasses.replace(O.LLADA, lazy=True), dataclasses.replace(O.DREAM, lazy=True, block=32)):
        g, o, _ = _check(w, P)
        eager = run_gpu(w, dataclasses.replace(P, lazy=False))
        m = w.mask != 0
        np.testing.assert_array_equal(g["token"][m], eager["token"][m])
        band = m & (g["confidence"] >= P.theta_c) & (g["confidence"] < P.theta_h)
        assert (g["persistence"][m & ~band] == -1).all() and np.isnan(g["stability"][m & ~band]).all()


@pytest.mark.parametrize("name,ov,seed", LAZY_CASES, ids=[c[0] for c in LAZY_CASES])
def test_lazy_projection_walking_every_position(name, ov, seed):
    # RPD_PARAM_LAZY_ALL: every masked position walks its layers down to its first disagreement (the
    # procedure of Appendix A.6 without the band restriction): persistence, drop and stability are
    # reported at every position and equal the eager projection's
    base = CONFIGS["llada_late"].with_(name="lazyall_" + name, sharp=("calibrated",), unstable_frac=0.4).with_(**ov)
    w = make_workload(base, seed)
    for P in (dataclasses.replace(O.LLADA, lazy=True, lazy_all=True),
              dataclasses.replace(O.DREAM, lazy=True, lazy_all=True, block=32)):
        g, o, _ = _check(w, P)
        eager = run_gpu(w, dataclasses.replace(P, lazy=False, lazy_all=False))
        m = w.mask != 0
        np.testing.assert_array_equal(g["token"][m], eager["token"][m])
        same = m & (g["persistence"] == eager["persistence"])
        assert same.sum() >= m.sum() - 2
        assert (g["persistence"][m] >= 1).all()
        assert np.abs(g["drop"][same] - eager["drop"][same]).max(initial=0.0) <= 2 * CONF_TOL


def test_lazy_projection_with_normalization_and_fp32():
    w = make_workload(CONFIGS["tiny"].with_(sharp=("calibrated",), unstable_frac=0.4), 8)
    _check(w, dataclasses.replace(O.LLADA, lazy=True), norm=(_gain(w, 3), 1e-6, False))
    wb = make_workload(CONFIGS["llada_late"].with_(name="lazy_norm", B=1, L=64, K=4, d=264, V=5003, n_masked=8,
                                                   masked_frac=None, sharp=("calibrated",), unstable_frac=0.4), 12)
    _check(wb, dataclasses.replace(O.LLADA, lazy=True), norm=(_gain(wb, 4), 1e-5, True))
    # 200 positions, most in the band: the passes after the first run once per size class, each
    # normalizing only its rows
    wc = make_workload(CONFIGS["llada_late"].with_(name="lazy_norm_classes", B=1, L=208, K=4, d=200, V=6007,
                                                   n_masked=200, masked_frac=None, sharp=("calibrated", 0.5, 2.5),
                                                   unstable_frac=0.1), 13)
    _check(wc, dataclasses.replace(O.LLADA, lazy=True), norm=(_gain(wc, 5), 1e-5, False))


# ------------------------------------------------------------- edge cases --

def _small_bf16(seed=5, **ov):
    kw = dict(name="edge", B=2, L=48, K=4, d=128, V=2000, n_masked=20, sharp=("calibrated",), unstable_frac=0.3)
    kw.update(ov)
    return make_workload(CONFIGS["llada_late"].with_(**kw), seed)


def test_no_masked_positions():
    w = _small_bf16(n_masked=0)
    g = run_gpu(w, O.LLADA, max_masked=0)
    assert (g["commit"] == 0).all() and (g["token"] == -1).all() and (g["n_commit"] == 0).all()
    g = run_gpu(w, O.LLADA, max_masked=-1)
    assert (g["commit"] == 0).all() and (g["n_commit"] == 0).all()


def test_empty_sequences_between_nonempty_ones():
    # sequences 1 and 3 of five have no masked position: they commit nothing while their neighbours do
    w = _small_bf16(seed=11, B=5, L=48, n_masked=12)
    for b in (1, 3):
        w.mask[b] = 0
        w.hidden[:, b] = np.uint16(0x7FC0)
    for P in (O.LLADA, O.strict(4, 0.5), O.Params(theta_s=3.5, w=15.0, block=32),
              O.Params(beta=0.0, theta_h=0.999999, theta_c=0.999998)):
        g, o, _ = _check(w, P, max_masked=int(w.mask.sum()))
        assert g["n_commit"][1] == 0 and g["n_commit"][3] == 0
        assert (g["n_commit"][[0, 2, 4]] >= 1).all()
    # also through the read-back of the count and the bound covering the whole canvas
    _check(w, O.LLADA, max_masked=-1)
    _check(w, O.LLADA, max_masked=w.cfg.B * w.cfg.L)


DUP_CASES = [  # name, overrides (rows = K * masked decide the projection variant)
    ("bf16_s32", dict(B=1, L=64, K=4, d=264, V=5003, n_masked=8)),
    ("bf16_s64", dict(B=2, L=40, K=3, d=512, V=4099, n_masked=10)),
    ("bf16_big128", dict(B=2, L=40, K=4, d=520, V=7001, n_masked=12)),
    ("bf16_big", dict(B=1, L=80, K=3, d=200, V=6007, n_masked=80)),
    ("bf16_big_row_split", dict(B=2, L=256, K=4, d=136, V=30011, n_masked=None, masked_frac=1.0)),
    ("f32", dict(B=1, L=64, K=3, d=256, V=4096, n_masked=40, dtype="f32")),
    # more than 512 vocabulary tiles (768): the tie check reads the tile states past the first 512 again
    ("bf16_s32_768_tiles", dict(B=1, L=64, K=4, d=128, V=140001, n_masked=8)),
]


def _duplicate_rows(w, shifts):
    """Copy the unembedding row of every layer's target token to the rows
    `t + s` (mod V) for each shift s, so that the top logit is an exact tie
    (gap 0) between the target and its copies: the lowest index must win."""
    w.w_u = w.w_u.copy()   # the cached matrix stays intact
    V = w.cfg.V
    pos = O.masked_positions(w.mask)
    st = O.project_layer_stats(w.hidden, w.w_u, w.cfg.dtype, pos)
    tops = sorted({int(t) for t in st["argmax"].ravel()})
    for t in tops:
        for s in shifts:
            u = (t + s) % V
            if u not in tops:
                w.w_u[u] = w.w_u[t]
    return tops


@pytest.mark.parametrize("name,ov", DUP_CASES, ids=[c[0] for c in DUP_CASES])
@pytest.mark.parametrize("where", ["near", "far"])
def test_exact_ties_take_the_lowest_index(name, ov, where):
    # An exact tie (gap 0 in exact arithmetic) is never excused by the comparator: duplicated rows must
    # give the lowest index at every layer, within a vocabulary tile ("near": copies 1-3 rows away, before
    # and after the target) and across tiles ("far": about V/2 away, in another tile and another XCD's
    # range). The streaming kernel sums each tile in its own chunk order and the MFMA tile with a single row
    # tile one order per XCD, so across their tiles the reduction resolves such ties; the eager and the lazy
    # path (every position walking) are both checked.
    cfg = CONFIGS["llada_late"].with_(name="dup_" + name, masked_frac=None, sharp=("calibrated", 0.0, 3.0),
                                      unstable_frac=0.3).with_(**ov)
    w = make_workload(cfg, 60)
    variant = rpd.projection_variant(cfg.K, cfg.B, cfg.L, cfg.d, cfg.V,
                                     rpd.DTYPE_BF16 if cfg.dtype == "bf16" else rpd.DTYPE_F32,
                                     max_masked=w.n_masked)
    assert name.startswith(variant), (name, variant)
    shifts = (1, 3, -2) if where == "near" else (cfg.V // 2 + 7, -(cfg.V // 2) - 5)
    _duplicate_rows(w, shifts)
    o = run_oracle(w, O.LLADA)
    m = w.mask != 0
    assert (o["layer_gap"][:, m] == 0.0).mean() > 0.9     # nearly every position's top is an exact tie
    lazy = dataclasses.replace(O.LLADA, lazy=True, lazy_all=True)
    for P in (O.LLADA,) + ((lazy,) if w.n_masked <= 100 else ()):   # the lazy oracle projects row by row
        _check(w, P)     # an exact tie is never excused: any other index than the oracle's fails


@pytest.mark.parametrize("name,ov", DUP_CASES, ids=[c[0] for c in DUP_CASES])
def test_zero_hidden_rows_give_the_uniform_distribution(name, ov):
    # Eq. 1 on z = 0: every logit exactly 0, p = 1/V, H = ln V, c = 1/V, and the argmax is index 0 (the
    # lowest index among V exact ties) at every layer
    cfg = CONFIGS["llada_late"].with_(name="zero_" + name, masked_frac=None).with_(**ov)
    w = make_workload(cfg, 61)
    w.hidden[:, w.mask != 0] = 0
    g, o, rep = _check(w, O.LLADA)
    m = w.mask != 0
    V = cfg.V
    assert (g["layer_argmax"][:, m] == 0).all() and (g["token"][m] == 0).all()
    np.testing.assert_allclose(g["layer_entropy"][:, m], math.log(V), atol=2e-3)
    np.testing.assert_allclose(g["layer_conf"][:, m], 1.0 / V, rtol=1e-3)
    assert not (g["flags"][m] & rpd.FLAG_CANDIDATE).any()
    assert (g["n_commit"] == (w.mask.sum(1) > 0)).all()     # the fallback alone commits


SMALL_V_CASES = [   # name (the projection variant), overrides; d = 264: four full 64-wide chunks and a tail
    ("bf16_s32", dict(B=1, L=64, K=4, d=264, n_masked=8)),
    ("bf16_big128", dict(B=1, L=64, K=4, d=264, n_masked=24)),
    ("bf16_big", dict(B=1, L=80, K=4, d=264, n_masked=64)),
    ("f32", dict(B=1, L=64, K=3, d=72, n_masked=10, dtype="f32")),
]


@pytest.mark.parametrize("name,ov", SMALL_V_CASES, ids=[c[0] for c in SMALL_V_CASES])
@pytest.mark.parametrize("V", [1, 2, 255, 257])
def test_vocabularies_smaller_than_a_tile(name, ov, V):
    # fewer vocabulary rows than one 256-row tile (or just above it): one ragged tile for the MFMA forms, tiles
    # of one or two rows for the streaming form. V = 1 is a point mass: H = 0, c = 1, argmax 0, so every
    # masked position is a candidate through theta_h and, with zero entropy, every one commits.
    cfg = CONFIGS["llada_late"].with_(name=f"smallV{V}_{name}", masked_frac=None, V=max(V, 2),
                                      sharp=("calibrated", 0.0, 3.0), unstable_frac=0.3).with_(**ov)
    w = make_workload(cfg, 70 + V)
    if V == 1:
        w.w_u = np.ascontiguousarray(w.w_u[:1])
        w.cfg = w.cfg.with_(V=1)
    variant = rpd.projection_variant(w.cfg.K, w.cfg.B, w.cfg.L, w.cfg.d, w.cfg.V,
                                     rpd.DTYPE_BF16 if w.cfg.dtype == "bf16" else rpd.DTYPE_F32,
                                     max_masked=w.n_masked)
    assert name == variant, (name, variant)
    for P in (O.LLADA, O.strict(w.cfg.K, 1.0)):
        g, o, _ = _check(w, P)
        if V == 1:
            m = w.mask != 0
            assert (g["token"][m] == 0).all() and (g["entropy"][m] == 0.0).all() and (g["confidence"][m] == 1.0).all()
            assert (g["commit"][m] == 1).all()


MANY_LAYER_CASES = [   # name (the projection variant), overrides
    ("bf16_s64", dict(B=1, L=40, K=64, d=136, V=3001, n_masked=1)),
    ("bf16_big128", dict(B=1, L=40, K=13, d=136, V=3001, n_masked=8)),
    ("bf16_big", dict(B=2, L=40, K=64, d=136, V=3001, n_masked=4)),
]


@pytest.mark.parametrize("name,ov", MANY_LAYER_CASES, ids=[c[0] + "_K%d" % c[1]["K"] for c in MANY_LAYER_CASES])
def test_many_layers(name, ov):
    # K = 13 (several layers per reduction wave, K above k_max = 6, so Eq. 4 caps the persistence) and
    # K = 64 (the largest the boundary takes: one lane per layer in the stability evaluation), eager and
    # with the lazy walk over every position
    cfg = CONFIGS["llada_late"].with_(name=f"layers_{name}", masked_frac=None, sharp=("calibrated", 0.0, 4.0),
                                      unstable_frac=0.3).with_(**ov)
    w = make_workload(cfg, 90 + cfg.K)
    variant = rpd.projection_variant(cfg.K, cfg.B, cfg.L, cfg.d, cfg.V, rpd.DTYPE_BF16, max_masked=w.n_masked)
    assert name == variant, (name, variant)
    for P in (O.LLADA, O.strict(cfg.K, 1.0), dataclasses.replace(O.LLADA, lazy=True, lazy_all=True)):
        _check(w, P)


def test_all_masked_and_single_layer():
    w = _small_bf16(n_masked=48)
    _check(w, O.LLADA)
    w1 = _small_bf16(n_masked=30, K=1)
    _check(w1, O.Params(theta_s=1.0, w=1.0))


@pytest.mark.parametrize("beta", [0.0, 0.5, 2.0, math.inf])
def test_budget_extremes(beta):
    w = _small_bf16(seed=7)
    P = O.Params(theta_s=2.5, w=20.0, beta=beta)
    _check(w, P)


@pytest.mark.parametrize("n_masked", [4, 3])
def test_small_call_four_sequences(n_masked):
    # a late-decode call over four sequences (64 and 48 projected rows, the 64-row streaming form): budget,
    # RPD-block and fallback per sequence
    w = _small_bf16(seed=9, B=4, L=64, n_masked=n_masked)
    for P in (O.LLADA, O.Params(theta_s=3.5, w=15.0, block=32), O.strict(4, 0.5),
              O.Params(beta=0.0, theta_h=0.999999, theta_c=0.999998)):
        g, o, _ = _check(w, P)
        assert (g["n_commit"] >= 1).all()


def test_fewer_masked_than_window_and_tiny_window():
    w = _small_bf16(seed=8, n_masked=5)
    _check(w, O.Params(beta=0.0, theta_h=0.999999, theta_c=0.999998))
    _check(w, O.Params(beta=0.0, window=2, theta_h=0.999999, theta_c=0.999998))


def test_nan_in_masked_row_is_contained():
    w = _small_bf16(seed=9)
    i = int(np.nonzero(w.mask[0])[0][3])
    w.hidden[:, 0, i, 5] = np.uint16(0x7FC0)      # one NaN element in every layer's row
    g = run_gpu(w, O.Params(beta=100.0))
    assert np.isnan(g["entropy"][0, i]) and np.isnan(g["confidence"][0, i])
    assert not (g["flags"][0, i] & rpd.FLAG_CANDIDATE)
    later = np.nonzero(w.mask[0])[0]
    later = later[later > i]
    assert not ((g["commit"][0, later] != 0) & ((g["flags"][0, later] & rpd.FLAG_FALLBACK) == 0)).any()
    _check(w, O.Params(beta=100.0))


def test_masked_hint_variants_agree_and_overflow_flagged():
    w = _small_bf16(seed=10)
    P = O.DREAM
    a = run_gpu(w, P)
    b = run_gpu(w, P, max_masked=-1)
    c = run_gpu(w, P, max_masked=w.cfg.B * w.cfg.L)
    # the exact count and -1 plan the same tiling: identical bits. A looser
    # bound may select another projection tiling, which changes only the
    # order of the fp32 sums: the discrete outputs agree, floats to rounding.
    for k in a:
        if k != "status":
            np.testing.assert_array_equal(a[k], b[k], err_msg=k)
            if a[k].dtype.kind == "f":
                np.testing.assert_allclose(a[k], c[k], rtol=1e-5, atol=1e-5, err_msg=k)
            else:
                np.testing.assert_array_equal(a[k], c[k], err_msg=k)
    assert a["status"][0] == 0
    d = run_gpu(w, P, max_masked=w.n_masked - 3)
    assert d["status"][0] & rpd.DEVICE_STATUS_MASKED_OVERFLOW


def test_deterministic_bitwise():
    w = make_workload(CONFIGS["llada_late"].with_(name="det", d=512, V=9000, L=128, n_masked=40,
                                                  sharp=("calibrated",)), 21)
    t = to_device(w)
    a = run_gpu(w, O.LLADA, tensors=t)
    b = run_gpu(w, O.LLADA, tensors=t)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)


@pytest.mark.parametrize("block", [0, 32, 5])
def test_gate_commit_matches_oracle_selection(block):
    rng = np.random.default_rng(3)
    K, B, L = 6, 3, 200
    mask = (rng.random((B, L)) < 0.7).astype(np.uint8)
    y = rng.integers(0, 50, size=(K, B, L)).astype(np.int32)
    keep = rng.random((B, L)) < 0.7               # many agreeing suffixes
    for l in range(K - 1):
        y[l][keep] = y[K - 1][keep]
    conf = rng.uniform(0.3, 1.0, size=(K, B, L)).astype(np.float32)
    ent = rng.exponential(0.7, size=(K, B, L)).astype(np.float32)
    P = O.Params(theta_s=4.5, w=10.0, beta=3.0, block=block)
    pos = O.masked_positions(mask)
    layer = {"argmax": np.array([y[:, b, i] for b, i in pos]).reshape(-1, K),
             "conf": np.array([conf[:, b, i] for b, i in pos], np.float64).reshape(-1, K),
             "entropy": np.array([ent[:, b, i] for b, i in pos], np.float64).reshape(-1, K)}
    # inside the agreement suffix the final token's probability is the layer's top probability
    layer["p_final"] = np.where(layer["argmax"] == layer["argmax"][:, -1:], layer["conf"], 0.0)
    o = O.select(mask, layer, P, pos)
    dev = "cuda:0"
    note("  gpu call: gate_commit K=6 B=3 L=200")
    g = rpd.gate_commit(torch.from_numpy(mask).to(dev), torch.from_numpy(y).to(dev),
                        torch.from_numpy(conf).to(dev), torch.from_numpy(ent).to(dev), gpu_params(P))
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in g.items()}
    m = mask != 0
    np.testing.assert_array_equal(g["token"][m], o["token"][m])
    np.testing.assert_array_equal(g["persistence"][m], o["persistence"][m])
    np.testing.assert_allclose(g["drop"][m], o["drop"][m], atol=1e-6)
    np.testing.assert_allclose(g["stability"][m], o["stability"][m], atol=1e-4)
    near = np.abs(o["stability"] - P.theta_s) < 1e-4
    np.testing.assert_array_equal(g["flags"][m & ~near] & 7, o["flags"][m & ~near] & 7)
    seq_ok = ~near.any(1)
    for b in np.nonzero(seq_ok)[0]:
        Nb = o["budget_prefix"][b][m[b]]
        if block == 0 and np.any(np.abs(Nb - P.beta) < 1e-4):
            continue
        np.testing.assert_array_equal(g["commit"][b], o["commit"][b])
        np.testing.assert_array_equal(g["flags"][b], o["flags"][b])
        np.testing.assert_allclose(g["upstream_entropy"][b][m[b]], o["upstream_entropy"][b][m[b]], atol=1e-4)
        assert g["n_commit"][b] == o["n_commit"][b]
    assert (g["token"][~m] == -1).all() and (g["commit"][~m] == 0).all()


def test_largest_canvas_the_boundary_takes():
    # B * L = 2^24 positions (4096 sequences of 4096), the boundary's maximum, with 300 masked positions
    # scattered over them: the compaction scans the whole canvas, the commitment runs one workgroup per
    # sequence (most of them empty), and every masked position is compared with the oracle
    from paper_2609_36452_amd.workload import Workload
    B, L, K, d, V, n = 4096, 4096, 2, 8, 300, 300
    assert B * L == 1 << 24
    src = make_workload(CONFIGS["llada_late"].with_(name="max_canvas_rows", B=1, L=n, K=K, d=d, V=V, n_masked=n,
                                                    masked_frac=None, sharp=("calibrated",), unstable_frac=0.3), 5)
    flat = np.sort(np.random.default_rng(5).choice(B * L, size=n, replace=False))
    hidden = np.zeros((K, B * L, d), np.uint16)
    hidden[:, flat] = src.hidden[:, 0]
    mask = np.zeros(B * L, np.uint8)
    mask[flat] = 1
    w = Workload(src.cfg.with_(name="max_canvas", B=B, L=L, n_masked=None), 5, src.w_u, hidden.reshape(K, B, L, d),
                 mask.reshape(B, L), np.full((B, L), -1, np.int64))
    g, o, _ = _check(w, O.LLADA)
    assert int(g["n_commit"].sum()) == int((w.mask.sum(1) > 0).sum())   # one masked position each: one commit


@pytest.mark.parametrize("n", [64, 72])
def test_big_tile_wide_row_offsets(n):
    # With more than 2^31 bytes of hidden states the big tile gathers rows through 64-bit addresses
    # instead of 32-bit buffer offsets. The same rows at the same relative order in a small canvas take
    # the buffer path: every output at the masked positions must agree bit for bit (and the small
    # canvas agrees with the oracle). n = 64: one 256-row tile; 72: two 192-row tiles.
    cfg = CONFIGS["llada_late"].with_(name=f"wide{n}", B=1, L=n, K=4, d=4096, V=3001, n_masked=n,
                                      masked_frac=None)
    w = make_workload(cfg, 40 + n)
    P = O.strict(4, 1.0)
    g_small, _, _ = _check(w, P)
    Lbig = 65600   # 4 layers x 65600 x 4096 bf16 = 2.15 GB
    assert 4 * Lbig * 4096 * 2 > 2 ** 31
    pos = torch.arange(n, device="cuda:0") * 911 + 17   # increasing, spread over the canvas
    assert int(pos[-1]) < Lbig
    hidden_s, w_u, _ = to_device(w)
    hidden = torch.zeros((4, 1, Lbig, 4096), dtype=torch.bfloat16, device="cuda:0")
    hidden[:, 0, pos] = hidden_s[:, 0, :]
    mask = torch.zeros((1, Lbig), dtype=torch.uint8, device="cuda:0")
    mask[0, pos] = 1
    variant = rpd.projection_variant(4, 1, Lbig, 4096, 3001, hidden.dtype, max_masked=n)
    note(f"  wide canvas L={Lbig}, {n} masked, variant {variant}")
    assert variant == ("bf16_big" if n == 64 else "bf16_big192")
    out = rpd.score_commit(hidden, w_u, mask, gpu_params(P), max_masked=n, layer_stats=True)
    torch.cuda.synchronize()
    pc = pos.cpu().numpy()
    for k, v in out.items():
        a = v.cpu().numpy()
        b = g_small[k]
        if a.shape[-1] == Lbig:
            a = a[..., pc]
        assert a.shape == b.shape, k
        assert np.array_equal(np.ascontiguousarray(a).view(np.uint8), np.ascontiguousarray(b).view(np.uint8)), k
    del hidden, out
    torch.cuda.empty_cache()


# -------------------------------------------------------------- full size --

@pytest.fixture(scope="module")
def llada_wu():
    return draw_unembedding(126464, 4096, "bf16", 1)


def test_llada_late_full_oracle(llada_wu):
    """Late-decode LLaDA-8B shape (8 masked of 256, K=4): every position
    against the full oracle, with the launch configuration the benchmark times."""
    w = make_workload("llada_late", 1, w_u=llada_wu)
    for P in (O.strict(4, 1.0), O.LLADA):
        _check(w, P)


def _sampled(w, P, g, nsample, rng):
    """Oracle per-layer statistics at sampled masked positions, compared with
    the GPU's; scoring re-derived for those positions from the oracle."""
    pos = O.masked_positions(w.mask)
    pick = sorted(rng.choice(len(pos), size=min(nsample, len(pos)), replace=False))
    sel = [pos[a] for a in pick]
    st = O.project_layer_stats(w.hidden, w.w_u, w.cfg.dtype, sel)
    K = w.cfg.K
    bad = []
    for a, (b, i) in enumerate(sel):
        for l in range(K):
            tie = st["gap"][a, l] < gap_tol(w.cfg.d, st["absbound"][a, l])
            if abs(g["layer_entropy"][l, b, i] - st["entropy"][a, l]) > ENTROPY_TOL:
                bad.append(("entropy", l, b, i))
            if abs(g["layer_conf"][l, b, i] - st["conf"][a, l]) > CONF_TOL:
                bad.append(("conf", l, b, i))
            if g["layer_argmax"][l, b, i] != st["argmax"][a, l] and not tie:
                bad.append(("argmax", l, b, i))
        k_i = O.persistence(st["argmax"][a])
        r_i = O.confidence_drop(st["p_final"][a], k_i)
        if g["persistence"][b, i] != k_i and not (st["gap"][a] < gap_tol(w.cfg.d, st["absbound"][a])).any():
            bad.append(("persistence", b, i))
        if g["persistence"][b, i] == k_i and abs(g["drop"][b, i] - r_i) > 2 * CONF_TOL:
            bad.append(("drop", b, i))
    assert not bad, bad[:10]


def _commit_property(g, mask, P):
    """Prefix-sum identity on the GPU's own outputs: a candidate is committed
    iff the entropy of earlier masked non-candidates is within the budget
    (fp64 recomputation; fp32 near-ties tolerated), else the fallback fired."""
    B = mask.shape[0]
    for b in range(B):
        idx = np.nonzero(mask[b])[0]
        if idx.size == 0:
            continue
        cand = (g["flags"][b, idx] & rpd.FLAG_CANDIDATE) > 0
        H = g["entropy"][b, idx].astype(np.float64)
        N = np.concatenate([[0.0], np.cumsum(np.where(cand, 0.0, H))[:-1]])
        expect = cand & (N <= P.beta)
        got = g["commit"][b, idx] != 0
        fb = (g["flags"][b, idx] & rpd.FLAG_FALLBACK) > 0
        if fb.any():
            assert not expect[np.abs(N - P.beta) > 1e-3].any()
            assert got.sum() == 1 and fb.sum() == 1
            win = idx[:P.window]
            assert idx[fb][0] in win
            assert g["confidence"][b, idx[fb][0]] == np.nanmax(g["confidence"][b, win])
        else:
            diff = got != expect
            assert not (diff & (np.abs(N - P.beta) > 1e-3 * (1 + P.beta))).any()
        assert g["n_commit"][b] == got.sum()


@pytest.mark.parametrize("cfgname,seed,nsample", [("llada_100", 2, 12), ("llada_25", 102, 12),
                                                   ("llada_10", 202, 12), ("llada_batched", 4, 10),
                                                   ("llada_batched32", 204, 8)])
def test_llada_full_size_sampled(cfgname, seed, nsample, llada_wu):
    w = make_workload(cfgname, seed, w_u=llada_wu)
    P = O.strict(4, 1.0)
    g = run_gpu(w, P)
    _sampled(w, P, g, nsample, np.random.default_rng(seed))
    _commit_property(g, w.mask, P)


def test_dream_full_size_sampled():
    w = make_workload("dream_50", 3)
    for P in (O.strict(4, 1.0), O.DREAM):
        g = run_gpu(w, P)
        _commit_property(g, w.mask, P)
    _sampled(w, P, g, 10, np.random.default_rng(3))


# Whole full-size calls against the oracle at every masked position and layer (the fp64 projection of
# 64-256 positions at the LLaDA-8B / Dream-7B shapes takes the host some seconds to a minute). The oracle's
# per-layer statistics are computed once per workload and reused for every rule and budget.

@pytest.mark.slow
@pytest.mark.parametrize("cfgname,seed", [("llada_100", 2), ("llada_50", 102), ("llada_25", 202), ("llada_10", 302)])
def test_llada_full_size_full_oracle(cfgname, seed, llada_wu):
    w = make_workload(cfgname, seed, w_u=llada_wu)
    for P in (O.strict(4, 0.5), O.strict(4, 1.0), O.strict(4, 2.0), O.LLADA):
        note(f"  rule theta_s={P.theta_s} w={P.w} beta={P.beta}")
        _check(w, P)


@pytest.mark.slow
@pytest.mark.parametrize("cfgname,seed", [("dream_100", 3), ("dream_50", 103)])
def test_dream_full_size_full_oracle(cfgname, seed):
    w = make_workload(cfgname, seed)
    for P in (O.strict(4, 1.0), O.DREAM):
        note(f"  rule theta_s={P.theta_s} w={P.w} beta={P.beta}")
        _check(w, P)


class _Seq:
    """One sequence of a batched workload, as a workload of its own (the
    oracle treats sequences independently)."""

    def __init__(self, w, b):
        self.cfg = w.cfg.with_(name=f"{w.cfg.name}[{b}]", B=1)
        self.seed = w.seed
        self.w_u = w.w_u
        self.hidden = w.hidden[:, b:b + 1]
        self.mask = w.mask[b:b + 1]

    @property
    def n_masked(self):
        return int(self.mask.sum())


@pytest.mark.slow
@pytest.mark.parametrize("cfgname,seed,seqs", [("llada_batched", 4, (0, 5)), ("llada_batched32", 204, (17,))])
def test_batched_whole_sequences_full_oracle(cfgname, seed, seqs, llada_wu):
    # the batch runs as one call (12,288 / 49,152 projected rows: the 256 x 256 tiles in per-XCD groups);
    # whole sequences of it are compared with the oracle run on that sequence alone
    w = make_workload(cfgname, seed, w_u=llada_wu)
    P = O.strict(4, 1.0)
    g = run_gpu(w, P)
    K = w.cfg.K
    for b in seqs:
        sw = _Seq(w, b)
        gs = {k: (v[:, b:b + 1] if v.ndim == 3 else v[b:b + 1]) for k, v in g.items() if k != "status"}
        o = run_oracle(sw, P)
        rep = compare(gs, o, sw.mask, P, w.cfg.d)
        note(f"  sequence {b}: " + rep.summary()[:300])
        assert rep.ok(), rep.summary()
        assert sum(rep.excused.values()) <= max(2, 0.05 * sw.n_masked * (K + 3)), rep.summary()


BAND_HEAVY = dict(sharp=("calibrated", 1.0, 2.2), unstable_frac=0.05)


@pytest.mark.parametrize("cfgname,seed,ov", [("llada_25", 102, {}), ("llada_100", 2, {}), ("llada_batched", 4, {}),
                                             ("llada_100", 5, BAND_HEAVY)],
                         ids=["llada_25", "llada_100", "llada_batched", "llada_100_band_heavy"])
def test_lazy_full_size_matches_eager(cfgname, seed, ov, llada_wu):
    # At the benchmark's sizes (64 masked positions: one streaming pass per layer; 256: passes launched per
    # size class, with about half the positions in the band for the last case, so that later passes list
    # more than 128 rows; 3072: counts read back), lazy projection takes the eager path's decisions: tokens,
    # candidacy and, inside the band, persistence and drop. A difference is allowed only at a near-tie of the
    # oracle's statistics for that position (the two paths project a layer with different tile plans).
    w = make_workload(CONFIGS[cfgname].with_(**ov), seed, w_u=llada_wu)
    P = O.LLADA
    eager = run_gpu(w, P)
    lazy = run_gpu(w, dataclasses.replace(P, lazy=True))
    m = w.mask != 0
    cand = lambda g: (g["flags"] & rpd.FLAG_CANDIDATE) > 0   # noqa: E731
    band = m & (eager["confidence"] >= P.theta_c) & (eager["confidence"] < P.theta_h)
    diff = m & ((lazy["token"] != eager["token"]) | (cand(lazy) != cand(eager))
                | (band & (lazy["persistence"] != eager["persistence"])))
    bi = [tuple(int(x) for x in v) for v in np.argwhere(diff)]
    note(f"    {int(m.sum())} positions, {int(band.sum())} in the band, {len(bi)} differing")
    assert len(bi) <= max(2, 0.01 * int(m.sum()))
    if bi:
        st = O.project_layer_stats(w.hidden, w.w_u, w.cfg.dtype, bi)
        for a, (b, i) in enumerate(bi):
            c = st["conf"][a, -1]
            near = ((st["gap"][a] < gap_tol(w.cfg.d, st["absbound"][a])).any()
                    or min(abs(c - P.theta_c), abs(c - P.theta_h)) < CONF_TOL
                    or abs(eager["stability"][b, i] - P.theta_s) <= P.w * 2 * CONF_TOL)
            assert near, (b, i)
    same = band & ~diff
    assert np.abs(lazy["drop"][same] - eager["drop"][same]).max(initial=0.0) <= 2 * CONF_TOL
    assert (lazy["persistence"][m & ~band & ~diff] == -1).all()
    _commit_property(lazy, w.mask, P)
