"""The seeded input generator: exact bf16 rounding, determinism, shapes."""
import numpy as np
import torch

from paper_2609_36452_amd.workload import (CONFIGS, bf16_bits_to_f32, make_workload,
                                           round_bf16_bits)


def test_bf16_rounding_matches_torch_on_f32_values():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10 ** rng.uniform(-6, 6, 100000),
                        np.array([1.00390625, 1.01171875, -1.00390625, 0.0, -0.0], np.float32)]).astype(np.float32)
    ours = round_bf16_bits(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


def test_bf16_rounding_is_single_rounding_from_f64():
    # 1 + 2^-8 + 2^-30 must round up (a detour through f32 would keep it a tie)
    v = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert bf16_bits_to_f32(round_bf16_bits(np.array([v])))[0] == np.float32(1.0 + 2.0 ** -7)


def test_deterministic_and_shaped():
    cfg = CONFIGS["tiny"]
    a = make_workload(cfg, 3)
    b = make_workload(cfg, 3)
    for k in ("w_u", "hidden", "mask", "targets"):
        np.testing.assert_array_equal(getattr(a, k), getattr(b, k))
    assert a.hidden.shape == (cfg.K, cfg.B, cfg.L, cfg.d)
    assert a.mask.sum() == 40
    um = a.mask[0] == 0
    assert np.isnan(a.hidden[:, 0, um]).all() and np.isfinite(a.hidden[:, 0, ~um]).all()


def test_bf16_config_small():
    cfg = CONFIGS["llada_late"].with_(d=128, V=1000, L=32)
    w = make_workload(cfg, 1)
    assert w.w_u.dtype == np.uint16 and w.hidden.dtype == np.uint16
    h = bf16_bits_to_f32(w.hidden[:, 0, w.mask[0] == 1])
    assert np.isfinite(h).all()
    assert w.mask.sum() == 8


def test_calibrated_level_range():
    # calibrated mode draws the target-logit level from ln V + U(lo, hi): (-3, 6) by default, or the
    # offsets given in the sharpness tuple (the lazy-projection cases narrow it to fill the band)
    base = CONFIGS["llada_late"].with_(d=64, V=1000, L=200, n_masked=150, masked_frac=None)
    lnv = np.log(1000.0)
    for sharp, lo, hi in ((("calibrated",), -3.0, 6.0), (("calibrated", 0.5, 2.5), 0.5, 2.5)):
        w = make_workload(base.with_(sharp=sharp), 4)
        s = np.concatenate(w.meta["sharpness"])
        assert s.size == 150 and (s >= lnv + lo).all() and (s < lnv + hi).all()
        assert s.max() - s.min() > 0.8 * (hi - lo)     # spread over the range, not a point
