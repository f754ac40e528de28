"""The C-ABI library loads on the host and exports every symbol that
include/*.h declares; host-side validation answers without touching a GPU."""
import ctypes
import glob
import math
import os
import re

import pytest

from paper_2609_36452_amd import binding as rpd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        txt = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(rpd_[a-z_]+)\s*\(", txt))
    return names


def test_exports_every_declared_symbol():
    names = _declared()
    assert {"rpd_score_commit", "rpd_score_commit_timed", "rpd_gate_commit", "rpd_workspace_size",
            "rpd_status_string", "rpd_last_error", "rpd_abi_version"} <= names
    L = ctypes.CDLL(rpd._LIB_PATH)
    for n in sorted(names):
        assert hasattr(L, n), n


def test_struct_layouts():
    # rpd_params of include/rpd.h: eight 4-byte fields, then block and logit_scale
    assert ctypes.sizeof(rpd.RpdParams) == 40 and rpd.RpdParams.block.offset == 32
    assert rpd.RpdParams.logit_scale.offset == 36
    # rpd_problem: six ints, three pointers, max_masked, then the normalization fields
    assert rpd.RpdProblem.norm_weight.offset == 56 and rpd.RpdProblem.norm_eps.offset == 64
    assert ctypes.sizeof(rpd.RpdProblem) == 72


def test_version_and_status_strings():
    assert rpd.abi_version() == 3 == rpd.ABI_VERSION
    hdr = open(os.path.join(ROOT, "include", "rpd.h")).read()
    assert "#define RPD_ABI_VERSION 3\n" in hdr
    assert rpd.status_string(0) == "ok"
    assert rpd.status_string(4) == "workspace too small"


def _a256(x):
    return (x + 255) // 256 * 256


def _lazy(cap):
    # per-position state of the lazy projection: one 8-byte and eight 4-byte arrays
    return _a256(cap * 8) + 8 * _a256(cap * 4)


def test_workspace_size():
    # late-decode LLaDA shape: header + row list + (32 rows x 512 tiles of 256 vocabulary rows x 16 B)
    n = rpd.workspace_size(4, 1, 256, 4096, 126464, rpd.DTYPE_BF16, max_masked=8)
    assert n == 256 + 1024 + _a256(32 * 512 * 16) + _lazy(8)
    # 10% masked: 104 rows x 494 tiles of 256 vocabulary rows (one 128-row MFMA tile per vocabulary tile)
    n = rpd.workspace_size(4, 1, 256, 4096, 126464, rpd.DTYPE_BF16, max_masked=26)
    assert n == 256 + 1024 + _a256(104 * 494 * 16) + _lazy(26)   # 65..128 rows: MFMA tiles, V / 256 of them
    # 100% masked: 1024 rows x 494 tiles of 256 vocabulary rows
    n = rpd.workspace_size(4, 1, 256, 4096, 126464, rpd.DTYPE_BF16, max_masked=256)
    assert n == 256 + 1024 + _a256(1024 * 494 * 16) + _lazy(256)
    # with the final normalization: + the normalized rows (32 x 4096 bf16)
    n = rpd.workspace_size(4, 1, 256, 4096, 126464, rpd.DTYPE_BF16, max_masked=8, norm=True)
    assert n == 256 + 1024 + _a256(32 * 512 * 16) + _lazy(8) + 32 * 4096 * 2
    assert rpd.workspace_size(0, 1, 256, 4096, 126464, rpd.DTYPE_BF16) == 0
    assert rpd.workspace_size(65, 1, 256, 4096, 126464, rpd.DTYPE_BF16) == 0
    assert rpd.workspace_size(4, 1, 256, 4096, 126464, 7) == 0


def test_projection_variant_thresholds():
    pv = lambda n, dt=rpd.DTYPE_BF16: rpd.projection_variant(4, 1, 256, 4096, 126464, dt, max_masked=n)  # noqa: E731
    assert [pv(n) for n in (1, 8, 9, 16, 17, 32, 33, 48, 49, 64, 65, 256)] == \
        ["bf16_s32", "bf16_s32", "bf16_s64", "bf16_s64", "bf16_big128", "bf16_big128", "bf16_big192", "bf16_big192",
         "bf16_big", "bf16_big", "bf16_big192", "bf16_big"]
    # 65..128 rows: one 128-row MFMA tile; above: the tile of 192 or 256 rows that pads the rows less (ties to 256)
    assert [pv(n) for n in (96, 144, 192, 225)] == ["bf16_big192", "bf16_big192", "bf16_big", "bf16_big192"]
    assert pv(8, rpd.DTYPE_F32) == "f32" and pv(256, rpd.DTYPE_F32) == "f32"
    assert pv(-1) == "bf16_big"          # -1 plans for every position masked
    with pytest.raises(rpd.RpdError):
        rpd.projection_variant(0, 1, 256, 4096, 126464, rpd.DTYPE_BF16)


def _call(prob, params, outs, ws=256, ws_bytes=1 << 40):
    L = rpd.lib()
    s = L.rpd_score_commit(ctypes.byref(prob) if prob is not None else None,
                           ctypes.byref(params) if params is not None else None,
                           ctypes.byref(outs) if outs is not None else None, ws, ws_bytes, None)
    return s, rpd.last_error()


def _fake_outputs():
    # non-NULL, never dereferenced: validation fails before anything is enqueued
    return rpd.RpdOutputs(*([4096] * 10 + [None] * 4))


def _prob(**kw):
    base = dict(K=4, B=1, L=256, d=4096, V=126464, dtype=0, hidden=4096, w_u=8192, mask=64, max_masked=8,
                norm_weight=None, norm_eps=1e-5, norm_final=0)
    base.update(kw)
    return rpd.RpdProblem(base["K"], base["B"], base["L"], base["d"], base["V"], base["dtype"],
                          base["hidden"], base["w_u"], base["mask"], base["max_masked"], base["norm_weight"],
                          base["norm_eps"], base["norm_final"])


def _params(**kw):
    p = dict(theta_h=0.9, theta_c=0.6, theta_s=3.5, w=15.0, k_max=6, beta=4.0, window=32, flags=0, block=0,
             logit_scale=1.0)
    p.update(kw)
    return rpd.RpdParams(**p)


@pytest.mark.parametrize("kw,status", [
    (dict(K=0), 2), (dict(K=65), 2), (dict(B=0), 2), (dict(L=0), 2), (dict(d=0), 2), (dict(d=(1 << 20) + 8), 2),
    (dict(V=0), 2),
    (dict(B=1 << 13, L=1 << 12), 2), (dict(dtype=3), 5), (dict(d=4100), 5), (dict(w_u=8200), 5),
    (dict(hidden=None), 1), (dict(mask=None), 1),
    (dict(norm_weight=8200), 5), (dict(norm_weight=8192, norm_eps=-1.0), 3),
    (dict(norm_weight=8192, norm_eps=math.nan), 3), (dict(norm_weight=8192, norm_final=2), 3),
])
def test_problem_validation(kw, status):
    s, msg = _call(_prob(**kw), _params(), _fake_outputs())
    assert s == status, msg
    assert msg


@pytest.mark.parametrize("kw", [dict(theta_c=0.95), dict(theta_c=-0.1), dict(w=-1.0), dict(k_max=0),
                                dict(beta=-1.0), dict(beta=math.nan), dict(window=0), dict(flags=2), dict(flags=4), dict(flags=7),
                                dict(theta_h=math.nan), dict(theta_s=math.inf), dict(block=-1),
                                dict(logit_scale=-1.0), dict(logit_scale=math.inf)])
def test_param_validation(kw):
    s, msg = _call(_prob(), _params(**kw), _fake_outputs())
    assert s == 3, msg


def test_null_and_workspace_checks():
    assert _call(None, _params(), _fake_outputs())[0] == 1
    assert _call(_prob(), None, _fake_outputs())[0] == 1
    assert _call(_prob(), _params(), None)[0] == 1
    o = _fake_outputs()
    o.drop = None
    assert _call(_prob(), _params(), o)[0] == 1
    o = _fake_outputs()
    o.layer_conf = 4096                       # only one of the three per-layer outputs
    assert _call(_prob(), _params(), o)[0] == 1
    s, msg = _call(_prob(), _params(), _fake_outputs(), ws_bytes=1000)
    assert s == 4 and "needed" in msg
    assert _call(_prob(), _params(), _fake_outputs(), ws=None)[0] == 1
    assert _call(_prob(), _params(), _fake_outputs(), ws=256 + 16)[0] == 5


def test_noalloc_refuses_problems_beyond_its_array_before_any_device_call():
    # RPD_NOALLOC_SCRATCH_BYTES = 64 MiB; 32768 projected rows at the LLaDA-8B vocabulary need about 260 MB
    p = _prob(B=8, L=1024, max_masked=-1)
    need = int(rpd.lib().rpd_workspace_size(ctypes.byref(p)))
    assert need > rpd.NOALLOC_SCRATCH_BYTES
    s = rpd.lib().rpd_score_commit_noalloc(ctypes.byref(p), ctypes.byref(_params()), ctypes.byref(_fake_outputs()),
                                           None)
    assert s == 4 and "workspace" in rpd.last_error()
    assert rpd.lib().rpd_score_commit_noalloc(None, ctypes.byref(_params()), ctypes.byref(_fake_outputs()), None) == 1


def test_gate_validation():
    L = rpd.lib()
    q = _params()
    o = _fake_outputs()
    assert L.rpd_gate_commit(4, 1, 16, None, 64, 64, 64, ctypes.byref(q), ctypes.byref(o), None) == 1
    assert L.rpd_gate_commit(0, 1, 16, 64, 64, 64, 64, ctypes.byref(q), ctypes.byref(o), None) == 2
    bad = _params(beta=-2.0)
    assert L.rpd_gate_commit(4, 1, 16, 64, 64, 64, 64, ctypes.byref(bad), ctypes.byref(o), None) == 3


def test_apply_commit_validation():
    L = rpd.lib()
    # (B, L, mask, canvas, commit, token, progress, progress_len, step, stream); nothing is launched
    assert L.rpd_apply_commit(1, 16, None, 64, 64, 64, None, 0, None, None) == 1
    assert L.rpd_apply_commit(1, 16, 64, 64, 64, None, None, 0, None, None) == 1
    assert L.rpd_apply_commit(1, 16, 64, 64, 64, 64, None, 0, 64, None) == 1      # step needs progress
    assert L.rpd_apply_commit(0, 16, 64, 64, 64, 64, None, 0, None, None) == 2
    assert L.rpd_apply_commit(1 << 13, 1 << 12, 64, 64, 64, 64, None, 0, None, None) == 2
    assert L.rpd_apply_commit(1, 16, 64, 64, 64, 64, 64, -1, None, None) == 3
    assert "progress" in rpd.last_error()
