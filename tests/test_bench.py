"""bench.py without a GPU: the one-GPU contract, the roofline arithmetic and
the committed counter summary the benchmark reports HBM traffic from."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and not r.stdout


def test_algorithmic_cost_of_a_projection():
    # W_U read once (V*d bf16) plus the projected rows; 2 flops per multiply-add
    class Cfg:
        V, d, dtype = 126464, 4096, "bf16"
    by, fl = bench.proj_cost(Cfg, 32)
    assert by == 1036255232 == 126464 * 4096 * 2 + 32 * 4096 * 2
    assert fl == 2.0 * 32 * 126464 * 4096
    # below the ridge the bytes bound, above it the flops (2.5 PFLOP/s over 8 TB/s, in rows)
    assert bench.RIDGE_ROWS == 315
    by1, fl1 = bench.proj_cost(Cfg, 1024)
    assert fl1 / 2.5e15 > by1 / 8e12
    assert fl / 2.5e15 < by / 8e12


@pytest.mark.parametrize("variant", sorted(bench.VARIANT_SOURCES))
def test_every_variant_names_its_kernel_sources(variant):
    for f in bench.VARIANT_SOURCES[variant]:
        assert os.path.exists(os.path.join(bench.CSRC, f)), f
    assert bench.VARIANT_KERNEL[variant].startswith("k_proj_")


def test_source_hash_ignores_comments_and_layout_only():
    a = 'int f(int x) {  // twice\n  return 2 * x; /* doubled */ }\nconst char* s = "// kept";\n'
    b = 'int f(int x) {\n    return 2 * x;\n}\nconst char* s = "// kept";  // a new comment\n'
    assert bench.code_tokens(a) == bench.code_tokens(b)
    assert bench.code_tokens(a) != bench.code_tokens(a.replace("2 * x", "3 * x"))
    assert bench.code_tokens(a) != bench.code_tokens(a.replace('"// kept"', '"// changed"'))
    assert '"// kept"' in bench.code_tokens(a)


def test_committed_traffic_summary_matches_the_kernel_source():
    # the benchmark's default workload runs the 32-row streaming variant; its committed counter summary
    # must have been taken on the kernel source as it is now, or the bench line reports no traffic
    path = bench.traffic_path("bf16_s32", "llada_late")
    assert os.path.exists(path)
    t = bench.read_traffic("bf16_s32", "llada_late")
    assert t is not None, "the kernel source changed since the counters were taken: measure again"
    assert 1.0e9 < t < 1.2e9        # about the 1.036 GB that W_U and the rows occupy
