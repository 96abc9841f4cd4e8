"""Host-side parts of ``bench.py`` (no GPU): the algorithmic byte counts of
each workload against their closed forms, the workload names of the profile
summaries, the measured-traffic lookup keyed to the kernel sources, and the
single-GPU contract of the command line."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_algorithmic_bytes_7b():
    # packed signs k*d/8 + fp16 x + three fp16 rows per kept row + fp32 y, 1101 kept rows at s = 0.9
    k, d, n = 11008, 4096, 1101
    assert bench.algorithmic_bytes(k, d, 1, n, n, n) == k * d // 8 + 2 * d + 3 * 2 * d * n + 4 * d == 32_718_848


def test_algorithmic_bytes_forms():
    k, d, n = 11008, 4096, 1101
    # INT8 rows are d bytes, plus the float scales of the kept gate/up rows and of the columns of y
    assert bench.algorithmic_bytes(k, d, 1, n, n, n, int8=True) == 19_214_952
    # the decoder-block call reads the fp32 residual and the fp32 norm weight instead of the fp16 x
    plain = bench.algorithmic_bytes(k, d, 1, n, n, n)
    assert bench.algorithmic_bytes(k, d, 1, n, n, n, block=True) == plain - 2 * d + 4 * d + 4 * d
    # the non-gated MLP reads no W_up rows
    assert bench.algorithmic_bytes(16384, 4096, 1, 1638, 0, 1638) == 35_250_176
    # b tokens: b fp16 x rows and b fp32 y rows
    assert bench.algorithmic_bytes(k, d, 8, 6266, 6266, 6266) - bench.algorithmic_bytes(k, d, 1, 6266, 6266, 6266) \
        == 7 * (2 * d + 4 * d)


class _Args:
    def __init__(self, mlp="gated", shape="7b", batch=1):
        self.mlp, self.shape, self.batch = mlp, shape, batch


@pytest.mark.parametrize("args,tag", [
    (_Args(), "k_owned_7b_s0.9"),
    (_Args(mlp="int8"), "k_owned_7b_int8_s0.9"),
    (_Args(mlp="block"), "k_owned_7b_block_s0.9"),
    (_Args(mlp="relu"), "k_owned_opt6.7b_relu_s0.9"),
    (_Args(shape="13b"), "k_owned_13b_s0.88"),
    (_Args(mlp="int8", shape="13b"), "k_owned_13b_int8_s0.88"),
    (_Args(batch=4), "k_owned_7b_b4_union_s0.9"),
    (_Args(batch=8), "k_owned_7b_b8_union_s0.9"),
])
def test_workload_tags_name_committed_summaries(args, tag):
    assert bench.workload_tag(args) == tag
    for suffix in ("_trace.md", "_counters.txt"):
        assert os.path.exists(os.path.join(ROOT, "profiles", tag + suffix)), tag + suffix


def test_measured_traffic_follows_the_sources(tmp_path):
    good = tmp_path / "good.txt"
    good.write_text("# comment: ignored\nkernel: k\nsources_sha256: %s\ntraffic_bytes_per_launch: 1234\n"
                    % bench.kernel_sources_sha256())
    assert bench.measured_traffic(str(good)) == 1234
    stale = tmp_path / "stale.txt"
    stale.write_text("sources_sha256: %s\ntraffic_bytes_per_launch: 1234\n" % ("0" * 64))
    assert bench.measured_traffic(str(stale)) is None
    assert bench.measured_traffic(str(tmp_path / "missing.txt")) is None


def test_committed_counters_match_the_sources():
    """Every committed counter summary was taken on (or re-keyed to
    instruction-identical builds of) the current kernel sources, so the
    benchmark reports its traffic."""
    for tag in ("k_owned_7b_s0.9", "k_owned_7b_int8_s0.9", "k_owned_7b_block_s0.9", "k_owned_opt6.7b_relu_s0.9",
                "k_owned_13b_s0.88", "k_owned_13b_int8_s0.88", "k_owned_7b_b4_union_s0.9", "k_owned_7b_b8_union_s0.9"):
        assert bench.measured_traffic(os.path.join(ROOT, "profiles", tag + "_counters.txt")) is not None, tag


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr
