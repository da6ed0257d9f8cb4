"""Host-side logic of bench.py (CPU only): the one-GPU guard, argument
defaults, the algorithmic byte counts and the code hash that keeps counter
data attached to the kernels they were taken on."""

import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_steps_default_by_workload():
    assert bench.parse([]).steps == 50
    assert bench.parse(["--workload", "stack31_m512_h4096_i12288"]).steps == 32
    assert bench.parse(["--workload", "stack31_m512_h4096_i12288", "--steps", "3"]).steps == 3
    # the largest single-GPU configuration is the default line; the decode block is nested in it
    assert bench.parse([]).workload == "batch8x1024_h4096_i12288" == bench.DEFAULT_WORKLOAD
    assert bench.NESTED_WORKLOAD == "block32_h4096_i12288"


def test_trace_kernel_us_reads_the_committed_summary():
    """The live kernel time is compared with the same kernel's average in the
    committed rocprofv3 summary; the parser reads that file's table."""
    us = bench.trace_kernel_us("batch8x1024_h4096_i12288", "void lacache::gemm_tiled_kernel<true")
    assert us is not None and 100.0 < us < 5000.0
    assert bench.trace_kernel_us("no_such_workload", "x") is None


def test_stage_bytes_at_the_decode_block():
    # H = 4096, I = 12288, M = 32: 2IH + IH weight bytes plus scales and activations
    b = bench.stage_bytes(32, 4096, 12288)
    H, I, M = 4096, 12288, 32
    w_gu, w_d = 2 * I * H, H * I
    s_gu, s_d = 4 * (2 * I // 128) * (H // 128), 4 * (H // 128) * (I // 128)
    assert b["gateup_stream"] == w_gu + s_gu + M * H + 4 * M * H // 128 + 4 * M * I
    assert b["gateup"] == w_gu + s_gu + M * H + 4 * M * H // 128 + M * I + 4 * M * I // 128
    assert b["down"] == w_d + s_d + M * I + 4 * M * I // 128 + 2 * M * H
    assert b["gateup_stream"] == 102395904  # the figure the bench line reports


def test_code_hash_ignores_comments_and_blank_space_only():
    a = "int f(int x) {\n  return x + 1;  // one more\n}\n"
    b = "/* header */\nint f(int x) {\n\n    return x + 1;\n}  // end\n"
    c = "int f(int x) {\n  return x + 2;\n}\n"
    assert bench.code_hash([a]) == bench.code_hash([b])
    assert bench.code_hash([a]) != bench.code_hash([c])
