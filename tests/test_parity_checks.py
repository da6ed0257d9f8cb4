"""CPU tests of the GPU parity checks themselves: an output that follows the
MFMA model passes, and small planted mistakes (far below the old worst-case
envelope) fail. The "kernel output" here is simulated on the CPU from the
oracle's operands and the model; no GPU is involved."""

import numpy as np
import pytest

import oracle.ffn as O
import synth
from gpu_util import (check_down_model, check_gateup_model, code_rank_distance, model_gemm_tol)

W = synth.Workload(93, "checks", 8, 256, 384, act="outlier", outlier_ratio=0.02)


@pytest.fixture(scope="module")
def case():
    b = synth.make_weights(W, 1)
    x = synth.make_x(W, layer=1)
    wgu_q, wgu_s = O.quant_weights(np.concatenate([b["w_gate"], b["w_up"]], axis=0))
    wd_q, wd_s = O.quant_weights(b["w_down"])
    xq, xs = O.rmsnorm_quant(x, b["norm_w"])
    acc, _ = model_gemm_tol(xq, xs, wgu_q, wgu_s)
    h = (O.silu(acc[:, :W.I]) * acc[:, W.I:]).astype(np.float32)  # a kernel that follows the model
    hq, hs = O.requant(h)
    return dict(xq=xq, xs=xs, wgu_q=wgu_q, wgu_s=wgu_s, wd_q=wd_q, wd_s=wd_s, h=h, hq=hq, hs=hs)


def _run(c, h=None, hq=None, hs=None):
    return check_gateup_model(c["xq"], c["xs"], c["wgu_q"], c["wgu_s"], W.I, c["h"] if h is None else h,
                              c["hq"] if hq is None else hq, c["hs"] if hs is None else hs)


def test_model_following_output_passes(case):
    r = _run(case)
    assert r["h_err_vs_model_of_tol"] <= 0.1  # only the fp32 rounding of h
    assert r["mismatch_frac"] <= 1e-2


def test_h_off_by_1e_minus_4_fails(case):
    h = case["h"].copy()
    i = np.unravel_index(np.argmax(np.abs(h)), h.shape)
    h[i] *= np.float32(1 + 1e-4)
    with pytest.raises(AssertionError, match="MFMA model"):
        _run(case, h=h)


def test_code_one_step_off_fails(case):
    hq = case["hq"].copy()
    # a mid-range code moved to its neighbour (same sign)
    i = np.argwhere(((hq & 0x7F) > 0x20) & ((hq & 0x7F) < 0x70))[0]
    hq[tuple(i)] += 1
    assert code_rank_distance(hq, case["hq"]).max() == 1
    with pytest.raises(AssertionError, match="outside the model"):
        _run(case, hq=hq)


def test_code_far_from_oracle_fails(case):
    """A code that the model window would not flag (the window is bypassed
    here by moving h_tap with it) but that lies two steps from the oracle's at
    a large magnitude fails the oracle adjacency rule."""
    import oracle.ffn as O2
    h = case["h"].copy()
    i = np.unravel_index(np.argmax(np.abs(h)), h.shape)
    g = i[1] // 128
    row = np.abs(h[i[0], g * 128:(g + 1) * 128])
    j = g * 128 + int(np.argsort(row)[-2])  # the group's second largest value
    h[i[0], j] *= np.float32(1.2)
    hq, hs = O2.requant(h)
    with pytest.raises(AssertionError):
        _run(case, h=h, hq=hq, hs=hs)


def test_scale_off_fails(case):
    hs = case["hs"].copy()
    hs[0, 0] *= np.float32(1 + 1e-5)
    with pytest.raises(AssertionError, match="scale"):
        _run(case, hs=hs)


def test_down_model_check(case):
    acc, _ = model_gemm_tol(case["hq"], case["hs"], case["wd_q"], case["wd_s"])
    out = acc.astype(np.float32)
    assert check_down_model(case["hq"], case["hs"], case["wd_q"], case["wd_s"], out) <= 0.5
    out[0, 0] *= np.float32(1 + 1e-4)
    with pytest.raises(AssertionError, match="MFMA model"):
        check_down_model(case["hq"], case["hs"], case["wd_q"], case["wd_s"], out)


def test_rank_distance():
    a = np.array([0x38, 0x38, 0x00, 0x80, 0x01, 0x7E], np.uint8)
    b = np.array([0x39, 0x37, 0x80, 0x01, 0x81, 0xFE], np.uint8)
    assert list(code_rank_distance(a, b)) == [1, 1, 0, 1, 2, 252]
