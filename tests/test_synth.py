"""The seeded input generators: determinism, shapes and activation structure."""

import numpy as np

import synth
from oracle.bf16 import bf16_to_f32


def test_deterministic_and_independent_streams():
    w = synth.WORKLOADS["tiny_m64_h256_i768"]
    a = synth.make_weights(w, layer=1)
    b = synth.make_weights(w, layer=1)
    c = synth.make_weights(w, layer=2)
    for k in a:
        assert np.array_equal(a[k], b[k])
        assert not np.array_equal(a[k], c[k])
    assert a["w_gate"].shape == (768, 256) and a["w_down"].shape == (256, 768) and a["norm_w"].shape == (256,)
    assert np.array_equal(synth.make_x(w, 1, 0), synth.make_x(w, 1, 0))
    assert not np.array_equal(synth.make_x(w, 1, 0), synth.make_x(w, 1, 1))


def test_outlier_channels_and_scales():
    w = synth.WORKLOADS["block32_h4096_i12288"]
    ch = synth.outlier_channels(w, 1, 0, w.outlier_ratio)
    assert len(ch) == 41 and len(set(ch.tolist())) == 41
    x = bf16_to_f32(synth.make_x(w, 1, 0))
    col = np.abs(x).mean(axis=0)
    others = np.setdiff1d(np.arange(4096), ch)
    assert col[ch].mean() > 20 * col[others].mean()
    # row subsets are the same rows
    assert np.array_equal(synth.make_x(w, 1, 0, rows=[3, 7]), synth.make_x(w, 1, 0)[[3, 7]])


def test_step_and_sequence_scales():
    w3 = synth.WORKLOADS["sar512_h4096_i12288"]
    s = synth.step_std(w3, 1, 5)
    assert np.all(s == s[0]) and 0.5 <= s[0] <= 8.0
    w4 = synth.WORKLOADS["batch8x1024_h4096_i12288"]
    s4 = synth.step_std(w4, 1, 0)
    assert len(np.unique(s4)) == 8 and np.all(s4[:1024] == s4[0])
    w4b = synth.WORKLOADS["batch4x1024_h4096_i12288"]
    s4b = synth.step_std(w4b, 1, 0)
    assert w4b.M == 4096 and len(np.unique(s4b)) == 4 and np.all(s4b[:1024] == s4b[0])
    assert len({w.wid for w in synth.WORKLOADS.values()}) == len(synth.WORKLOADS)
    w5 = synth.WORKLOADS["stack31_m512_h4096_i12288"]
    assert abs(synth.step_std(w5, 1, 0)[0] - 0.5) < 1e-6 and abs(synth.step_std(w5, 1, 31)[0] - 8.0) < 1e-5
    assert abs(synth.outlier_ratio(w5, 0) - 0.03) < 1e-12 and abs(synth.outlier_ratio(w5, 31) - 0.005) < 1e-12
