"""Pins of the attention / FACache oracle against closed forms, a library
routine and the invariants of softmax attention."""

import numpy as np
import torch

import oracle.attention as A
from oracle.bf16 import bf16_to_f32


def _bits(a):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _rand(shape, seed, std=1.0):
    return _bits(np.random.default_rng(seed).standard_normal(shape).astype(np.float32) * std)


def test_equal_keys_average_the_values():
    # every score equal -> uniform weights -> the mean of V
    q = _rand((1, 3, 8), 1)
    k = np.tile(_rand((1, 1, 8), 2), (1, 6, 1))
    v = _rand((1, 6, 8), 3)
    got = A.attention(q, k, v)
    want = bf16_to_f32(v).astype(np.float64).mean(axis=1, keepdims=True)
    assert np.allclose(got, np.broadcast_to(want, got.shape), rtol=0, atol=1e-14)


def test_dominant_key_selects_its_value():
    d = 4
    q = _bits(np.full((1, 2, d), 8.0))
    k = _bits(np.zeros((1, 5, d)))
    k[0, 3] = _bits(np.full(d, 64.0))  # score gap 8 * 64 * 4 / 2 = 1024
    v = _rand((1, 5, d), 4)
    got = A.attention(q, k, v)
    assert np.array_equal(got[0, 0], bf16_to_f32(v[0, 3]).astype(np.float64))


def test_two_keys_are_a_logistic_mix():
    d = 2
    q = _bits(np.array([[[1.0, 0.0]]]))
    k = _bits(np.array([[[3.0, 0.0], [1.0, 0.0]]]))
    v = _bits(np.array([[[1.0, 0.0], [0.0, 1.0]]]))
    got = A.attention(q, k, v)[0, 0]
    delta = (3.0 - 1.0) / np.sqrt(d)
    w = 1.0 / (1.0 + np.exp(-delta))
    assert np.allclose(got, [w, 1.0 - w], rtol=0, atol=1e-15)


def test_against_torch_sdpa_in_fp64():
    q, k, v = _rand((3, 37, 16), 5), _rand((3, 37, 16), 6), _rand((3, 37, 16), 7)
    f = lambda b: torch.from_numpy(bf16_to_f32(b).astype(np.float64))
    ref = torch.nn.functional.scaled_dot_product_attention(f(q), f(k), f(v)).numpy()
    assert np.allclose(A.attention(q, k, v), ref, rtol=0, atol=1e-13)


def test_key_permutation_and_query_permutation():
    q, k, v = _rand((1, 9, 8), 8), _rand((1, 11, 8), 9), _rand((1, 11, 8), 10)
    base = A.attention(q, k, v)
    pk = np.random.default_rng(1).permutation(11)
    assert np.allclose(A.attention(q, k[:, pk], v[:, pk]), base, rtol=0, atol=1e-14)
    pq = np.random.default_rng(2).permutation(9)
    assert np.allclose(A.attention(q[:, pq], k, v), base[:, pq], rtol=0, atol=1e-14)


def test_online_update_equals_attention_for_any_partition_and_order():
    q, k, v = _rand((1, 13, 8), 11, 2.0), _rand((1, 40, 8), 12, 2.0), _rand((1, 40, 8), 13)
    ref = A.attention(q, k, v)[0]
    qf, kf, vf = (bf16_to_f32(x[0]).astype(np.float64) for x in (q, k, v))
    scale = 1.0 / np.sqrt(8)
    for blocks in ([(0, 40)], [(0, 7), (7, 20), (20, 40)], [(33, 40), (0, 1), (1, 33)]):
        st = A.online_state(qf, kf, vf, blocks, scale, A.empty_state(13, 8))
        assert np.allclose(A.finalize(st), ref, rtol=0, atol=1e-13)


def test_first_block_ignores_the_empty_state():
    # alpha = exp(-inf) = 0: the empty state contributes nothing
    q, k, v = _rand((1, 4, 8), 14), _rand((1, 8, 8), 15), _rand((1, 8, 8), 16)
    qf, kf, vf = (bf16_to_f32(x[0]).astype(np.float64) for x in (q, k, v))
    m, l, o = A.online_state(qf, kf, vf, [(0, 8)], 0.25, A.empty_state(4, 8))
    s = qf @ kf.T * 0.25
    assert np.array_equal(m, s.max(axis=1))
    assert np.allclose(l, np.exp(s - m[:, None]).sum(axis=1), rtol=1e-15, atol=0)


def test_block_partition_for_the_current_block():
    u, c = A.facache_blocks(320, 64, 130, 160)
    assert c == [(128, 192)]
    assert u == [(0, 64), (64, 128), (192, 256), (256, 320)]
    u, c = A.facache_blocks(256, 64, 60, 130)  # C straddles three blocks
    assert c == [(0, 64), (64, 128), (128, 192)] and u == [(192, 256)]
    u, c = A.facache_blocks(128, 64, 128, 128)  # empty C
    assert c == [] and u == [(0, 64), (64, 128)]
    u, c = A.facache_blocks(192, 64, 100, 100)  # empty C inside a block overlaps nothing
    assert c == [] and u == [(0, 64), (64, 128), (128, 192)]
    u, c = A.facache_blocks(192, 64, 127, 129)  # two rows straddling a block edge
    assert c == [(64, 128), (128, 192)] and u == [(0, 64)]


def test_facache_schedule_is_plain_attention_across_steps():
    heads, N, d, blk = 2, 256, 16, 64
    c0, c1 = 96, 160
    q, k, v = _rand((heads, N, d), 17, 1.5), _rand((heads, N, d), 18, 1.5), _rand((heads, N, d), 19)
    out1, cache = A.facache_attention(q, k, v, c0, c1, blk)
    assert np.allclose(out1, A.attention(q, k, v), rtol=0, atol=1e-13)
    # next denoising step: only the rows of C change
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    q2[:, c0:c1], k2[:, c0:c1], v2[:, c0:c1] = (_rand((heads, c1 - c0, d), s) for s in (20, 21, 22))
    out2, _ = A.facache_attention(q2, k2, v2, c0, c1, blk, cache)
    assert np.allclose(out2, A.attention(q2, k2, v2), rtol=0, atol=1e-13)
    # the cache is really used: a changed U row goes unseen by the U-blocks' queries
    k3 = k2.copy()
    k3[:, 10] = _rand((heads, d), 23, 4.0)
    out3, _ = A.facache_attention(q2, k3, v2, c0, c1, blk, cache)
    assert np.allclose(out3[:, :64], out2[:, :64], rtol=0, atol=1e-13)
    assert not np.allclose(A.attention(q2, k3, v2)[:, :64], out2[:, :64], rtol=0, atol=1e-6)


def test_lse_closed_form_and_library():
    # equal keys: every score is s, so L = s + log(n)
    q = _rand((1, 3, 8), 30)
    k = np.tile(_rand((1, 1, 8), 31), (1, 5, 1))
    qf, kf = bf16_to_f32(q[0]).astype(np.float64), bf16_to_f32(k[0, 0]).astype(np.float64)
    want = qf @ kf / np.sqrt(8) + np.log(5.0)
    assert np.allclose(A.attention_lse(q, k)[0], want, rtol=0, atol=1e-14)
    # wide-range scores against torch.logsumexp in fp64
    q, k = _rand((2, 19, 16), 32, 6.0), _rand((2, 23, 16), 33, 6.0)
    f = lambda b: torch.from_numpy(bf16_to_f32(b).astype(np.float64))
    ref = torch.logsumexp(f(q) @ f(k).transpose(-1, -2) / 4.0, dim=-1).numpy()
    assert np.allclose(A.attention_lse(q, k), ref, rtol=1e-15, atol=1e-12)


def test_lse_from_the_online_state():
    # m + log(l) after any partition is the log-sum-exp
    q, k, v = _rand((1, 7, 8), 34, 3.0), _rand((1, 30, 8), 35, 3.0), _rand((1, 30, 8), 36)
    qf, kf, vf = (bf16_to_f32(x[0]).astype(np.float64) for x in (q, k, v))
    m, l, _ = A.online_state(qf, kf, vf, [(20, 30), (0, 9), (9, 20)], 1 / np.sqrt(8), A.empty_state(7, 8))
    assert np.allclose(m + np.log(l), A.attention_lse(q, k)[0], rtol=0, atol=1e-13)
