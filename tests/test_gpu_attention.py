"""GPU parity of the first-layer FACache attention (Sec. 3.3, Eqs. 2-6)
against the fp64 oracle, through the C ABI.

Acceptance (derived from the kernel's arithmetic: bf16 inputs, fp32 MFMA
accumulation, P rounded to bf16 for the P V product, bf16 output):
  |o - o_ref| <= 2^-8 max|v| + 2^-8 |o_ref|  element by element,
which covers the two bf16 roundings (2^-9 sum_j p_j |v_j| / l + 2^-9 |o|)
and the fp32 score sums (at most 128 u sum_i |q_i k_i| per score, u = 2^-24,
a relative change of p below 1e-3 for these inputs). Exact properties checked bit for bit: populate and plain modes
agree, resume on unchanged inputs reproduces populate, and resume on inputs
whose rows of C changed reproduces plain attention of the new inputs.
Full-size workloads are checked on sampled heads (heads are independent).
"""

import math

import numpy as np
import pytest
import torch

import oracle.attention as A
import paper_2607_16339_amd as lc
import synth
from oracle.bf16 import bf16_to_f32

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
LOG2E = 1.0 / math.log(2.0)


def _say(msg):
    print(msg, flush=True)


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def _host(t):
    return bf16_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)


class Run:
    """Device buffers of one attention problem and its FACache state."""

    def __init__(self, q, k, v, sentinel=float("nan")):
        self.heads, self.N, self.d = q.shape
        self.q, self.k, self.v = _dev(q), _dev(k), _dev(v)
        self.cm = torch.full((self.heads, self.N), sentinel, dtype=torch.float32, device=DEV)
        self.cl = torch.full((self.heads, self.N), sentinel, dtype=torch.float32, device=DEV)
        self.co = torch.full((self.heads, self.N, self.d), sentinel, dtype=torch.float32, device=DEV)

    def set_inputs(self, q, k, v):
        self.q.copy_(_dev(q)), self.k.copy_(_dev(k)), self.v.copy_(_dev(v))

    def __call__(self, c0, c1, mode, lse=None):
        o = torch.empty_like(self.q)
        lc.lacache_facache_attention(self.q, self.k, self.v, o, lse=lse, cache_m=self.cm, cache_l=self.cl,
                                     cache_o=self.co, c_begin=c0, c_end=c1, mode=mode)
        torch.cuda.synchronize()
        return o


def _check_close(o, ref, v_bits, what):
    got = _host(o)
    vmax = np.abs(bf16_to_f32(v_bits)).reshape(v_bits.shape[0], -1).max(axis=1)[:, None, None]
    bound = 2.0 ** -8 * vmax + 2.0 ** -8 * np.abs(ref)
    err = np.abs(got - ref)
    worst = float((err / bound).max())
    _say("%s: max |err| %.3e, worst err/bound %.3f" % (what, float(err.max()), worst))
    assert np.all(np.isfinite(got)), what
    assert worst <= 1.0, what


def _bits_equal(a, b):
    return torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("c0,c1", [(96, 160), (60, 130), (0, 256), (128, 128), (0, 0), (100, 100), (192, 256),
                                   (0, 64), (127, 129)])
def test_modes_against_oracle_tiny(c0, c1):
    w = synth.ATTN_WORKLOADS["attn_tiny_h2_n256"]
    q, k, v = synth.make_qkv(w, 0)
    ref = A.attention(q, k, v)
    r = Run(q, k, v)
    _say("tiny C=[%d,%d)" % (c0, c1))
    plain = r(c0, c1, 2)
    _check_close(plain, ref, v, "plain")
    pop = r(c0, c1, 0)
    assert _bits_equal(pop, plain)
    res = r(c0, c1, 1)  # inputs unchanged: the cached state reproduces populate exactly
    assert _bits_equal(res, pop)


def test_cache_contents_match_the_oracle_state():
    w = synth.ATTN_WORKLOADS["attn_tiny_h2_n256"]
    q, k, v = synth.make_qkv(w, 0)
    c0, c1 = 96, 160
    r = Run(q, k, v)
    r(c0, c1, 0)
    _, cache = A.facache_attention(q, k, v, c0, c1, 64)
    cm, cl, co = (t.cpu().numpy().astype(np.float64) for t in (r.cm, r.cl, r.co))
    u_blocks, _ = A.facache_blocks(256, 64, c0, c1)
    written = np.zeros(256, dtype=bool)
    for a, b in u_blocks:
        written[a:b] = True
    for h in range(2):
        # rows of query blocks overlapping C are never written
        assert np.all(np.isnan(cm[h, ~written])) and np.all(np.isnan(co[h, ~written]))
        for a, b in u_blocks:
            m, l, ot = cache[h][a]
            # fp32 sums of 128 exact products: |error| <= 128 u sum|q k| (u = 2^-24), under 1e-3 here
            assert np.allclose(cm[h, a:b], m * LOG2E, rtol=1e-5, atol=1e-3)
            assert np.allclose(cl[h, a:b], l, rtol=2e-3, atol=0)
            vmax = np.abs(bf16_to_f32(v[h])).max()
            assert np.all(np.abs(co[h, a:b] - ot) <= 2.0 ** -8 * vmax * l[:, None] + 1e-3 * np.abs(ot))


@pytest.mark.parametrize("name", ["attn_tiny_h2_n256", "attn_sar512_h32"])
def test_denoising_steps_resume_equals_plain(name):
    """Populate at step 0, then resume at steps 1..3 whose inputs differ only
    in the rows of C: each equals the oracle and, bit for bit, the plain
    attention of that step's inputs."""
    w = synth.ATTN_WORKLOADS[name]
    q, k, v = synth.make_qkv(w, 0)
    r = Run(q, k, v)
    _say("%s populate" % name)
    pop = r(w.c_begin, w.c_end, 0)
    _check_close(pop, A.attention(q, k, v), v, "%s step 0" % name)
    for step in (1, 2, 3):
        q, k, v = synth.make_qkv(w, step)
        r.set_inputs(q, k, v)
        _say("%s step %d" % (name, step))
        res = r(w.c_begin, w.c_end, 1)
        _check_close(res, A.attention(q, k, v), v, "%s step %d resume" % (name, step))
        assert _bits_equal(res, r(w.c_begin, w.c_end, 2))


def test_resume_really_uses_the_cache():
    """A changed key row outside C is not seen by the query blocks inside U
    on resume (their state comes from the cache), as in the oracle."""
    w = synth.ATTN_WORKLOADS["attn_tiny_h2_n256"]
    q, k, v = synth.make_qkv(w, 0)
    r = Run(q, k, v)
    before = r(w.c_begin, w.c_end, 0)
    k2 = k.copy()
    k2[:, 10] = synth.to_bf16_bits(np.full((2, 128), 3.0, dtype=np.float32))
    r.set_inputs(q, k2, v)
    res = r(w.c_begin, w.c_end, 1)
    _, cache = A.facache_attention(q, k, v, w.c_begin, w.c_end, 64)
    ref, _ = A.facache_attention(q, k2, v, w.c_begin, w.c_end, 64, cache)
    _check_close(res, ref, v, "stale-U resume")
    assert _bits_equal(res[:, :64], before[:, :64])
    assert not _bits_equal(res[:, :64], r(w.c_begin, w.c_end, 2)[:, :64])


def test_single_block_and_extreme_scores():
    """N = 64 (one block), and a head whose scores span a wide range."""
    g = np.random.default_rng(7)
    q = synth.to_bf16_bits(g.standard_normal((3, 64, 128), dtype=np.float32) * 4.0)
    k = synth.to_bf16_bits(g.standard_normal((3, 64, 128), dtype=np.float32) * 4.0)
    v = synth.to_bf16_bits(g.standard_normal((3, 64, 128), dtype=np.float32))
    r = Run(q, k, v)
    for c0, c1, mode in ((0, 64, 0), (0, 0, 0), (0, 0, 1), (10, 20, 2)):
        _check_close(r(c0, c1, mode), A.attention(q, k, v), v, "N=64 C=[%d,%d) mode %d" % (c0, c1, mode))


def test_batch8x1024_sampled_heads():
    """Full-size batched workload (256 heads x 1024 tokens), launched whole,
    checked on sampled heads against the oracle."""
    w = synth.ATTN_WORKLOADS["attn_batch8x1024_h32"]
    q, k, v = synth.make_qkv(w, 0)
    r = Run(q, k, v)
    _say("batch8x1024 populate")
    pop = r(w.c_begin, w.c_end, 0)
    heads = [0, 37, 128, 255]
    _check_close(pop[heads], A.attention(q[heads], k[heads], v[heads]), v[heads], "batch step 0")
    q, k, v = synth.make_qkv(w, 1)
    r.set_inputs(q, k, v)
    _say("batch8x1024 resume")
    res = r(w.c_begin, w.c_end, 1)
    _check_close(res[heads], A.attention(q[heads], k[heads], v[heads]), v[heads], "batch step 1 resume")
    assert _bits_equal(res, r(w.c_begin, w.c_end, 2))


def test_deterministic_and_stream_ordered():
    w = synth.ATTN_WORKLOADS["attn_sar512_h32"]
    q, k, v = synth.make_qkv(w, 0)
    r = Run(q, k, v)
    a = r(w.c_begin, w.c_end, 2)
    s = torch.cuda.Stream()
    o = torch.empty_like(r.q)
    with torch.cuda.stream(s):
        lc.lacache_facache_attention(r.q, r.k, r.v, o, c_begin=w.c_begin, c_end=w.c_end, mode=2, stream=s)
    s.synchronize()
    assert _bits_equal(a, o)


def _check_lse(lse, q, k, what):
    """|L - L_ref| <= max_j 128 u sum_i |q_i k_ji| / sqrt(d) (the fp32 score sums)
    + 1e-5 (1 + |L_ref|) (exp2, log2 and the sum of l)."""
    got = lse.cpu().numpy().astype(np.float64)
    ref = A.attention_lse(q, k)
    qf, kf = (np.abs(bf16_to_f32(x)).astype(np.float64) for x in (q, k))
    dot_bound = (qf @ np.swapaxes(kf, -1, -2)).max(axis=-1) * 128 * 2.0 ** -24 / math.sqrt(q.shape[-1])
    err = np.abs(got - ref)
    worst = float((err / (dot_bound + 1e-5 * (1 + np.abs(ref)))).max())
    _say("%s: max |err| %.3e, worst err/bound %.3f" % (what, float(err.max()), worst))
    assert worst <= 1.0, what


@pytest.mark.parametrize("name", ["attn_tiny_h2_n256", "attn_sar512_h32"])
def test_lse_in_every_mode(name):
    w = synth.ATTN_WORKLOADS[name]
    q, k, v = synth.make_qkv(w, 0)
    r = Run(q, k, v)
    for mode in (2, 0, 1):
        lse = torch.full((w.heads, w.N), float("nan"), dtype=torch.float32, device=DEV)
        r(w.c_begin, w.c_end, mode, lse=lse)
        _check_lse(lse, q, k, "%s lse mode %d" % (name, mode))
