"""The allocation-free FFN entry point (lacache_ffn_fp8_noalloc) through the C
ABI, against the library-workspace entry point (lacache_ffn_fp8): the same
kernels run, so the output bytes must be identical. Two calls in a row, the
second with a smaller input (the array keeps the first call's contents); a
shape beyond the array is refused before anything runs; and the call works
inside a HIP graph capture where the library workspace could not grow."""

import numpy as np
import pytest
import torch

import paper_2607_16339_amd as lc
import synth
from gpu_util import DEV, Layer, dev_bf16

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS["sar512_h4096_i12288"]


def _say(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module")
def layer():
    return Layer(W, layer=1)


def _args(lay):
    return (lay.norm_w, lay.wgu_q, lay.wgu_s, lay.wd_q, lay.wd_s)


def test_noalloc_equals_workspace_call_twice(layer):
    prev = lc.lacache_set_path_policy(0)
    try:
        for M in (512, 32):  # tiled with split-K partials, then the skinny path
            _say("noalloc M=%d" % M)
            x = dev_bf16(synth.make_x(W, layer=1, step=2)[:M])
            ref = lc.ffn_fp8(x, *_args(layer))
            out = torch.full((M, W.H), 7.0, dtype=torch.bfloat16, device=DEV)
            lc.lacache_ffn_fp8_noalloc(x, *_args(layer), out)
            torch.cuda.synchronize()
            assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), M
    finally:
        lc.lacache_set_path_policy(prev)


def test_noalloc_refuses_shapes_beyond_the_array(layer):
    M = 8192  # its workspace (xq, xs, hq, hs: 129 MiB) exceeds the 64 MiB array
    assert lc.lacache_ffn_workspace_bytes(M, W.H, W.I) > 64 << 20
    x = torch.zeros((M, W.H), dtype=torch.bfloat16, device=DEV)
    out = torch.full((M, W.H), 7.0, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(lc.LacacheError) as ei:
        lc.lacache_ffn_fp8_noalloc(x, *_args(layer), out)
    assert ei.value.status == lc.LACACHE_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert bool((out.float() == 7.0).all())


def test_noalloc_under_graph_capture(layer):
    """With the library workspace released, lacache_ffn_fp8 cannot run under
    capture (it would have to allocate), while the allocation-free call
    captures; its replays equal the eager result, with eager work between
    them."""
    M = 200  # tiled, down GEMM split 6 ways
    x = dev_bf16(synth.make_x(W, layer=1, step=3)[:M])
    ref = lc.ffn_fp8(x, *_args(layer))
    torch.cuda.synchronize()
    lc.lacache_release_workspace()
    out = torch.empty((M, W.H), dtype=torch.bfloat16, device=DEV)
    status = []
    g0 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g0):
        try:
            lc.lacache_ffn_fp8(x, *_args(layer), out)
        except lc.LacacheError as e:
            status.append(e.status)
    assert status == [lc.LACACHE_ERR_CAPTURE]
    del g0
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lc.lacache_ffn_fp8_noalloc(x, *_args(layer), out)
    y = dev_bf16(synth.make_x(W, layer=2, step=3)[:64])
    for i in range(3):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), i
        # eager work in between, on the same array
        o2 = torch.empty((64, W.H), dtype=torch.bfloat16, device=DEV)
        lc.lacache_ffn_fp8_noalloc(y, *_args(layer), o2)
        torch.cuda.synchronize()
    del g
