"""CPU oracle for the per-group FP8 FFN of LaCache (arxiv 2607.16339).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call, link or
execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.

The oracle is a plain, slow, obviously correct restatement of what the paper's
mixed-precision FFN computes (Sec. 3.4, Eqs. 7-8, and the fusion points named at
the end of Sec. 3.4 and in the Fig. 2 caption), written in NumPy with fp64
arithmetic wherever the paper does not fix a precision. It shares no code with
the HIP path. Each function names the passage it follows; the readings taken
where the paper is silent are stated in each function.

Modules
-------
e4m3    OCP e4m3fn codec (closed-form decode, saturating round-to-nearest-even
        encode).
bf16    bfloat16 bit conversions (exact widening, RNE narrowing).
ffn     the FFN steps: weight block quantization, RMSNorm + group quantization,
        gate/up GEMM with per-group dequant, SwiGLU + re-quantization, down
        GEMM, residual add, and the unquantized bf16 context reference.
csweep  ctypes wrapper of ``e4m3_sweep.c``: the same e4m3 encoder in plain C,
        used only to check a device encoder over all 2^32 fp32 bit patterns
        fast enough for a test.
attention  the first-layer attention and the FACache schedule (Sec. 3.3,
        Eqs. 2-6): plain softmax attention, the online-softmax update and
        the populate / resume steps of the cached state.
granularity  the per-token and per-tensor quantization granularities
        compared with the per-group scheme (Sec. 4, Table fp8-granularities).
first_layer  the token-wise first-layer operators with EmbedCache and
        RoPECache (Sec. 3.3): embedding, attention norm, QKV projection, RoPE.
"""

from . import attention, bf16, e4m3, ffn, first_layer, granularity  # noqa: F401
