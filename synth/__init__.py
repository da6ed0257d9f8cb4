"""Seeded synthetic inputs for the FP8 FFN workloads.

This module only draws random numbers and rounds them to bf16; it holds none
of the FFN's arithmetic, so the oracle and the HIP path can both read its
output without sharing any code of the method itself.

Every draw comes from NumPy's PCG64 seeded with
SeedSequence([260716339, workload_id, layer, step, kind]); normals are drawn in
fp32 and rounded to bf16 (nearest-even) by PyTorch's cast. Arrays are returned
as raw bf16 bit patterns (uint16).

The workloads stand in for the paper's LLaDA-8B activations on its reasoning
and code benchmarks (activations with a few channels of large magnitude, whose
density changes with the denoising step; Sec. 3.2 and Fig. 4); no dataset is
used. Shapes are LLaDA-8B's FFN: hidden H = 4096, intermediate I = 12288.
"""

from dataclasses import dataclass, field

import numpy as np
import torch

SEED_ROOT = 260716339
KIND_X, KIND_NORM_W, KIND_W_GATE, KIND_W_UP, KIND_W_DOWN, KIND_OUTLIER, KIND_STEP = range(7)
OUTLIER_GAIN = 40.0
WEIGHT_STD = 0.02


@dataclass(frozen=True)
class Workload:
    wid: int           # index used in the seed
    name: str
    M: int             # tokens per call (rows of x)
    H: int
    I: int
    group: int = 128
    act: str = "plain"  # plain | outlier | step_scale | seq_scale | stack
    outlier_ratio: float = 0.0
    seqs: int = 1       # sequences flattened into M (seq_scale)
    layers: int = 1     # stacked layers (stack)
    steps: int = 1      # denoising steps (step_scale, stack)
    notes: str = field(default="", compare=False)


WORKLOADS = {
    "tiny_m64_h256_i768": Workload(0, "tiny_m64_h256_i768", 64, 256, 768, notes="1 layer; x ~ N(0,1)"),
    "block32_h4096_i12288": Workload(
        1, "block32_h4096_i12288", 32, 4096, 12288, act="outlier", outlier_ratio=0.01,
        notes="one 32-token decode block; 1% outlier channels x40"),
    "sar512_h4096_i12288": Workload(
        2, "sar512_h4096_i12288", 512, 4096, 12288, act="step_scale", outlier_ratio=0.01, steps=32,
        notes="256 prompt + 256 generated tokens; per-step scale logU(0.5, 8); 1% outliers x40"),
    "batch8x1024_h4096_i12288": Workload(
        3, "batch8x1024_h4096_i12288", 8192, 4096, 12288, act="seq_scale", outlier_ratio=0.01, seqs=8,
        notes="8 sequences x 1024 tokens; per-sequence scale logU(0.5, 8); 1% outliers x40"),
    "batch4x1024_h4096_i12288": Workload(
        5, "batch4x1024_h4096_i12288", 4096, 4096, 12288, act="seq_scale", outlier_ratio=0.01, seqs=4,
        notes="4 sequences x 1024 tokens (the smallest M of the MFMA-bound range); as batch8x1024"),
    "stack31_m512_h4096_i12288": Workload(
        4, "stack31_m512_h4096_i12288", 512, 4096, 12288, act="stack", layers=31, steps=32,
        notes="31 FFN layers with residual adds over 32 denoising steps; std 0.5->8, outliers 3%->0.5%"),
}


def rng_for(w: Workload, layer: int, step: int, kind: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, w.wid, layer, step, kind])))


def to_bf16_bits(a) -> np.ndarray:
    """Round an fp32 array to bf16 (torch's nearest-even cast); returns uint16 bits."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def make_weights(w: Workload, layer: int = 1) -> dict:
    """bf16 FFN weights of one layer: norm_w [H] ~ 1 + N(0, 0.02); W_gate, W_up [I, H]
    and W_down [H, I] ~ N(0, 0.02)."""
    H, I = w.H, w.I

    def normal(kind, shape, std, mean=0.0):
        g = rng_for(w, layer, 0, kind)
        return to_bf16_bits(g.standard_normal(shape, dtype=np.float32) * np.float32(std) + np.float32(mean))

    return {
        "norm_w": normal(KIND_NORM_W, (H,), WEIGHT_STD, 1.0),
        "w_gate": normal(KIND_W_GATE, (I, H), WEIGHT_STD),
        "w_up": normal(KIND_W_UP, (I, H), WEIGHT_STD),
        "w_down": normal(KIND_W_DOWN, (H, I), WEIGHT_STD),
    }


def outlier_channels(w: Workload, layer: int, step: int, ratio: float) -> np.ndarray:
    """round(ratio * H) distinct channel indices, the same for every token."""
    n = int(round(ratio * w.H))
    return np.sort(rng_for(w, layer, step, KIND_OUTLIER).choice(w.H, size=n, replace=False))


def step_std(w: Workload, layer: int, step: int) -> np.ndarray:
    """Per-row standard deviation of x for the workload's activation model."""
    if w.act in ("plain", "outlier"):
        return np.ones(w.M, dtype=np.float32)
    g = rng_for(w, layer, step, KIND_STEP)
    if w.act == "step_scale":  # one log-uniform draw in [0.5, 8] per step
        return np.full(w.M, np.exp(g.uniform(np.log(0.5), np.log(8.0))), dtype=np.float32)
    if w.act == "seq_scale":  # one draw per flattened sequence
        s = np.exp(g.uniform(np.log(0.5), np.log(8.0), size=w.seqs))
        return np.repeat(s, w.M // w.seqs).astype(np.float32)
    if w.act == "stack":  # log-linear 0.5 -> 8 over the steps
        t = step / max(w.steps - 1, 1)
        return np.full(w.M, 0.5 * 16.0 ** t, dtype=np.float32)
    raise ValueError(w.act)


def outlier_ratio(w: Workload, step: int) -> float:
    if w.act == "stack":  # decreasing 3% -> 0.5% as future tokens get unmasked
        return 0.03 - 0.025 * step / max(w.steps - 1, 1)
    return w.outlier_ratio


def make_x(w: Workload, layer: int = 1, step: int = 0, rows=None) -> np.ndarray:
    """bf16 activations [M, H] (or the given row subset) for (layer, step)."""
    g = rng_for(w, layer, step, KIND_X)
    x = g.standard_normal((w.M, w.H), dtype=np.float32)
    x *= step_std(w, layer, step)[:, None]
    ratio = outlier_ratio(w, step)
    if ratio > 0:
        x[:, outlier_channels(w, layer, step, ratio)] *= np.float32(OUTLIER_GAIN)
    if rows is not None:
        x = x[rows]
    return to_bf16_bits(x)


# ---------------------------------------------------------------------------
# First-layer attention inputs (FACache)
# ---------------------------------------------------------------------------

KIND_Q, KIND_K, KIND_V, KIND_SINK = range(10, 14)
SINK_GAIN = 4.0


@dataclass(frozen=True)
class AttnWorkload:
    wid: int
    name: str
    heads: int          # attention problems (sequences x heads)
    N: int              # tokens per sequence: prompt + generated
    c_begin: int        # current SAR block C = [c_begin, c_end)
    c_end: int
    d: int = 128
    qk_std: float = 1.5
    sinks: int = 2      # key rows per head with SINK_GAIN x the norm
    notes: str = field(default="", compare=False)


ATTN_WORKLOADS = {
    "attn_tiny_h2_n256": AttnWorkload(
        100, "attn_tiny_h2_n256", 2, 256, 96, 160, notes="C straddles two key blocks"),
    "attn_sar512_h32": AttnWorkload(
        101, "attn_sar512_h32", 32, 512, 288, 320,
        notes="LLaDA-8B layer 1: 32 heads x 128; 256 prompt + 256 generated tokens, block 32, second block"),
    "attn_batch8x1024_h32": AttnWorkload(
        102, "attn_batch8x1024_h32", 256, 1024, 544, 576,
        notes="8 sequences x 32 heads; 512 prompt + 512 generated tokens, block 32, second block"),
}


def attn_rng(w: AttnWorkload, step: int, kind: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, w.wid, 0, step, kind])))


def make_qkv(w: AttnWorkload, step: int = 0, heads=None):
    """bf16 (q, k, v) [heads, N, d] of denoising step `step` of the SAR block.

    q, k ~ N(0, qk_std^2) and v ~ N(0, 1) per element; `sinks` key rows per
    head (drawn once) are scaled by SINK_GAIN, giving a few dominant keys.
    Step 0 draws every row; a later step redraws only the rows of C, so the
    rows outside C stay those of step 0 (the premise of FACache). `heads`
    selects a subset of the heads (the draw is the same)."""
    shape = (w.heads, w.N, w.d)
    out = []
    for kind, std in ((KIND_Q, w.qk_std), (KIND_K, w.qk_std), (KIND_V, 1.0)):
        a = attn_rng(w, 0, kind).standard_normal(shape, dtype=np.float32) * np.float32(std)
        if kind == KIND_K and w.sinks:
            rows = attn_rng(w, 0, KIND_SINK).integers(0, w.N, size=(w.heads, w.sinks))
            for h in range(w.heads):
                a[h, rows[h]] *= np.float32(SINK_GAIN)
        if step > 0:
            g = attn_rng(w, step, kind)
            a[:, w.c_begin:w.c_end] = g.standard_normal((w.heads, w.c_end - w.c_begin, w.d),
                                                        dtype=np.float32) * np.float32(std)
        if heads is not None:
            a = a[heads]
        out.append(to_bf16_bits(a))
    return tuple(out)
