"""First-layer attention with FACache, written out plainly (test infrastructure only).

FACache (Sec. 3.3, FACache; Eqs. 2-6) keeps FlashAttention's online-softmax
state of the query rows that stay unchanged inside a SAR block, restricted
to the key/value blocks that also stay unchanged, and resumes from it in the
later denoising steps of the block. Its result is the plain attention of the
current Q, K, V: the state is an exact re-association of the softmax sums.

Everything here is fp64 on bf16 inputs (raw uint16 bit patterns):
  attention          softmax(Q K^T * scale) V per head, the definition;
  online_state       the streaming update of Eqs. 2-6 over a list of key
                     blocks, in the paper's order of operations;
  attention_lse      the row-wise log-sum-exp L of the scaled scores;
  finalize           O = diag(l)^-1 O~;
  facache_blocks     which key/value blocks lie inside U and which overlap C;
  facache_attention  the schedule: populate (first step of a block) or
                     resume from the cached state (later steps).
Readings taken where the paper is silent: attention is bidirectional (no
mask: the model is a diffusion LM), scale = 1/sqrt(d), and a block of rows is
"inside U" when none of its rows lies in the current block C.
"""

import numpy as np

from .bf16 import bf16_to_f32


def _f64(bits):
    return bf16_to_f32(np.asarray(bits, dtype=np.uint16)).astype(np.float64)


def attention(q_bits, k_bits, v_bits, scale=None):
    """softmax(Q K^T * scale) V for every head. q, k, v: [heads, N, d] bf16 bits."""
    q, k, v = _f64(q_bits), _f64(k_bits), _f64(v_bits)
    d = q.shape[-1]
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    s = np.matmul(q, np.swapaxes(k, -1, -2)) * scale
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    return np.matmul(p, v)


def attention_lse(q_bits, k_bits, scale=None):
    """L = log sum_j exp(s_ij) of the scaled scores s = Q K^T * scale, per head
    and query row (the log-sum-exp the algorithm of the first layer's
    FlashAttention also writes out, Appendix, Alg. 1)."""
    q, k = _f64(q_bits), _f64(k_bits)
    d = q.shape[-1]
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    s = np.matmul(q, np.swapaxes(k, -1, -2)) * scale
    m = s.max(axis=-1)
    return m + np.log(np.exp(s - m[..., None]).sum(axis=-1))


def empty_state(rows, d):
    """(m, l, O~) before any key block: m = -inf, l = 0, O~ = 0."""
    return np.full(rows, -np.inf), np.zeros(rows), np.zeros((rows, d))


def online_state(q, k, v, blocks, scale, state):
    """Eqs. 2-6 for one head: q [rows, d], k and v [N, d] (fp64); stream the
    key blocks (start, end) in order into the state (m, l, O~)."""
    m, l, o = (np.array(x, dtype=np.float64) for x in state)
    for a, b in blocks:
        s = q @ k[a:b].T * scale                                 # S^(j) = Q K_j^T
        m_new = np.maximum(m, s.max(axis=1))                     # Eq. 2
        alpha = np.exp(m - m_new)                                # Eq. 3 (exp(-inf) = 0 for the first block)
        p = np.exp(s - m_new[:, None])                           # Eq. 4
        l = alpha * l + p.sum(axis=1)                            # Eq. 5
        o = alpha[:, None] * o + p @ v[a:b]                      # Eq. 6
        m = m_new
    return m, l, o


def finalize(state):
    """O = diag(l)^-1 O~."""
    m, l, o = state
    return o / l[:, None]


def facache_blocks(N, block, c_begin, c_end):
    """Key/value blocks of `block` rows: those with no row in [c_begin, c_end)
    (inside U) and those overlapping the current block C. An empty C
    (c_begin == c_end) overlaps no block."""
    u, c = [], []
    for a in range(0, N, block):
        b = min(a + block, N)
        (c if (c_begin < c_end and a < c_end and c_begin < b) else u).append((a, b))
    return u, c


def facache_attention(q_bits, k_bits, v_bits, c_begin, c_end, block, cache=None):
    """The FACache schedule for all heads. With cache None (the first step of
    a SAR block) every query block streams all key blocks, and the query
    blocks inside U record their state after the key blocks inside U. With a
    cache (a later step: only the rows of C changed) the query blocks inside
    U resume from it and stream only the key blocks that overlap C. Returns
    (O [heads, N, d], cache) where cache[h][query block start] = (m, l, O~)."""
    q, k, v = _f64(q_bits), _f64(k_bits), _f64(v_bits)
    heads, N, d = q.shape
    scale = 1.0 / np.sqrt(d)
    u_blocks, c_blocks = facache_blocks(N, block, c_begin, c_end)
    u_starts = {a for a, _ in u_blocks}
    out = np.zeros((heads, N, d))
    new_cache = [dict() for _ in range(heads)]
    for h in range(heads):
        for a in range(0, N, block):
            b = min(a + block, N)
            rows = q[h, a:b]
            if a in u_starts:
                if cache is None:
                    st = online_state(rows, k[h], v[h], u_blocks, scale, empty_state(b - a, d))
                else:
                    st = cache[h][a]
                new_cache[h][a] = st
                st = online_state(rows, k[h], v[h], c_blocks, scale, st)
            else:
                st = online_state(rows, k[h], v[h], u_blocks + c_blocks, scale, empty_state(b - a, d))
            out[h, a:b] = finalize(st)
    return out, new_cache
