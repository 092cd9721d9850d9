"""fp64 oracle of one decoder block with cache-aware attention (test infrastructure).

Follows Algorithm 1 and Section 4.1 (cache-aware attention), Appendix A (the
standard attention equation and the two-segment online-softmax form) and
Section 4.2 (per-key attention mass from the generating tokens).  The block
internals the paper leaves open are read as a pre-LN residual block with a
4x GELU MLP, LayerNorm with population variance and eps inside the square
root, exact-erf GELU, a QKV bias, and q|k|v thirds that are head-major inside
each third; the attention scale is 1/sqrt(d_h) per head (Appendix A's
1/sqrt(d) with d the per-head width).

Shapes are per image: x [N][D]; cache k/v [H][N][d_h]; parameters in
``nn.Linear`` layout [out][in].

Pins (tests/test_oracle_block.py): the full layer against PyTorch's own
float64 pre-LN TransformerEncoderLayer and MultiheadAttention weights; the
cache-aware layer against the full layer on a consistent cache (Appendix A's
equivalence); softmax invariants; LayerNorm / GELU special cases.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, Optional, Sequence

import numpy as np
from scipy.special import erf

F64 = np.float64


def layer_norm(x: np.ndarray, gamma: np.ndarray, beta: np.ndarray, eps: float) -> np.ndarray:
    """gamma * (x - mean) / sqrt(var + eps) + beta over the last axis; var is the
    population variance (divide by D)."""
    x = np.asarray(x, F64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return np.asarray(gamma, F64) * (x - mu) / np.sqrt(var + eps) + np.asarray(beta, F64)


def gelu(z: np.ndarray) -> np.ndarray:
    """Exact GELU: z * Phi(z) = z/2 * (1 + erf(z / sqrt(2)))."""
    z = np.asarray(z, F64)
    return 0.5 * z * (1.0 + erf(z / math.sqrt(2.0)))


def linear(u: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """u W^T + b with W in [out][in] layout."""
    return np.asarray(u, F64) @ np.asarray(w, F64).T + np.asarray(b, F64)


def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Row softmax with the row maximum subtracted first (the shared max m_i of
    Appendix A)."""
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray):
    """Standard scaled dot-product attention of Appendix A, single pass over all
    keys: o_i = sum_j softmax_j(q_i . k_j / sqrt(d)) v_j.

    q [n][d], k/v [N][d] -> (o [n][d], P [n][N]).
    """
    q, k, v = (np.asarray(a, F64) for a in (q, k, v))
    s = (q @ k.T) / math.sqrt(q.shape[-1])
    p = softmax_rows(s)
    return p @ v, p


def attention_two_segment(q: np.ndarray, k_a: np.ndarray, v_a: np.ndarray,
                          k_c: np.ndarray, v_c: np.ndarray) -> np.ndarray:
    """Appendix A's cache-aware form: logits of the active segment A and of the
    cached segment C are formed separately, share one maximum m_i, and the
    output is (alpha_A V_A + alpha_C V_C) / l_i with l_i the sum of both
    segments' exponentials.  Either segment may be empty."""
    q = np.asarray(q, F64)
    scale = 1.0 / math.sqrt(q.shape[-1])
    n = q.shape[0]
    s_a = (q @ np.asarray(k_a, F64).T) * scale
    s_c = (q @ np.asarray(k_c, F64).T) * scale
    m_a = s_a.max(axis=-1) if s_a.shape[1] else np.full(n, -np.inf)
    m_c = s_c.max(axis=-1) if s_c.shape[1] else np.full(n, -np.inf)
    m = np.maximum(m_a, m_c)[:, None]
    a_a = np.exp(s_a - m)
    a_c = np.exp(s_c - m)
    l = a_a.sum(axis=-1, keepdims=True) + a_c.sum(axis=-1, keepdims=True)
    return (a_a @ np.asarray(v_a, F64) + a_c @ np.asarray(v_c, F64)) / l


@dataclass
class LayerResult:
    """Everything one block computes for one image.

    ``rows``   sorted active tokens (the canonical order of every row-indexed field);
    ``u``      LN1 of the active rows [n_a][D];
    ``q``, ``k``, ``v``  fresh projections of the active rows [n_a][D] (head-major);
    ``o``      attention output of the active rows [n_a][D], heads concatenated;
    ``x_mid``  residual stream after the attention half [N][D] (rows not active
               keep their input values);
    ``x_out``  residual stream after the MLP half [N][D];
    ``k_cache``, ``v_cache``  cache after the write-back [H][N][d_h];
    ``probs``  per-head attention probabilities of the active rows [H][n_a][N];
    ``scores`` per-head attention mass from the generating rows [H][N], or None.
    """

    rows: np.ndarray
    u: np.ndarray
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    o: np.ndarray
    x_mid: np.ndarray
    x_out: np.ndarray
    k_cache: np.ndarray
    v_cache: np.ndarray
    probs: np.ndarray
    scores: Optional[np.ndarray]


def cache_aware_layer(p: Dict[str, np.ndarray], x: np.ndarray, k_cache: np.ndarray,
                      v_cache: np.ndarray, active: Sequence[int], gen: Sequence[int] = (),
                      n_heads: int = 1, eps: float = 1e-6, score: bool = False) -> LayerResult:
    """One pre-LN block run the cache-aware way (Algorithm 1):

    1. queries, keys and values are computed for the active tokens only;
    2. the fresh keys/values overwrite the cache at the active tokens (the
       cache update of Algorithm 1), every other cache row keeps its bits;
    3. each active query attends over all N tokens: fresh K/V at the active
       tokens, cached K/V elsewhere;
    4. the output projection and the feed-forward network run on the active
       rows only; inactive rows of x are left as they were;
    5. with ``score``, the attention mass that the generating tokens ``gen``
       put on every key is summed per head (Section 4.2): scores[h][j] =
       sum_{i in gen} P_h[i][j].

    The result does not depend on the order of ``active``: rows are processed
    in ascending token order.
    """
    x = np.asarray(x, F64)
    N, D = x.shape
    H = n_heads
    dh = D // H
    rows = np.array(sorted(int(i) for i in active), dtype=np.int64)
    if len(set(rows.tolist())) != len(rows) or (len(rows) and (rows[0] < 0 or rows[-1] >= N)):
        raise ValueError("active tokens must be distinct and in [0, N)")
    gen_set = set(int(i) for i in gen)
    if not gen_set <= set(rows.tolist()):
        raise ValueError("generating tokens must be active")

    kc = np.array(k_cache, dtype=F64, copy=True)
    vc = np.array(v_cache, dtype=F64, copy=True)

    u = layer_norm(x[rows], p["ln1_g"], p["ln1_b"], eps)
    qkv = linear(u, p["w_qkv"], p["b_qkv"])
    q, k, v = qkv[:, :D], qkv[:, D:2 * D], qkv[:, 2 * D:]

    for h in range(H):
        kc[h, rows] = k[:, h * dh:(h + 1) * dh]
        vc[h, rows] = v[:, h * dh:(h + 1) * dh]

    o = np.empty_like(q)
    probs = np.empty((H, len(rows), N))
    for h in range(H):
        o_h, p_h = attention(q[:, h * dh:(h + 1) * dh], kc[h], vc[h])
        o[:, h * dh:(h + 1) * dh] = o_h
        probs[h] = p_h

    x_mid = x.copy()
    x_mid[rows] = x[rows] + linear(o, p["w_o"], p["b_o"])
    u2 = layer_norm(x_mid[rows], p["ln2_g"], p["ln2_b"], eps)
    hid = gelu(linear(u2, p["w_1"], p["b_1"]))
    x_out = x_mid.copy()
    x_out[rows] = x_mid[rows] + linear(hid, p["w_2"], p["b_2"])

    scores = None
    if score:
        g_pos = np.array([i for i, r in enumerate(rows.tolist()) if r in gen_set], dtype=np.int64)
        scores = probs[:, g_pos, :].sum(axis=1)
    return LayerResult(rows, u, q, k, v, o, x_mid, x_out, kc, vc, probs, scores)


def full_layer(p: Dict[str, np.ndarray], x: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray,
               gen: Sequence[int] = (), n_heads: int = 1, eps: float = 1e-6,
               score: bool = False) -> LayerResult:
    """Standard (full-recompute) block: every token is active."""
    N = np.asarray(x).shape[0]
    return cache_aware_layer(p, x, k_cache, v_cache, range(N), gen, n_heads, eps, score)


def cache_aware_attention_two_segment(q: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray,
                                      active: Sequence[int], n_heads: int) -> np.ndarray:
    """Attention of the active rows computed with Appendix A's split into the
    active segment A and the cached segment C = {0..N-1} minus A, per head.
    ``k_cache``/``v_cache`` must already hold the fresh K/V at A.  Returns o
    [n_a][D] with rows in ascending token order."""
    kc = np.asarray(k_cache, F64)
    vc = np.asarray(v_cache, F64)
    H, N, dh = kc.shape
    a = np.array(sorted(int(i) for i in active), dtype=np.int64)
    c = np.setdiff1d(np.arange(N), a)
    q = np.asarray(q, F64)
    o = np.empty((len(a), H * dh))
    for h in range(H):
        sl = slice(h * dh, (h + 1) * dh)
        o[:, sl] = attention_two_segment(q[:, sl], kc[h, a], vc[h, a], kc[h, c], vc[h, c])
    return o
