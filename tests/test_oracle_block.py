"""Pins of the fp64 oracle's block, attention and scores (CPU only).

Each check ties the oracle to something other than itself: PyTorch's own
float64 pre-LN TransformerEncoderLayer and MultiheadAttention, closed forms,
invariants of softmax attention, and Appendix A's equivalence of the
cache-aware and standard attention.
"""
import math

import numpy as np
import pytest
import torch

from oracle import block

RNG = np.random.default_rng(1234)


def _params(D, F, std=0.02, rng=RNG):
    return {
        "ln1_g": 1 + rng.normal(0, std, D), "ln1_b": rng.normal(0, std, D),
        "w_qkv": rng.normal(0, std, (3 * D, D)), "b_qkv": rng.normal(0, std, 3 * D),
        "w_o": rng.normal(0, std, (D, D)), "b_o": rng.normal(0, std, D),
        "ln2_g": 1 + rng.normal(0, std, D), "ln2_b": rng.normal(0, std, D),
        "w_1": rng.normal(0, std, (F, D)), "b_1": rng.normal(0, std, F),
        "w_2": rng.normal(0, std, (D, F)), "b_2": rng.normal(0, std, D),
    }


def _torch_layer(p, D, H, F, eps):
    layer = torch.nn.TransformerEncoderLayer(D, H, F, dropout=0.0, activation="gelu",
                                             layer_norm_eps=eps, batch_first=True,
                                             norm_first=True, dtype=torch.float64)
    t = lambda a: torch.tensor(np.asarray(a), dtype=torch.float64)
    with torch.no_grad():
        layer.self_attn.in_proj_weight.copy_(t(p["w_qkv"]))
        layer.self_attn.in_proj_bias.copy_(t(p["b_qkv"]))
        layer.self_attn.out_proj.weight.copy_(t(p["w_o"]))
        layer.self_attn.out_proj.bias.copy_(t(p["b_o"]))
        layer.linear1.weight.copy_(t(p["w_1"]))
        layer.linear1.bias.copy_(t(p["b_1"]))
        layer.linear2.weight.copy_(t(p["w_2"]))
        layer.linear2.bias.copy_(t(p["b_2"]))
        layer.norm1.weight.copy_(t(p["ln1_g"]))
        layer.norm1.bias.copy_(t(p["ln1_b"]))
        layer.norm2.weight.copy_(t(p["ln2_g"]))
        layer.norm2.bias.copy_(t(p["ln2_b"]))
    return layer.eval()


# ---------------------------------------------------------------- LayerNorm / GELU / linear

def test_layer_norm_constant_row_gives_beta():
    D = 17
    g, b = RNG.normal(size=D), RNG.normal(size=D)
    x = np.full((3, D), 2.5)
    np.testing.assert_array_equal(block.layer_norm(x, g, b, 1e-6), np.broadcast_to(b, (3, D)))


def test_layer_norm_moments_closed_form():
    # gamma = 1, beta = 0: each output row has mean 0 and mean square
    # var / (var + eps) with var the population variance of the input row.
    D, eps = 64, 0.25
    x = RNG.normal(3.0, 0.7, size=(5, D))
    y = block.layer_norm(x, np.ones(D), np.zeros(D), eps)
    var = x.var(axis=1)  # numpy's default ddof=0 is the population variance
    np.testing.assert_allclose(y.mean(axis=1), 0, atol=1e-12)
    np.testing.assert_allclose((y ** 2).mean(axis=1), var / (var + eps), rtol=1e-12)


def test_layer_norm_matches_torch():
    D = 48
    x, g, b = RNG.normal(size=(7, D)), RNG.normal(size=D), RNG.normal(size=D)
    ref = torch.nn.functional.layer_norm(torch.tensor(x), (D,), torch.tensor(g), torch.tensor(b), 1e-6)
    np.testing.assert_allclose(block.layer_norm(x, g, b, 1e-6), ref.numpy(), rtol=1e-12, atol=1e-12)


def test_gelu_special_values_and_torch():
    assert block.gelu(np.array([0.0]))[0] == 0.0
    z = np.linspace(-6, 6, 97)
    # Phi(z) + Phi(-z) = 1  =>  gelu(z) - gelu(-z) = z
    np.testing.assert_allclose(block.gelu(z) - block.gelu(-z), z, atol=1e-14)
    ref = torch.nn.functional.gelu(torch.tensor(z), approximate="none").numpy()
    np.testing.assert_allclose(block.gelu(z), ref, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(block.gelu(np.array([40.0])), [40.0])
    scalar = [0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in (-1.3, 0.2, 2.7)]
    np.testing.assert_allclose(block.gelu(np.array([-1.3, 0.2, 2.7])), scalar, rtol=1e-15)


def test_linear_matches_torch_layout():
    w, b, u = RNG.normal(size=(5, 3)), RNG.normal(size=5), RNG.normal(size=(4, 3))
    ref = torch.nn.functional.linear(torch.tensor(u), torch.tensor(w), torch.tensor(b)).numpy()
    np.testing.assert_allclose(block.linear(u, w, b), ref, rtol=1e-14)
    # one row, written out: out[o] = sum_i u[i] w[o][i] + b[o]
    out = [sum(u[0, i] * w[o, i] for i in range(3)) + b[o] for o in range(5)]
    np.testing.assert_allclose(block.linear(u[:1], w, b)[0], out, rtol=1e-14)


# ---------------------------------------------------------------- attention

def test_attention_matches_torch_sdpa():
    q, k, v = RNG.normal(size=(6, 16)), RNG.normal(size=(29, 16)), RNG.normal(size=(29, 16))
    o, p = block.attention(q, k, v)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q)[None], torch.tensor(k)[None], torch.tensor(v)[None])[0].numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-12)


def test_attention_closed_forms():
    d = 8
    # one key: output is that key's value
    v1 = RNG.normal(size=(1, d))
    o, _ = block.attention(RNG.normal(size=(3, d)), RNG.normal(size=(1, d)), v1)
    np.testing.assert_allclose(o, np.repeat(v1, 3, 0), rtol=1e-14)
    # zero query: uniform weights, output is the mean of V
    k, v = RNG.normal(size=(11, d)), RNG.normal(size=(11, d))
    o, p = block.attention(np.zeros((2, d)), k, v)
    np.testing.assert_allclose(p, 1 / 11, rtol=1e-14)
    np.testing.assert_allclose(o, np.repeat(v.mean(0, keepdims=True), 2, 0), rtol=1e-13)
    # adding one vector c to every key shifts row i's logits by q_i.c: P unchanged
    q = RNG.normal(size=(4, d))
    c = RNG.normal(size=d)
    _, p0 = block.attention(q, k, v)
    _, p1 = block.attention(q, k + c, v)
    np.testing.assert_allclose(p1, p0, rtol=1e-12)
    # a dominant key takes (almost) all the mass
    k2 = k.copy()
    k2[5] = 200 * q[0] / np.linalg.norm(q[0])
    o2, p2 = block.attention(q[:1], k2, v)
    assert p2[0, 5] > 1 - 1e-12
    np.testing.assert_allclose(o2[0], v[5], atol=1e-10)


@pytest.mark.parametrize("n_active", [0, 1, 7, 31, 32])
def test_two_segment_equals_single_pass(n_active):
    # Appendix A: splitting keys into A and C with a shared max is exact.
    N, d = 32, 16
    q, k, v = RNG.normal(size=(5, d)), RNG.normal(size=(N, d)), RNG.normal(size=(N, d))
    a = np.sort(RNG.choice(N, n_active, replace=False))
    c = np.setdiff1d(np.arange(N), a)
    o1, _ = block.attention(q, k, v)
    o2 = block.attention_two_segment(q, k[a], v[a], k[c], v[c])
    np.testing.assert_allclose(o2, o1, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- whole block

@pytest.mark.parametrize("D,H,N", [(32, 4, 19), (48, 3, 12)])
def test_full_layer_matches_torch_encoder_layer(D, H, N):
    F, eps = 4 * D, 1e-6
    p = _params(D, F, std=0.3)
    x = RNG.normal(size=(N, D))
    dh = D // H
    res = block.full_layer(p, x, np.zeros((H, N, dh)), np.zeros((H, N, dh)), gen=[1, 4, 5],
                           n_heads=H, eps=eps, score=True)
    layer = _torch_layer(p, D, H, F, eps)
    with torch.no_grad():
        ref = layer(torch.tensor(x)[None])[0].numpy()
        h = layer.norm1(torch.tensor(x)[None])
        attn_out, w = layer.self_attn(h, h, h, need_weights=True, average_attn_weights=False)
        mid = (torch.tensor(x)[None] + attn_out)[0].numpy()
    np.testing.assert_allclose(res.x_out, ref, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(res.x_mid, mid, rtol=1e-11, atol=1e-11)
    w = w[0].numpy()  # [H][N][N]
    np.testing.assert_allclose(res.probs, w, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(res.scores, w[:, [1, 4, 5], :].sum(axis=1), rtol=1e-11, atol=1e-13)
    # the scatter wrote the fresh K/V of every token, head-major inside each third
    kk = (h[0].numpy() @ p["w_qkv"][D:2 * D].T + p["b_qkv"][D:2 * D]).reshape(N, H, dh)
    np.testing.assert_allclose(res.k_cache, kk.transpose(1, 0, 2), rtol=1e-11, atol=1e-13)


def _consistent_cache(p, x, H, eps):
    N, D = x.shape
    full = block.full_layer(p, x, np.zeros((H, N, D // H)), np.zeros((H, N, D // H)), n_heads=H, eps=eps)
    return full


@pytest.mark.parametrize("n_active", [1, 5, 16])
def test_cache_aware_equals_full_on_consistent_cache(n_active):
    # With a cache that holds exactly the K/V full recomputation would produce,
    # the cache-aware layer reproduces the full layer's rows in A (Appendix A).
    D, H, N, eps = 32, 4, 23, 1e-6
    p = _params(D, 4 * D, std=0.2)
    x = RNG.normal(size=(N, D))
    full = _consistent_cache(p, x, H, eps)
    act = RNG.choice(N, n_active, replace=False)
    res = block.cache_aware_layer(p, x, full.k_cache, full.v_cache, act, act[:1], n_heads=H, eps=eps)
    rows = np.sort(act)
    np.testing.assert_allclose(res.x_out[rows], full.x_out[rows], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(res.o, full.o[rows], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(res.k_cache, full.k_cache, rtol=1e-12, atol=1e-14)
    # the two-segment form agrees with the single-pass one inside the layer
    o2 = block.cache_aware_attention_two_segment(res.q, res.k_cache, res.v_cache, act, H)
    np.testing.assert_allclose(o2, res.o, rtol=1e-12, atol=1e-13)


def test_cache_aware_invariants_on_stale_cache():
    D, H, N, eps = 32, 4, 21, 1e-6
    dh = D // H
    p = _params(D, 4 * D, std=0.2)
    x = RNG.normal(size=(N, D))
    kc, vc = RNG.normal(size=(H, N, dh)), RNG.normal(size=(H, N, dh))
    act = [17, 3, 9, 0, 12]
    res = block.cache_aware_layer(p, x, kc, vc, act, [17, 3], n_heads=H, eps=eps, score=True)
    inactive = np.setdiff1d(np.arange(N), act)
    rows = np.sort(act)
    # cache rows outside A keep their bits; rows in A hold the fresh projections
    np.testing.assert_array_equal(res.k_cache[:, inactive], kc[:, inactive])
    np.testing.assert_array_equal(res.v_cache[:, inactive], vc[:, inactive])
    np.testing.assert_array_equal(res.k_cache[:, rows], res.k.reshape(len(rows), H, dh).transpose(1, 0, 2))
    np.testing.assert_array_equal(res.v_cache[:, rows], res.v.reshape(len(rows), H, dh).transpose(1, 0, 2))
    # x rows outside A are untouched
    np.testing.assert_array_equal(res.x_out[inactive], x[inactive])
    # each query's probabilities over the N keys sum to one
    np.testing.assert_allclose(res.probs.sum(axis=2), 1.0, atol=1e-12)
    # scores: total mass of the two generating rows per head is 2
    np.testing.assert_allclose(res.scores.sum(axis=1), 2.0, atol=1e-12)
    # attention of each active row, recomputed from an explicitly concatenated
    # K = [K_A ; K_C] (the concatenate-then-attend baseline of Appendix B)
    for h in range(H):
        sl = slice(h * dh, (h + 1) * dh)
        kcat = np.concatenate([res.k[:, sl], kc[h, inactive]])
        vcat = np.concatenate([res.v[:, sl], vc[h, inactive]])
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.tensor(res.q[:, sl])[None], torch.tensor(kcat)[None], torch.tensor(vcat)[None])[0]
        np.testing.assert_allclose(res.o[:, sl], ref.numpy(), rtol=1e-12, atol=1e-13)


def test_all_active_any_order_is_bitwise_full():
    D, H, N, eps = 32, 4, 13, 1e-6
    dh = D // H
    p = _params(D, 4 * D, std=0.2)
    x = RNG.normal(size=(N, D))
    kc, vc = RNG.normal(size=(H, N, dh)), RNG.normal(size=(H, N, dh))
    full = block.full_layer(p, x, kc, vc, [2, 3], n_heads=H, eps=eps, score=True)
    perm = RNG.permutation(N)
    ca = block.cache_aware_layer(p, x, kc, vc, perm, [3, 2], n_heads=H, eps=eps, score=True)
    for f in ("x_out", "x_mid", "k_cache", "v_cache", "o", "q", "probs", "scores"):
        np.testing.assert_array_equal(getattr(ca, f), getattr(full, f))


def test_active_order_does_not_matter():
    D, H, N, eps = 16, 2, 15, 1e-6
    dh = D // H
    p = _params(D, 4 * D, std=0.2)
    x = RNG.normal(size=(N, D))
    kc, vc = RNG.normal(size=(H, N, dh)), RNG.normal(size=(H, N, dh))
    a = [4, 11, 0, 7]
    r1 = block.cache_aware_layer(p, x, kc, vc, a, [11], n_heads=H, eps=eps, score=True)
    r2 = block.cache_aware_layer(p, x, kc, vc, a[::-1], [11], n_heads=H, eps=eps, score=True)
    for f in ("x_out", "k_cache", "v_cache", "o", "scores"):
        np.testing.assert_array_equal(getattr(r1, f), getattr(r2, f))


def test_rejects_bad_active_sets():
    D, H, N = 16, 2, 6
    p = _params(D, 4 * D)
    x = RNG.normal(size=(N, D))
    kc = np.zeros((H, N, D // H))
    with pytest.raises(ValueError):
        block.cache_aware_layer(p, x, kc, kc, [1, 1], [], n_heads=H)
    with pytest.raises(ValueError):
        block.cache_aware_layer(p, x, kc, kc, [1, 6], [], n_heads=H)
    with pytest.raises(ValueError):
        block.cache_aware_layer(p, x, kc, kc, [1, 2], [3], n_heads=H)
