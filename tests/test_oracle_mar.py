"""Pins of the fp64 oracle for the encoder, decoder input and sampler (CPU only).

Each check ties ``oracle.mar`` to something other than itself: torch's own
float64 LayerNorm / Linear / SiLU for the special cases the denoiser reduces
to, closed-form values of the sinusoidal time embedding, the DDPM posterior
mean in its x0 form against the noise form and against Gaussian conditioning,
exact recovery of x0 from the true noise, permutation equivariance of the
encoder over the known tokens, and the row bookkeeping of the decoder input.
"""
import math

import numpy as np
import pytest
import torch

from oracle import block, mar

RNG = np.random.default_rng(2506)
T64 = lambda a: torch.tensor(np.asarray(a), dtype=torch.float64)


def _head(hs, rng=RNG, std=0.05):
    W, n, C, D, Ft = hs.width, hs.n_blocks, hs.c_tok, hs.d_cond, hs.t_freq
    return {
        "w_t1": rng.normal(0, std, (W, Ft)), "b_t1": rng.normal(0, std, W),
        "w_t2": rng.normal(0, std, (W, W)), "b_t2": rng.normal(0, std, W),
        "w_c": rng.normal(0, std, (W, D)), "b_c": rng.normal(0, std, W),
        "w_in": rng.normal(0, std, (W, C)), "b_in": rng.normal(0, std, W),
        "w_ada": rng.normal(0, std, ((3 * n + 2) * W, W)), "b_ada": rng.normal(0, std, (3 * n + 2) * W),
        "w_1": rng.normal(0, std, (n, W, W)), "b_1": rng.normal(0, std, (n, W)),
        "w_2": rng.normal(0, std, (n, W, W)), "b_2": rng.normal(0, std, (n, W)),
        "w_out": rng.normal(0, std, (C, W)), "b_out": rng.normal(0, std, C),
    }


HS = mar.HeadShape(width=32, n_blocks=3, c_tok=4, d_cond=24, t_freq=16)


def _linear(w, b):
    lin = torch.nn.Linear(w.shape[1], w.shape[0], dtype=torch.float64)
    with torch.no_grad():
        lin.weight.copy_(T64(w))
        lin.bias.copy_(T64(b))
    return lin


def test_silu_matches_torch():
    z = np.linspace(-30, 30, 241)
    np.testing.assert_allclose(mar.silu(z), torch.nn.functional.silu(T64(z)).numpy(), rtol=1e-15, atol=1e-300)
    assert mar.silu(0.0) == 0.0


def test_timestep_embedding_closed_forms():
    # dim 8: frequencies 10000^(-i/4) = 1, 0.1, 0.01, 0.001
    e0 = mar.timestep_embedding(0, 8)
    np.testing.assert_array_equal(e0, [1, 1, 1, 1, 0, 0, 0, 0])
    e = mar.timestep_embedding(100, 8)
    np.testing.assert_allclose(e[[0, 1, 2, 3]], [math.cos(100), math.cos(10), math.cos(1), math.cos(0.1)], rtol=1e-12)
    np.testing.assert_allclose(e[[4, 5, 6, 7]], [math.sin(100), math.sin(10), math.sin(1), math.sin(0.1)], rtol=1e-12)
    # vector of timesteps: one row per timestep
    np.testing.assert_array_equal(mar.timestep_embedding(np.array([0, 100]), 8), np.stack([e0, e]))


def _torch_ln(h, eps):
    return torch.nn.LayerNorm(h.shape[-1], eps=eps, elementwise_affine=False, dtype=torch.float64)(h)


def test_denoiser_zero_modulation_reduces_to_ln_linear():
    head = _head(HS)
    head["w_ada"][:] = 0
    head["b_ada"][:] = 0  # shift = scale = gate = 0: blocks do nothing, final layer is a plain LN
    x = RNG.normal(size=(5, HS.c_tok))
    z = RNG.normal(size=(5, HS.d_cond))
    got = mar.denoiser(x, 7, z, head, HS)
    with torch.no_grad():
        h = _linear(head["w_in"], head["b_in"])(T64(x))
        ref = _linear(head["w_out"], head["b_out"])(_torch_ln(h, HS.eps)).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-14)


def test_denoiser_fixed_modulation_matches_torch_mlp():
    """w_ada = 0 and b_ada = (shift, scale, gate) per block: each block is
    h + gate * MLP(LN(h) * (1 + scale) + shift) with MLP = Linear, SiLU, Linear."""
    head = _head(HS)
    W, n = HS.width, HS.n_blocks
    head["w_ada"][:] = 0
    sh = RNG.normal(0, 0.3, (n + 1, W))
    sc = RNG.normal(0, 0.3, (n + 1, W))
    gt = RNG.normal(1, 0.3, (n, W))
    for k in range(n):
        s0, s1, s2 = mar.modulation_slices(HS, k)
        head["b_ada"][s0], head["b_ada"][s1], head["b_ada"][s2] = sh[k], sc[k], gt[k]
    f0, f1 = mar.modulation_slices(HS, n)
    head["b_ada"][f0], head["b_ada"][f1] = sh[n], sc[n]
    x = RNG.normal(size=(6, HS.c_tok))
    z = RNG.normal(size=(6, HS.d_cond))
    got = mar.denoiser(x, 3, z, head, HS)
    with torch.no_grad():
        h = _linear(head["w_in"], head["b_in"])(T64(x))
        for k in range(n):
            mlp = torch.nn.Sequential(_linear(head["w_1"][k], head["b_1"][k]), torch.nn.SiLU(),
                                      _linear(head["w_2"][k], head["b_2"][k]))
            h = h + T64(gt[k]) * mlp(_torch_ln(h, HS.eps) * (1 + T64(sc[k])) + T64(sh[k]))
        ref = _linear(head["w_out"], head["b_out"])(_torch_ln(h, HS.eps) * (1 + T64(sc[n])) + T64(sh[n])).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-14)


def test_denoiser_time_enters_only_through_condition_and_rows_are_independent():
    head = _head(HS)
    x = RNG.normal(size=(4, HS.c_tok))
    z = RNG.normal(size=(4, HS.d_cond))
    assert not np.allclose(mar.denoiser(x, 1, z, head, HS), mar.denoiser(x, 9, z, head, HS))
    flat = dict(head)
    flat["w_t1"] = np.zeros_like(head["w_t1"])
    np.testing.assert_array_equal(mar.denoiser(x, 1, z, flat, HS), mar.denoiser(x, 9, z, flat, HS))
    whole = mar.denoiser(x, 5, z, head, HS)
    for r in range(4):
        np.testing.assert_allclose(mar.denoiser(x[r:r + 1], 5, z[r:r + 1], head, HS)[0], whole[r], rtol=1e-13)


def test_cosine_schedule_invariants():
    for T in (1, 10, 100):
        sch = mar.cosine_schedule(T)
        assert np.all(sch.betas > 0) and np.all(sch.betas <= 0.999)
        assert np.all(np.diff(sch.alphas_bar) < 0)
        np.testing.assert_allclose(sch.alphas_bar[0], 1 - sch.betas[0], rtol=1e-15)
        assert sch.alphas_bar[-1] <= 1e-3 * (1 + 1e-12)  # the last beta is clipped at 0.999 when T = 1


@pytest.mark.parametrize("i", [0, 1, 17, 98, 99])
def test_posterior_mean_x0_form_equals_noise_form(i):
    """With x_i = sqrt(ab_i) x0 + sqrt(1 - ab_i) eps and the true eps, the step's
    mean (x0 form) equals (x_i - beta_i / sqrt(1 - ab_i) eps) / sqrt(alpha_i)."""
    sch = mar.cosine_schedule(100)
    x0 = RNG.normal(size=(3, 5))
    eps = RNG.normal(size=(3, 5))
    ab, b = sch.alphas_bar[i], sch.betas[i]
    xi = math.sqrt(ab) * x0 + math.sqrt(1 - ab) * eps
    np.testing.assert_allclose(mar.predict_x0(sch, i, xi, eps), x0, rtol=1e-9, atol=1e-9)
    got = mar.ddpm_step(sch, i, xi, eps, tau=0.0, noise=np.zeros_like(xi))
    ref = (xi - b / math.sqrt(1 - ab) * eps) / math.sqrt(1 - b)
    np.testing.assert_allclose(got, ref, rtol=1e-9, atol=1e-9)


@pytest.mark.parametrize("i", [1, 2, 50, 99])
def test_posterior_from_gaussian_conditioning(i):
    """q(x_{i-1} | x_i, x0) from the joint Gaussian of (x_{i-1}, x_i) given x0:
    Var = 1 - ab_{i-1}, Cov = sqrt(alpha_i) (1 - ab_{i-1}), Var(x_i) = 1 - ab_i."""
    sch = mar.cosine_schedule(100)
    abp, ab, a = sch.alphas_bar[i - 1], sch.alphas_bar[i], 1 - sch.betas[i]
    cov, v_prev, v_i = math.sqrt(a) * (1 - abp), 1 - abp, 1 - ab
    c2 = cov / v_i
    c1 = math.sqrt(abp) - c2 * math.sqrt(ab)
    var = v_prev - cov * cov / v_i
    g1, g2, gv = mar.posterior(sch, i)
    np.testing.assert_allclose([g1, g2, gv], [c1, c2, var], rtol=1e-12)


def test_sampler_noise_use_and_single_step():
    head = _head(HS)
    z = RNG.normal(size=(3, HS.d_cond))
    T = 6
    noise = RNG.normal(size=(T + 1, 3, HS.c_tok))
    a = mar.sample(z, noise, T, 0.0, head, HS)
    other = noise.copy()
    other[:T] = RNG.normal(size=(T, 3, HS.c_tok))
    np.testing.assert_array_equal(mar.sample(z, other, T, 0.0, head, HS), a)  # tau = 0: only x_T matters
    assert not np.allclose(mar.sample(z, other, T, 1.0, head, HS), mar.sample(z, noise, T, 1.0, head, HS))
    # one step: alpha_bar_prev = 1, so the step returns the predicted x0 itself
    sch = mar.cosine_schedule(1)
    x1 = noise[1]
    ref = mar.predict_x0(sch, 0, x1, mar.denoiser(x1, 0, z, head, HS))
    np.testing.assert_allclose(mar.sample(z, noise[:2], 1, 1.0, head, HS), ref, rtol=1e-12)


def _block_params(D, F, rng, std=0.05):
    return {
        "ln1_g": 1 + rng.normal(0, std, D), "ln1_b": rng.normal(0, std, D),
        "w_qkv": rng.normal(0, std, (3 * D, D)), "b_qkv": rng.normal(0, std, 3 * D),
        "w_o": rng.normal(0, std, (D, D)), "b_o": rng.normal(0, std, D),
        "ln2_g": 1 + rng.normal(0, std, D), "ln2_b": rng.normal(0, std, D),
        "w_1": rng.normal(0, std, (F, D)), "b_1": rng.normal(0, std, F),
        "w_2": rng.normal(0, std, (D, F)), "b_2": rng.normal(0, std, D),
    }


def test_encoder_is_permutation_equivariant_over_known_tokens():
    D, H, C, n_buf, n_img = 16, 2, 4, 3, 10
    rng = np.random.default_rng(7)
    cls = rng.normal(size=D)
    tok = rng.normal(size=(n_img, C))
    w_z, b_z = rng.normal(0, 0.3, (D, C)), rng.normal(0, 0.1, D)
    pe = rng.normal(size=(n_buf + n_img, D))
    params = [_block_params(D, 4 * D, rng) for _ in range(2)]
    known = [n_buf + p for p in (7, 1, 4, 8)]
    perm = [2, 0, 3, 1]
    e1 = mar.encoder(mar.encoder_input(cls, tok, w_z, b_z, pe, known, n_buf), params, H, 1e-6)
    e2 = mar.encoder(mar.encoder_input(cls, tok, w_z, b_z, pe, [known[j] for j in perm], n_buf),
                     params, H, 1e-6)
    np.testing.assert_allclose(e2[:n_buf], e1[:n_buf], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(e2[n_buf:], e1[n_buf:][perm], rtol=1e-12, atol=1e-12)
    # no known tokens: the buffer rows alone, class embedding plus position
    e0 = mar.encoder_input(cls, tok, w_z, b_z, pe, [], n_buf)
    np.testing.assert_array_equal(e0, cls + pe[:n_buf])


def test_decoder_input_row_bookkeeping():
    D, n_buf, n_img = 8, 2, 9
    rng = np.random.default_rng(11)
    known = [n_buf + p for p in (5, 0, 3)]
    h_enc = rng.normal(size=(n_buf + len(known), D))
    g, b = 1 + rng.normal(0, 0.1, D), rng.normal(0, 0.1, D)
    w_de, b_de = rng.normal(0, 0.3, (D, D)), rng.normal(0, 0.1, D)
    mask = rng.normal(size=D)
    pe = rng.normal(size=(n_buf + n_img, D))
    x = mar.encoder_to_decoder(h_enc, g, b, 1e-6, w_de, b_de, mask, pe, known, n_buf)
    with torch.no_grad():
        ln = torch.nn.LayerNorm(D, eps=1e-6, dtype=torch.float64)
        ln.weight.copy_(T64(g))
        ln.bias.copy_(T64(b))
        v = _linear(w_de, b_de)(ln(T64(h_enc))).numpy()
    targets = list(range(n_buf)) + known
    for r, j in enumerate(targets):
        np.testing.assert_allclose(x[j], v[r] + pe[j], rtol=1e-12, atol=1e-12)
    for j in set(range(n_buf + n_img)) - set(targets):
        np.testing.assert_array_equal(x[j], mask + pe[j])


def test_decoder_cond_matches_torch_layernorm():
    D, n_buf, N = 12, 3, 11
    rng = np.random.default_rng(5)
    x = rng.normal(size=(N, D))
    g, b = 1 + rng.normal(0, 0.1, D), rng.normal(0, 0.1, D)
    pe_diff = rng.normal(size=(N - n_buf, D))
    gen = [9, 4, 3]
    got = mar.decoder_cond(x, g, b, 1e-6, pe_diff, gen, n_buf)
    with torch.no_grad():
        ln = torch.nn.LayerNorm(D, eps=1e-6, dtype=torch.float64)
        ln.weight.copy_(T64(g))
        ln.bias.copy_(T64(b))
        ref = ln(T64(x[gen])).numpy() + pe_diff[[j - n_buf for j in gen]]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("T", [2, 10, 100, 1000])
def test_cosine_schedule_closed_form(T):
    """The cosine schedule is defined by its cumulative product,
    alpha_bar(u) = f(u) / f(0) with f(u) = cos^2((u + s) / (1 + s) * pi / 2) and
    s = 0.008; the betas are the ratios of consecutive values, clipped at 0.999.
    The product of (1 - beta) telescopes back to f((i + 1) / T) / f(0) wherever
    no beta was clipped (every step but the last, where f(1) = 0)."""
    f = lambda u: math.cos((u + 0.008) / 1.008 * math.pi / 2) ** 2
    sch = mar.cosine_schedule(T)
    want = np.array([f((i + 1) / T) / f(0.0) for i in range(T - 1)])
    np.testing.assert_allclose(sch.alphas_bar[:T - 1], want, rtol=1e-12)
    # the offset s matters: without the f(0) normalisation the first value
    # would be f(1/T) itself, off by 1 - f(0) = 1.55e-4
    assert abs(1.0 - f(0.0) - 1.5542e-4) < 1e-7
    assert sch.betas[-1] == 0.999
    # cos^2, not cos: half way through the schedule alpha_bar is near 1/2
    if T % 2 == 0:
        assert abs(sch.alphas_bar[T // 2 - 1] - 0.5) < 0.01
