"""Parity of the rest of a MAR step on the GPU against the fp64 oracle
(``oracle.mar``): the encoder input rows (Eq. 1), the decoder input built from
the encoder output (Eq. 2) and the sampler of Eq. 3, element by element on the
same seeded inputs, through the C ABI."""
import numpy as np
import pytest

from oracle import mar
from paper_2506_12035_amd import workload

from gpu_util import TOL, rel_err, say

pytestmark = pytest.mark.gpu


def _dev(a, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to("cuda").contiguous()


def _known_and_rank(rng, B, n_img, n_known):
    """Per image a random generation order; rank[b][p] its position; the known
    tokens (rank < n_known) in ascending order."""
    rank = np.empty((B, n_img), np.int32)
    known = np.empty((B, n_known), np.int32)
    for b in range(B):
        order = rng.permutation(n_img)
        rank[b, order] = np.arange(n_img)
        known[b] = np.sort(order[:n_known])
    return known, rank


@pytest.mark.parametrize("D", [256, 768])
@pytest.mark.parametrize("n_known", [0, 13, 40])
def test_encoder_input(D, n_known):
    import torch
    from paper_2506_12035_amd import binding

    B, n_buf, n_img, C = 3, 5, 40, 16
    rng = np.random.default_rng(100 + n_known)
    say(f"encoder input D={D} n_known={n_known}")
    cls = rng.standard_normal((B, D)).astype(np.float32)
    tok = rng.standard_normal((B, n_img, C)).astype(np.float32)
    w_z = (0.25 * rng.standard_normal((D, C))).astype(np.float32)
    b_z = (0.1 * rng.standard_normal(D)).astype(np.float32)
    pe = rng.standard_normal((n_buf + n_img, D)).astype(np.float32)
    known, _ = _known_and_rank(rng, B, n_img, n_known)
    n_enc = n_buf + n_known
    x = torch.full((B, n_enc, D), float("nan"), device="cuda")
    binding.encoder_input(x, _dev(cls), _dev(tok), _dev(w_z), _dev(b_z), _dev(pe),
                          _dev(known) if n_known else None, B, n_buf, n_img, n_known, D, C)
    torch.cuda.synchronize()
    got = x.cpu().numpy()
    for b in range(B):
        ref = mar.encoder_input(cls[b], tok[b], w_z, b_z, pe, [n_buf + int(p) for p in known[b]], n_buf)
        e = rel_err(got[b], ref)
        assert e <= 1e-6, (b, e)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(3, 4, 32, 0, 256), (3, 4, 32, 9, 256), (3, 4, 32, 32, 256),
                                   (8, 8, 200, 150, 512)],
                         ids=lambda s: "B{}-buf{}-img{}-known{}-D{}".format(*s))
def test_encoder_to_decoder(dtype, shape):
    import torch
    from paper_2506_12035_amd import binding

    B, n_buf, n_img, n_known, D = shape
    say(f"encoder to decoder {dtype} {shape}")
    rng = np.random.default_rng(200 + n_known + D)
    n_enc, N = n_buf + n_known, n_buf + n_img
    x_enc = rng.standard_normal((B, n_enc, D)).astype(np.float32)
    g = (1 + 0.1 * rng.standard_normal(D)).astype(np.float32)
    bb = (0.1 * rng.standard_normal(D)).astype(np.float32)
    w_de = workload.round_to((0.05 * rng.standard_normal((D, D))).astype(np.float32), dtype)
    b_de = (0.1 * rng.standard_normal(D)).astype(np.float32)
    mask = rng.standard_normal(D).astype(np.float32)
    pe = rng.standard_normal((N, D)).astype(np.float32)
    known, rank = _known_and_rank(rng, B, n_img, n_known)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    dt = binding.MARCHE_BF16 if dtype == "bf16" else binding.MARCHE_F32
    x_dec = torch.full((B, N, D), float("nan"), device="cuda")
    wsb = binding.encoder_to_decoder_workspace_bytes(B, n_buf, n_known, D, dt)
    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device="cuda")
    binding.encoder_to_decoder(x_dec, _dev(x_enc), _dev(g), _dev(bb), 1e-6, _dev(w_de, td), _dev(b_de),
                               _dev(mask), _dev(pe), _dev(known) if n_known else None, _dev(rank),
                               B, n_buf, n_img, n_known, D, dt, ws, wsb)
    torch.cuda.synchronize()
    got = x_dec.cpu().numpy()
    assert np.isfinite(got).all()  # every row written
    worst = 0.0
    for b in range(B):
        ref = mar.encoder_to_decoder(x_enc[b], g, bb, 1e-6, w_de, b_de, mask, pe,
                                     [n_buf + int(p) for p in known[b]], n_buf)
        worst = max(worst, rel_err(got[b], ref))
        masked = [n_buf + p for p in range(n_img) if rank[b, p] >= n_known]
        np.testing.assert_allclose(got[b, masked], ref[masked], rtol=1e-6, atol=1e-6)
    say(f"  max rel err {worst:.2e}")
    assert worst <= TOL[dtype]


def _head_case(dtype, n_rows, T, seed):
    mc = workload.MAR_CONFIGS["tiny"]
    mc = workload.MarConfig(mc.name, mc.dec.with_(dtype=dtype), mc.enc_layers, mc.head_width,
                            mc.head_blocks, sample_steps=T, head_std=mc.head_std)
    cfg = mc.dec
    hs = mar.HeadShape(mc.head_width, mc.head_blocks, mc.c_tok, cfg.d_model, mc.t_freq, mc.head_eps)
    head = workload.head_weights(mc)
    emb = workload.mar_embeddings(mc)
    rng = np.random.default_rng(seed)
    N, D = cfg.n_tokens, cfg.d_model
    B = n_rows // cfg.n_img + 2
    x_dec = rng.standard_normal((B, N, D)).astype(np.float32)
    cells = rng.choice(B * cfg.n_img, size=n_rows, replace=False)
    b_of, p_of = cells // cfg.n_img, cells % cfg.n_img
    rows = (b_of * N + cfg.n_buf + p_of).astype(np.int32)
    out_rows = (b_of * cfg.n_img + p_of).astype(np.int32)
    noise = workload.head_noise(mc, seed, n_rows)
    return mc, hs, head, emb, x_dec, rows, out_rows, noise, b_of, p_of


def _run_head(mc, head, emb, x_dec, rows, out_rows, noise, tau):
    import torch
    from paper_2506_12035_amd import binding

    cfg = mc.dec
    td = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    dt = binding.MARCHE_BF16 if cfg.dtype == "bf16" else binding.MARCHE_F32
    hdev = {k: _dev(v, td if k in ("w_t1", "w_t2", "w_c", "w_ada", "w_1", "w_2") else None)
            for k, v in head.items()}
    hd = binding.make_head(mc.head_width, mc.head_blocks, mc.c_tok, cfg.d_model, mc.t_freq, dt,
                           mc.head_eps)
    hw = binding.make_head_weights(hdev)
    B = x_dec.shape[0]
    tok_out = torch.full((B * cfg.n_img, mc.c_tok), float("nan"), device="cuda")
    n_rows = len(rows)
    wsb = binding.diffusion_workspace_bytes(hd, n_rows, mc.sample_steps)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    binding.diffusion_sample(hd, hw, _dev(x_dec), cfg.n_tokens, cfg.n_buf, _dev(emb["dec_ln_g"]),
                             _dev(emb["dec_ln_b"]), cfg.ln_eps, _dev(emb["pe_diff"]), _dev(rows),
                             _dev(out_rows), n_rows, _dev(noise), mc.sample_steps, tau, tok_out, ws,
                             wsb)
    torch.cuda.synchronize()
    return tok_out.cpu().numpy()


def _oracle_head(mc, hs, head, emb, x_dec, b_of, p_of, noise, tau):
    cfg = mc.dec
    z = np.concatenate([mar.decoder_cond(x_dec[b], emb["dec_ln_g"], emb["dec_ln_b"], cfg.ln_eps,
                                         emb["pe_diff"], [cfg.n_buf + p], cfg.n_buf)
                        for b, p in zip(b_of, p_of)])
    h64 = {k: np.asarray(v, np.float64) for k, v in head.items()}
    return mar.sample(z, noise, mc.sample_steps, tau, h64, hs)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n_rows,T", [(37, 1), (37, 8), (300, 8)])
def test_diffusion_sample(dtype, n_rows, T):
    say(f"diffusion sample {dtype} rows={n_rows} T={T}")
    mc, hs, head, emb, x_dec, rows, out_rows, noise, b_of, p_of = _head_case(dtype, n_rows, T, 7 + n_rows)
    tau = 1.0
    got = _run_head(mc, head, emb, x_dec, rows, out_rows, noise, tau)
    ref = _oracle_head(mc, hs, head, emb, x_dec, b_of, p_of, noise, tau)
    sel = got[out_rows]
    e = rel_err(sel, ref)
    say(f"  max rel err {e:.2e}")
    assert e <= TOL[dtype]
    others = np.setdiff1d(np.arange(got.shape[0]), out_rows)
    assert np.isnan(got[others]).all()  # rows not sampled are untouched


def test_diffusion_sample_temperature_zero_ignores_step_noise():
    mc, hs, head, emb, x_dec, rows, out_rows, noise, b_of, p_of = _head_case("bf16", 40, 6, 3)
    a = _run_head(mc, head, emb, x_dec, rows, out_rows, noise, 0.0)[out_rows]
    other = noise.copy()
    other[:mc.sample_steps] = np.random.default_rng(9).standard_normal(other[:mc.sample_steps].shape)
    b = _run_head(mc, head, emb, x_dec, rows, out_rows, other.astype(np.float32), 0.0)[out_rows]
    np.testing.assert_array_equal(a, b)


def _oracle_whole_step(eng, t, tok_before, noise):
    """One whole step of every image by the oracle, from the GPU's token values
    before the step: encoder input, encoder, decoder input, the decoder (all
    layers full), condition and sampler.  Returns (x_out [B][N][D], new token
    values [B][g][C])."""
    from oracle import block

    mc = eng.mc
    c, ec = mc.dec, mc.enc
    emb = workload.mar_embeddings(mc, eng.B)
    enc_p = [workload.layer_weights(ec, l) for l in range(ec.n_layers)]
    dec_p = [workload.layer_weights(c, l) for l in range(c.n_layers)]
    head = {k: np.asarray(v, np.float64) for k, v in workload.head_weights(mc).items()}
    hs = mar.HeadShape(mc.head_width, mc.head_blocks, mc.c_tok, c.d_model, mc.t_freq, mc.head_eps)
    n_known = eng.dec.plans[t].n_known
    gens = eng._gen_tokens(t)
    g = len(gens[0])
    xs, toks = [], []
    for b in range(eng.B):
        known = [c.n_buf + int(p) for p in np.sort(eng.dec.orders[b, :n_known])]
        e = mar.encoder_input(emb["cls"][b], tok_before[b], emb["w_z"], emb["b_z"], emb["pe_enc"],
                              known, c.n_buf)
        h = mar.encoder(e, enc_p, ec.n_heads, ec.ln_eps)
        x = mar.encoder_to_decoder(h, emb["enc_ln_g"], emb["enc_ln_b"], c.ln_eps, emb["w_de"],
                                   emb["b_de"], emb["mask"], emb["pe_dec"], known, c.n_buf)
        kc = np.zeros((c.n_heads, c.n_tokens, c.head_dim))
        for p in dec_p:
            x = block.full_layer(p, x, kc, kc.copy(), n_heads=c.n_heads, eps=c.ln_eps).x_out
        gen = [int(j) for j in gens[b]]
        z = mar.decoder_cond(x, emb["dec_ln_g"], emb["dec_ln_b"], c.ln_eps, emb["pe_diff"], gen, c.n_buf)
        toks.append(mar.sample(z, noise[:, b * g:(b + 1) * g], mc.sample_steps, mc.temperature, head, hs))
        xs.append(x)
    return np.stack(xs), np.stack(toks)


def test_whole_mar_steps_against_oracle():
    """Four whole steps (every decoder step full) of the tiny model: the decoder
    output and the sampled token values of each step against the oracle given
    the same token values before the step."""
    import torch
    from paper_2506_12035_amd import driver

    mc = workload.MAR_CONFIGS["tiny"]
    eng = driver.MarEngine(mc, steps=[0, 1, 2, 3], full_every=1)
    eng.tok.zero_()
    c = mc.dec
    for t in eng.steps:
        say(f"whole MAR step {t}")
        tok_before = eng.tok.cpu().numpy().copy()
        eng.step(t)
        torch.cuda.synchronize()
        x_gpu = eng.dec.x.cpu().numpy()
        tok_gpu = eng.tok.cpu().numpy()
        x_ref, tok_ref = _oracle_whole_step(eng, t, tok_before, eng.noise[t].cpu().numpy())
        ex = rel_err(x_gpu, x_ref)
        gens = eng._gen_tokens(t)
        got = np.stack([tok_gpu[b, gens[b] - c.n_buf] for b in range(eng.B)])
        et = rel_err(got, tok_ref)
        say(f"  decoder output {ex:.2e}, sampled tokens {et:.2e}")
        assert ex <= TOL["bf16"] and et <= TOL["bf16"]
        # tokens not generated at this step keep their values
        keep = np.ones(tok_gpu.shape[:2], bool)
        for b in range(eng.B):
            keep[b, gens[b] - c.n_buf] = False
        np.testing.assert_array_equal(tok_gpu[keep], tok_before[keep])


def test_whole_generation_default_schedule():
    """Every step of the tiny model under the paper's schedule (periodic full
    refresh, 10% refresh tokens): every image token is sampled exactly once and
    all values are finite."""
    import torch
    from paper_2506_12035_amd import driver

    mc = workload.MAR_CONFIGS["tiny"]
    eng = driver.MarEngine(mc)
    eng.generate()
    torch.cuda.synchronize()
    tok = eng.tok.cpu().numpy()
    assert np.isfinite(tok).all()
    assert (np.abs(tok).sum(axis=2) > 0).all()


def test_whole_generation_image_ranges_match_one_call():
    """Encoder and decoder as two image ranges on two streams (2 + 1 images of
    the tiny model's 3): every image is computed exactly as in one call, so
    the whole generation's token values match bit for bit."""
    import torch
    from paper_2506_12035_amd import driver

    mc = workload.MAR_CONFIGS["tiny"]
    ref = driver.MarEngine(mc)
    ref.generate()
    eng = driver.MarEngine(mc, micro_batches=2)
    assert [n for _, n in eng.dec.ranges] == [2, 1]
    eng.generate()
    torch.cuda.synchronize()
    assert torch.equal(eng.tok, ref.tok)
    assert torch.equal(eng.dec.x, ref.dec.x)


def test_sampler_full_size_sampled_rows():
    """The sampler at the MAR-L head (width 1280, 8 blocks, 100 DDPM steps) on
    512 rows (batch 128 x 4 generating tokens), as the whole-generation bench
    runs it; rows are independent, so the oracle recomputes sampled rows."""
    mc = workload.MAR_CONFIGS["mar-l-e2e"]
    cfg = mc.dec
    hs = mar.HeadShape(mc.head_width, mc.head_blocks, mc.c_tok, cfg.d_model, mc.t_freq, mc.head_eps)
    head = workload.head_weights(mc)
    emb = workload.mar_embeddings(mc)
    rng = np.random.default_rng(77)
    B, N, n_rows = cfg.batch, cfg.n_tokens, 512
    say(f"sampler full size: {n_rows} rows, {mc.sample_steps} steps")
    x_dec = rng.standard_normal((B, N, cfg.d_model)).astype(np.float32)
    cells = rng.choice(B * cfg.n_img, size=n_rows, replace=False)
    b_of, p_of = cells // cfg.n_img, cells % cfg.n_img
    rows = (b_of * N + cfg.n_buf + p_of).astype(np.int32)
    out_rows = (b_of * cfg.n_img + p_of).astype(np.int32)
    noise = workload.head_noise(mc, 5, n_rows)
    got = _run_head(mc, head, emb, x_dec, rows, out_rows, noise, mc.temperature)[out_rows]
    assert np.isfinite(got).all()
    pick = [0, 211, 511]
    ref = _oracle_head(mc, hs, head, emb, x_dec, b_of[pick], p_of[pick], noise[:, pick], mc.temperature)
    e = rel_err(got[pick], ref)
    say(f"  sampled rows max rel err {e:.2e}")
    assert e <= TOL["bf16"]


def test_encoder_to_decoder_full_size_sampled_images():
    """The decoder input at MAR-L size (batch 128, 64 buffer + 256 image tokens,
    half of them known), every row written, two sampled images against the
    oracle."""
    import torch
    from paper_2506_12035_amd import binding

    B, n_buf, n_img, n_known, D = 128, 64, 256, 128, 1024
    say("decoder input full size")
    rng = np.random.default_rng(314)
    N = n_buf + n_img
    x_enc = rng.standard_normal((B, n_buf + n_known, D)).astype(np.float32)
    g = (1 + 0.02 * rng.standard_normal(D)).astype(np.float32)
    bb = (0.02 * rng.standard_normal(D)).astype(np.float32)
    w_de = workload.round_to((0.02 * rng.standard_normal((D, D))).astype(np.float32), "bf16")
    b_de = (0.02 * rng.standard_normal(D)).astype(np.float32)
    mask = rng.standard_normal(D).astype(np.float32)
    pe = rng.standard_normal((N, D)).astype(np.float32)
    known, rank = _known_and_rank(rng, B, n_img, n_known)
    x_dec = torch.full((B, N, D), float("nan"), device="cuda")
    wsb = binding.encoder_to_decoder_workspace_bytes(B, n_buf, n_known, D, binding.MARCHE_BF16)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    binding.encoder_to_decoder(x_dec, _dev(x_enc), _dev(g), _dev(bb), 1e-6, _dev(w_de, torch.bfloat16),
                               _dev(b_de), _dev(mask), _dev(pe), _dev(known), _dev(rank), B, n_buf,
                               n_img, n_known, D, binding.MARCHE_BF16, ws, wsb)
    torch.cuda.synchronize()
    assert torch.isfinite(x_dec).all().item()
    got = x_dec[[5, 127]].cpu().numpy()
    for i, b in enumerate((5, 127)):
        ref = mar.encoder_to_decoder(x_enc[b], g, bb, 1e-6, w_de, b_de, mask, pe,
                                     [n_buf + int(p) for p in known[b]], n_buf)
        e = rel_err(got[i], ref)
        say(f"  image {b}: max rel err {e:.2e}")
        assert e <= TOL["bf16"]
