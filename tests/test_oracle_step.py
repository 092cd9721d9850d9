"""Pins of the oracle's decoding step over a stack (CPU only).

* at a 100% refresh ratio the MARche schedule equals full recomputation bit
  for bit at every step (the active set is then every token, and the
  cache-aware layer canonicalises its rows);
* at 0% the active set is exactly G u N (the "no refreshing tokens" setting of
  Section 5.3);
* a full step is the plain stack of full layers, and the selection layer's
  scores come from the generating rows only.
"""
import numpy as np
import pytest

from oracle import block, schedule, select, step
from paper_2506_12035_amd import workload

TINY = workload.Config(90, "tiny", n_layers=3, d_model=32, n_heads=4, head_dim=8, d_mlp=128,
                       n_tokens=20, n_buf=4, batch=2, dtype="f32", n_steps=6,
                       ratio_bp=1000, sel_layer=2, full_every=3, weight_std=0.2)


def _inputs(cfg):
    p = [{k: v.astype(np.float64) for k, v in w.items()} for w in workload.all_weights(cfg)]
    e = workload.embeddings(cfg)
    o = workload.orders(cfg)
    return p, e, o


def _run(cfg, b, **kw):
    p, e, o = _inputs(cfg)
    args = dict(n_buf=cfg.n_buf, n_steps=cfg.n_steps, n_heads=cfg.n_heads, eps=cfg.ln_eps,
                sel_layer=cfg.sel_layer, full_every=cfg.full_every)
    args.update(kw)
    return step.run_generation(p, e.cls[b], e.value[b], e.mask, e.pos, o[b], **args)


@pytest.mark.parametrize("full_every", [3, 0])
def test_ratio_100_is_bitwise_full_recompute(full_every):
    marche = _run(TINY, 1, full_every=full_every, policy="ratio", budget=10000)
    full = _run(TINY, 1, full_every=1, policy="ratio", budget=10000)
    for a, f in zip(marche, full):
        np.testing.assert_array_equal(a.x_out, f.x_out)
        for l in range(TINY.n_layers):
            np.testing.assert_array_equal(a.k_caches[l], f.k_caches[l])
            np.testing.assert_array_equal(a.v_caches[l], f.v_caches[l])
        if a.active is not None:
            assert sorted(a.active) == list(range(TINY.n_tokens))


def test_ratio_0_active_is_gen_and_caching():
    res = _run(TINY, 0, policy="ratio", budget=0)
    for t, r in enumerate(res):
        if schedule.is_full_step(t, TINY.full_every):
            assert r.refresh is None
        else:
            assert r.refresh == [] and r.active == r.gen + r.cache_tokens


def test_fixed_budget_fills_active_set():
    res = _run(TINY, 0, policy="fixed", budget=12)
    for r in res:
        if r.refresh is not None:
            assert len(r.active) == max(12, len(r.gen) + len(r.cache_tokens))
            assert len(set(r.active)) == len(r.active)


def test_full_step_is_stack_of_full_layers_and_scores_from_gen():
    cfg = TINY
    p, e, o = _inputs(cfg)
    H, N, dh = cfg.n_heads, cfg.n_tokens, cfg.head_dim
    rng = np.random.default_rng(5)
    kcs = [rng.normal(size=(H, N, dh)) for _ in p]
    vcs = [rng.normal(size=(H, N, dh)) for _ in p]
    t = 4
    gen = schedule.generating_tokens(o[0], cfg.n_buf, cfg.n_steps, t)
    cache = schedule.caching_tokens(o[0], cfg.n_buf, cfg.n_steps, t)
    known = schedule.known_before(o[0], cfg.n_buf, cfg.n_steps, t)
    x = step.decoder_input(e.cls[0], e.value[0], e.mask, e.pos, known, cfg.n_buf)
    # decoder input: buffer rows carry the class embedding, known image rows their
    # value embedding, masked rows the mask embedding; all add the position
    for j in range(N):
        base = e.cls[0] if j < cfg.n_buf else (e.value[0][j - cfg.n_buf] if j in known else e.mask)
        np.testing.assert_array_equal(x[j], base.astype(np.float64) + e.pos[j])
    full = step.marche_step(p, x, kcs, vcs, gen, cache, n_heads=H, eps=cfg.ln_eps,
                            sel_layer=2, full=True, k_refresh=3)
    xx = x
    for l in range(cfg.n_layers):
        xx = block.full_layer(p[l], xx, kcs[l], vcs[l], n_heads=H, eps=cfg.ln_eps).x_out
    np.testing.assert_array_equal(full.x_out, xx)
    assert full.refresh is None

    k = 3
    ca = step.marche_step(p, x, kcs, vcs, gen, cache, n_heads=H, eps=cfg.ln_eps,
                          sel_layer=2, full=False, k_refresh=k, keep_layers=True)
    # the selection layer (layer 2) is full; its scores are the attention mass
    # of the generating rows, which sums to |G| per head
    np.testing.assert_allclose(ca.scores.sum(axis=1), len(gen), rtol=1e-12)
    assert ca.refresh == select.select_topk(ca.scores.sum(axis=0), gen + cache, k)
    assert list(ca.layers[2].rows) == sorted(gen + cache + ca.refresh)
    # the first two layers are identical to the full step's
    np.testing.assert_array_equal(ca.layers[1].x_out, block.full_layer(
        p[1], ca.layers[0].x_out, kcs[1], vcs[1], n_heads=H, eps=cfg.ln_eps).x_out)


def test_no_generating_ablation_against_hand_composed_layers():
    """Table 2's variant without generating tokens: after the selection layer
    A = N u R, R is still chosen from G's attention mass and excludes G.  Pinned
    against the layers composed by hand, and by what the variant must leave
    alone: the rows of G and their cache rows after the selection layer."""
    cfg = TINY.with_(n_layers=4, sel_layer=2)
    p, e, o = _inputs(cfg)
    H, N, dh = cfg.n_heads, cfg.n_tokens, cfg.head_dim
    rng = np.random.default_rng(17)
    kcs = [rng.normal(size=(H, N, dh)) for _ in p]
    vcs = [rng.normal(size=(H, N, dh)) for _ in p]
    t = 4
    gen = schedule.generating_tokens(o[1], cfg.n_buf, cfg.n_steps, t)
    cache = schedule.caching_tokens(o[1], cfg.n_buf, cfg.n_steps, t)
    known = schedule.known_before(o[1], cfg.n_buf, cfg.n_steps, t)
    x = step.decoder_input(e.cls[1], e.value[1], e.mask, e.pos, known, cfg.n_buf)
    k = 5
    res = step.marche_step(p, x, kcs, vcs, gen, cache, n_heads=H, eps=cfg.ln_eps, sel_layer=2,
                           full=False, k_refresh=k, keep_layers=True, include_gen=False)
    with_g = step.marche_step(p, x, kcs, vcs, gen, cache, n_heads=H, eps=cfg.ln_eps, sel_layer=2,
                              full=False, k_refresh=k, include_gen=True)

    # by hand: two full layers (scores of G at the second), top-k over the
    # tokens outside G u N, then cache-aware layers on N u R with no scoring rows
    xx, kk, vv = x, [c.copy() for c in kcs], [c.copy() for c in vcs]
    for l in range(2):
        r = block.full_layer(p[l], xx, kk[l], vv[l], gen, H, cfg.ln_eps, score=(l == 1))
        xx, kk[l], vv[l] = r.x_out, r.k_cache, r.v_cache
        if l == 1:
            sc = r.scores
    R = select.select_topk_bruteforce(sc.sum(axis=0), gen + cache, k)
    assert res.refresh == R == with_g.refresh
    assert not set(R) & set(gen + cache) and len(R) == k
    x_sel = xx
    for l in range(2, cfg.n_layers):
        r = block.cache_aware_layer(p[l], xx, kk[l], vv[l], cache + R, [], H, cfg.ln_eps)
        xx, kk[l], vv[l] = r.x_out, r.k_cache, r.v_cache
    np.testing.assert_array_equal(res.x_out, xx)
    for l in range(cfg.n_layers):
        np.testing.assert_array_equal(res.k_caches[l], kk[l])
        np.testing.assert_array_equal(res.v_caches[l], vv[l])
    assert res.active == cache + R

    # G's rows keep the selection layer's output, and their cache rows in the
    # later layers keep the input's bits; with G included both change
    np.testing.assert_array_equal(res.x_out[gen], x_sel[gen])
    assert not np.allclose(with_g.x_out[gen], x_sel[gen])
    for l in range(2, cfg.n_layers):
        np.testing.assert_array_equal(res.k_caches[l][:, gen], kcs[l][:, gen])
        assert not np.allclose(with_g.k_caches[l][:, gen], kcs[l][:, gen])
    # the rows both variants recompute see different keys at G, so they differ too
    assert not np.allclose(res.x_out[cache], with_g.x_out[cache])


def test_decoder_input_row_kinds_and_positional_add():
    """The decoder input's rows (Eq. 2's stand-in): each buffer position holds
    the class row, each known image token its own value row (value_emb is
    indexed by image position j - n_buf), every other position the shared mask
    row, and the positional row adds on top of each.  Distinct random rows make
    a wrong branch, a value row taken at j instead of j - n_buf, or a dropped
    positional term fail."""
    rng = np.random.default_rng(11)
    n_buf, n_img, d = 3, 9, 5
    cls = rng.standard_normal(d)
    value = rng.standard_normal((n_img, d))
    mask = rng.standard_normal(d)
    known = [n_buf + 1, n_buf + 4, n_buf + 8]
    zero = np.zeros((n_buf + n_img, d))
    x0 = step.decoder_input(cls, value, mask, zero, known, n_buf)
    for j in range(n_buf + n_img):
        want = cls if j < n_buf else value[j - n_buf] if j in known else mask
        np.testing.assert_array_equal(x0[j], want)
    pos = rng.standard_normal((n_buf + n_img, d))
    np.testing.assert_allclose(step.decoder_input(cls, value, mask, pos, known, n_buf), x0 + pos,
                               rtol=0, atol=1e-15)
    # the order in which known tokens are listed does not matter
    np.testing.assert_array_equal(step.decoder_input(cls, value, mask, pos, known[::-1], n_buf),
                                  step.decoder_input(cls, value, mask, pos, known, n_buf))
