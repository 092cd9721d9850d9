"""GPU parity of one block through the C ABI against the fp64 oracle.

Covers the single-block fp32 case (one cache-aware layer + attention-mass
scores + top-16 refresh selection, plain and with planted structure), and bf16
layers at the MAR-L, MAR-H (head_dim 80) and long-KV (N=1088) widths with
ragged active sets that span several query chunks and a ragged key tail.
Checks: fresh K/V rows, attention output, block delta of x, per-head scores
within the dtype tolerance; cache rows and x rows outside A bitwise unchanged;
refresh sets exact when the oracle's gap at the k-th boundary exceeds the
tolerance, else tolerance-valid; selection on identical fp32 scores exact.
"""
import numpy as np
import pytest
import torch

from oracle import block, select
from paper_2506_12035_amd import binding, workload
from tests.gpu_util import DEV, TOL, SingleLayer, check_refresh_set, f64, rel_err, say

pytestmark = pytest.mark.gpu


def _oracle_layer(cfg, p64, x, kc, vc, active, n_gen):
    out = []
    for b in range(x.shape[0]):
        a = [int(v) for v in active[b]]
        out.append(block.cache_aware_layer(p64, x[b], kc[b], vc[b], a, a[:n_gen[b]],
                                           n_heads=cfg.n_heads, eps=cfg.ln_eps, score=True))
    return out


def _check_layer(cfg, x, kc, vc, active, n_gen, gpu, ref, tol):
    N = cfg.n_tokens
    off = gpu["off"]
    worst = {}
    for b, r in enumerate(ref):
        a = np.asarray(active[b])
        rest = np.setdiff1d(np.arange(N), a)
        # cache rows outside A keep their bits; x rows outside A are untouched
        np.testing.assert_array_equal(gpu["k"][b][:, rest], kc[b][:, rest])
        np.testing.assert_array_equal(gpu["v"][b][:, rest], vc[b][:, rest])
        np.testing.assert_array_equal(gpu["x"][b][rest], x[b][rest])
        rows = r.rows
        pos = {int(t): i for i, t in enumerate(rows)}
        perm = np.array([pos[int(t)] for t in a])
        errs = {
            "k": rel_err(gpu["k"][b][:, rows], r.k_cache[:, rows]),
            "v": rel_err(gpu["v"][b][:, rows], r.v_cache[:, rows]),
            "o": rel_err(gpu["o"][off[b]:off[b + 1]], r.o[perm]),
            "dx": rel_err(gpu["x"][b][rows] - x[b][rows], r.x_out[rows] - x[b][rows]),
            "x": rel_err(gpu["x"][b][rows], r.x_out[rows]),
            "scores": rel_err(gpu["scores"][b], r.scores),
        }
        for k, e in errs.items():
            worst[k] = max(worst.get(k, 0.0), e)
    say("  max rel err:", {k: f"{v:.2e}" for k, v in worst.items()})
    for k, e in worst.items():
        assert e <= tol, f"{k}: rel err {e:.3e} > {tol}"
    return worst


def _select_gpu(scores, excl_lists, k, lowest=False):
    B, H, N = scores.shape
    excl = np.concatenate([np.asarray(e, np.int32) for e in excl_lists])
    eoff = np.zeros(B + 1, np.int32)
    eoff[1:] = np.cumsum([len(e) for e in excl_lists])
    out = torch.full((B * k,), -7, dtype=torch.int32, device=DEV)
    ooff = torch.from_numpy(np.arange(B, dtype=np.int32) * k).to(DEV)
    s_dev = torch.from_numpy(np.ascontiguousarray(scores, np.float32)).to(DEV)
    say(f"  select_refresh: B={B} parts={H} N={N} k={k}")
    binding.select_refresh(s_dev, H, torch.from_numpy(excl).to(DEV), torch.from_numpy(eoff).to(DEV),
                           B, N, k, out, ooff, lowest=lowest)
    torch.cuda.synchronize()
    return out.cpu().numpy().reshape(B, k)


def _fp32_head_sum(scores_bh):
    """Head sum in float32, heads in order (the kernel's summation order)."""
    s = np.zeros(scores_bh.shape[1], np.float32)
    for h in range(scores_bh.shape[0]):
        s = (s + scores_bh[h].astype(np.float32)).astype(np.float32)
    return s


def _check_refresh(gpu_sel, ref_scores, excl, k, tol):
    """Gap rule: exact when the oracle's k-th boundary gap exceeds tol, else
    valid on both sides of the boundary (tests.gpu_util.check_refresh_set)."""
    got = [int(v) for v in gpu_sel]
    assert got == sorted(got), "refresh set not ascending"
    return check_refresh_set(got, ref_scores.sum(axis=0), excl, k, tol) == "exact"


def _single_block_inputs(planted=False):
    cfg = workload.CONFIGS[1]
    case = workload.single_block_case(cfg)
    p = workload.layer_weights(cfg, 0)
    kc = case.k_cache.copy()
    if planted:
        # Shift the cached keys of 16 candidate tokens towards the mean query
        # direction of the generating tokens (per head), computed by the oracle,
        # so that their attention mass clearly exceeds every other candidate's.
        p64 = f64(p)
        a = case.active[0]
        r = block.cache_aware_layer(p64, case.x[0], kc[0], case.v_cache[0], a, a[:case.n_gen],
                                    n_heads=cfg.n_heads, eps=cfg.ln_eps)
        gen_pos = [list(r.rows).index(int(t)) for t in a[:case.n_gen]]
        cand = np.setdiff1d(np.arange(cfg.n_tokens), a)
        planted_rows = workload.planted_rows(cfg, cand, case.k_top)[0]
        dh = cfg.head_dim
        for h in range(cfg.n_heads):
            qm = r.q[gen_pos, h * dh:(h + 1) * dh].mean(axis=0)
            shift = 3.0 * np.sqrt(dh) * qm / (qm @ qm)
            kc[0, h, planted_rows] += shift.astype(np.float32)
        kc = workload.round_to(kc, cfg.dtype)
        return cfg, case, p, kc, planted_rows
    return cfg, case, p, kc, None


@pytest.mark.parametrize("planted", [False, True])
def test_single_block_fp32_with_refresh(planted):
    cfg, case, p, kc, planted_rows = _single_block_inputs(planted)
    say(f"single block fp32 planted={planted}")
    ref = _oracle_layer(cfg, f64(p), case.x, kc, case.v_cache, case.active, [case.n_gen])
    run = SingleLayer(cfg, p, case.x, kc, case.v_cache)
    gpu = run.run(case.active, [case.n_gen])
    _check_layer(cfg, case.x, kc, case.v_cache, case.active, [case.n_gen], gpu, ref, TOL["f32"])

    excl = case.active[0]
    sel = _select_gpu(gpu["scores"], [excl], case.k_top)[0]
    # identical fp32 scores: selection is exact
    assert list(sel) == select.select_topk(_fp32_head_sum(gpu["scores"][0]), excl, case.k_top)
    exact = _check_refresh(sel, ref[0].scores, excl, case.k_top, TOL["f32"])
    if planted:
        assert exact and sorted(sel) == sorted(planted_rows.tolist())


BF16_SHAPES = {
    "mar-l": dict(cid=3, n_tokens=320),
    "mar-h": dict(cid=4, n_tokens=320),
    "hires": dict(cid=5, n_tokens=1088),
    # a key count that is not a multiple of the 64-key tile: masked tail
    "ragged-keys": dict(cid=3, n_tokens=300),
    "ragged-keys-dh80": dict(cid=4, n_tokens=203),
}


def _ragged_case(cfg, B, sizes, gens, seed):
    rng = np.random.default_rng(seed)
    N = cfg.n_tokens
    x = rng.standard_normal((B, N, cfg.d_model), dtype=np.float32)
    kc = workload.round_to(rng.standard_normal((B, cfg.n_heads, N, cfg.head_dim), dtype=np.float32), "bf16")
    vc = workload.round_to(rng.standard_normal((B, cfg.n_heads, N, cfg.head_dim), dtype=np.float32), "bf16")
    active = [rng.permutation(N)[:sizes[b]].astype(np.int32) for b in range(B)]
    return x, kc, vc, active, gens


@pytest.mark.parametrize("shape", list(BF16_SHAPES))
def test_bf16_layer_ragged(shape):
    spec = BF16_SHAPES[shape]
    cfg = workload.CONFIGS[spec["cid"]].with_(**{k: v for k, v in spec.items() if k != "cid"})
    N = cfg.n_tokens
    # ragged active sets: a single token, a typical cache-aware set, a set that
    # spans two query chunks, and every token (a full layer)
    sizes = [1, 39, 161, N]
    gens = [1, 5, 25, 7]
    B = len(sizes)
    x, kc, vc, active, gens = _ragged_case(cfg, B, sizes, gens, seed=11 + spec["cid"])
    p = workload.layer_weights(cfg, 0)
    say(f"bf16 layer {shape}: sizes={sizes}")
    ref = _oracle_layer(cfg, f64(p), x, kc, vc, active, gens)
    run = SingleLayer(cfg, p, x, kc, vc)
    gpu = run.run(active, gens)
    _check_layer(cfg, x, kc, vc, active, gens, gpu, ref, TOL["bf16"])
    # refresh selection over the complement of each active set
    k = 16
    excl = [a for a in active[:3]]
    sel = _select_gpu(gpu["scores"][:3], excl, k)
    for b in range(3):
        assert list(sel[b]) == select.select_topk(_fp32_head_sum(gpu["scores"][b]), excl[b], k)
        _check_refresh(sel[b], ref[b].scores, excl[b], k, TOL["bf16"])


@pytest.mark.parametrize("n_tokens", [320, 300])
def test_bf16_layer_short_active_sets(n_tokens):
    """Cache-aware layers where every image has at most 64 active rows (the
    short-query resident attention at head width 64): a single token, a
    typical set, exactly 64 and a ragged one; full and ragged key counts."""
    cfg = workload.CONFIGS[3].with_(n_tokens=n_tokens)
    sizes, gens = [1, 39, 64, 23], [1, 5, 9, 3]
    x, kc, vc, active, gens = _ragged_case(cfg, len(sizes), sizes, gens, seed=23 + n_tokens)
    p = workload.layer_weights(cfg, 2)
    say(f"bf16 layer short active sets N={n_tokens}")
    ref = _oracle_layer(cfg, f64(p), x, kc, vc, active, gens)
    gpu = SingleLayer(cfg, p, x, kc, vc).run(active, gens)
    _check_layer(cfg, x, kc, vc, active, gens, gpu, ref, TOL["bf16"])


def test_bf16_layer_deterministic():
    cfg = workload.CONFIGS[3]
    sizes, gens = [44, 320, 7], [6, 6, 1]
    x, kc, vc, active, gens = _ragged_case(cfg, 3, sizes, gens, seed=5)
    p = workload.layer_weights(cfg, 1)
    outs = []
    for rep in range(2):
        say(f"determinism run {rep}")
        outs.append(SingleLayer(cfg, p, x, kc, vc).run(active, gens))
    for key in ("x", "k", "v", "o", "scores"):
        np.testing.assert_array_equal(outs[0][key], outs[1][key])


def test_select_refresh_edge_cases():
    rng = np.random.default_rng(2)
    N, H = 37, 3
    s = rng.random((4, H, N)).astype(np.float32)
    s[1] = 0.25                      # all equal: the lowest candidate indices win
    s[2, :, 5] = np.nan              # NaN ranks below every number
    s[3, 0, :] = -0.0                # signed zeros tie
    excl = [[0, 3], [1, 2, 4], [], list(range(30))]
    k = 7
    sel = _select_gpu(s, excl, k)
    for b in range(4):
        if len(np.setdiff1d(np.arange(N), excl[b])) >= k:
            assert list(sel[b]) == select.select_topk(_fp32_head_sum(s[b]), excl[b], k)
    assert list(sel[1]) == [0, 3, 5, 6, 7, 8, 9]
    assert 5 not in sel[2]
    # image 3 has exactly 7 candidates
    assert list(sel[3]) == list(range(30, 37))
    # fewer candidates than k: trailing slots are -1
    sel2 = _select_gpu(s[:1], [list(range(33))], 6)
    assert list(sel2[0]) == [33, 34, 35, 36, -1, -1]


def test_select_refresh_lowest_first():
    # low-attention ablation: identical fp32 scores give the oracle's set exactly
    rng = np.random.default_rng(9)
    N, H, B = 1088, 16, 5
    s = rng.random((B, H, N)).astype(np.float32)
    s[1] = 0.5                       # all equal: lowest candidate indices
    s[2, :, 11] = np.nan             # NaN is never preferred
    excl = [rng.choice(N, 40, replace=False) for _ in range(B)]
    k = 31
    sel = _select_gpu(s, excl, k, lowest=True)
    for b in range(B):
        assert list(sel[b]) == select.select_topk(_fp32_head_sum(s[b]), excl[b], k, lowest=True)
    assert 11 not in sel[2]


def test_select_refresh_long_sequence_many_heads():
    # 20 heads (two batches of sixteen loads), 3000 tokens (two tokens per
    # thread), and an image with more exclusions than the workgroup has threads
    rng = np.random.default_rng(31)
    N, H, B = 3000, 20, 3
    s = rng.standard_normal((B, H, N)).astype(np.float32)
    s[1, :, 100:200] = 0.75          # a block of ties
    excl = [rng.choice(N, 1500, replace=False), rng.choice(N, 10, replace=False), np.arange(0)]
    k = 120
    for lowest in (False, True):
        sel = _select_gpu(s, excl, k, lowest=lowest)
        for b in range(B):
            assert list(sel[b]) == select.select_topk(_fp32_head_sum(s[b]), excl[b], k,
                                                      lowest=lowest)


def test_bf16_layer_cache_aware_range_size():
    """A cache-aware MAR-L layer on a 64-image range (34-44 active rows per
    image, about 2500 in all): the size at which the output projection and fc2
    take the 128x128 tile.  Every image against the oracle; the timing classes
    confirm which kernels ran."""
    cfg = workload.CONFIGS[3]
    B = 64
    rng = np.random.default_rng(77)
    sizes = [int(v) for v in rng.integers(34, 45, size=B)]
    gens = [int(v) for v in rng.integers(1, 8, size=B)]
    x, kc, vc, active, gens = _ragged_case(cfg, B, sizes, gens, seed=78)
    p = workload.layer_weights(cfg, 5)
    say(f"bf16 layer at a 64-image range: a_total={sum(sizes)}")
    ref = _oracle_layer(cfg, f64(p), x, kc, vc, active, gens)
    run = SingleLayer(cfg, p, x, kc, vc)
    binding.profile_reset()
    binding.profile_enable(True)
    try:
        gpu = run.run(active, gens)
        prof = binding.profile_collect()
    finally:
        binding.profile_enable(False)
        binding.profile_reset()
    _check_layer(cfg, x, kc, vc, active, gens, gpu, ref, TOL["bf16"])
    assert {"gemm_o_t128_ca", "gemm_fc2_t128_ca"} <= set(prof), sorted(prof)
