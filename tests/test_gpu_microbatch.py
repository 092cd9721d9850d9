"""Cache-aware layers split into ranges of consecutive images, each range on
its own HIP stream (marche_step_images), against the whole batch in one call.

Images are independent and every kernel computes a row (or an image and head)
the same way whatever else shares the launch, so the KV cache and the
residual stream must match bit for bit over full and cache-aware steps, with
the ranges overlapping on the GPU or run one after another."""
import pytest
import torch

from paper_2506_12035_amd import driver, workload
from tests.gpu_util import say

pytestmark = pytest.mark.gpu

STEPS = range(5)  # full step 0, cache-aware 1-2, periodic full 3, cache-aware 4


@pytest.fixture(scope="module")
def whole():
    cfg = workload.CONFIGS[2]
    ws = workload.all_weights(cfg)
    eng = driver.Engine(cfg, weights=ws)
    for t in STEPS:
        eng.step(t)
    torch.cuda.synchronize()
    return cfg, ws, eng


@pytest.mark.parametrize("parts,overlap", [(2, True), (3, True), (2, False)])
def test_image_ranges_match_the_whole_batch(whole, parts, overlap):
    cfg, ws, ref = whole
    say(f"image ranges: {cfg.name} B={ref.B} parts={parts} overlap={overlap}")
    eng = driver.Engine(cfg, weights=ws, micro_batches=parts)
    eng.overlap = overlap
    assert sum(n for _, n in eng.ranges) == ref.B
    for t in STEPS:
        eng.step(t)
        if not eng.plans[t].full:
            assert eng.plans[t].parts is not None and len(eng.plans[t].parts) == parts
    torch.cuda.synchronize()
    assert torch.equal(eng.x, ref.x)
    for l in range(cfg.n_layers):
        assert torch.equal(eng.k_layer(l), ref.k_layer(l)), f"K of layer {l}"
        assert torch.equal(eng.v_layer(l), ref.v_layer(l)), f"V of layer {l}"
    for t in STEPS:
        if not eng.plans[t].full:
            assert torch.equal(eng.plans[t].ca_idx, ref.plans[t].ca_idx), f"active lists of step {t}"


@pytest.mark.timeout(600)
def test_headline_ranges_match_the_whole_batch():
    """The benchmark's default launch configuration at the headline MAR-L
    size (batch 128, 32 layers): every step as two 64-image ranges on two
    streams gives the same bits as the whole batch in one call, over full and
    cache-aware steps.  Together with the stack parity test (whole batch
    against the oracle) this covers the configuration the benchmark times."""
    cfg = workload.CONFIGS[3]
    say(f"image ranges: {cfg.name} B={cfg.batch} default ranges vs one call")
    ws = workload.all_weights(cfg)
    ref = driver.Engine(cfg, weights=ws)
    for t in STEPS:
        ref.step(t)
    torch.cuda.synchronize()
    x_ref = ref.x.clone()
    k_ref = [ref.k_layer(l).clone() for l in range(cfg.n_layers)]
    v_ref = [ref.v_layer(l).clone() for l in range(cfg.n_layers)]
    del ref
    torch.cuda.empty_cache()
    eng = driver.Engine(cfg, weights=ws, micro_batches=2)
    assert [n for _, n in eng.ranges] == [64, 64]
    for t in STEPS:
        eng.step(t)
    torch.cuda.synchronize()
    assert torch.equal(eng.x, x_ref)
    for l in range(cfg.n_layers):
        assert torch.equal(eng.k_layer(l), k_ref[l]), f"K of layer {l}"
        assert torch.equal(eng.v_layer(l), v_ref[l]), f"V of layer {l}"


def test_uneven_range_sizes_match_the_whole_batch(whole):
    """Explicit image counts per range (Engine(range_sizes=...)): unequal
    ranges, the first larger than the rest, give the same bits as one call."""
    cfg, ws, ref = whole
    sizes = [ref.B // 2 + 3, ref.B // 4, ref.B - (ref.B // 2 + 3) - ref.B // 4]
    say(f"image ranges: {cfg.name} B={ref.B} sizes={sizes}")
    eng = driver.Engine(cfg, weights=ws, range_sizes=sizes)
    assert [n for _, n in eng.ranges] == sizes
    assert [f for f, _ in eng.ranges] == [0, sizes[0], sizes[0] + sizes[1]]
    for t in STEPS:
        eng.step(t)
    torch.cuda.synchronize()
    assert torch.equal(eng.x, ref.x)
    for l in range(cfg.n_layers):
        assert torch.equal(eng.k_layer(l), ref.k_layer(l)), f"K of layer {l}"
        assert torch.equal(eng.v_layer(l), ref.v_layer(l)), f"V of layer {l}"


def test_step_images_touches_only_its_range():
    """marche_step_images on images [2, 4) of a 4-image cache and residual
    stream: images 0 and 1 keep every bit of x and of both caches, and images
    2 and 3 equal what marche_step over all four images computes for them."""
    import numpy as np
    from paper_2506_12035_amd import binding

    cfg = workload.CONFIGS[2].with_(n_layers=2, batch=4)
    B, N, D, H, dh, L = 4, cfg.n_tokens, cfg.d_model, cfg.n_heads, cfg.head_dim, 2
    say(f"marche_step_images: {cfg.name} reduced to L={L}, B={B}, images [2, 4)")
    rng = np.random.default_rng(5)
    model = binding.make_model(L, D, H, dh, cfg.d_mlp, N, binding.MARCHE_BF16, cfg.ln_eps)
    params = []
    for l in range(L):
        w = workload.layer_weights(cfg, l)
        params.append({k: torch.from_numpy(np.ascontiguousarray(v, np.float32)).to(
            torch.bfloat16 if k.startswith("w_") else torch.float32).cuda() for k, v in w.items()})
    layers = binding.make_layers(params)
    x0 = torch.from_numpy(rng.standard_normal((B, N, D)).astype(np.float32)).cuda()
    n_el = L * B * H * N * dh
    k0 = torch.from_numpy(rng.standard_normal(n_el).astype(np.float32)).to(torch.bfloat16).cuda()
    v0 = torch.from_numpy(rng.standard_normal(n_el).astype(np.float32)).to(torch.bfloat16).cuda()
    act = [np.sort(rng.choice(N, size=a, replace=False)).astype(np.int32) for a in (40, 37, 44, 29)]
    n_gen = [5, 4, 6, 3]

    def run(first, count):
        x = x0.clone()
        k, v = k0.clone(), v0.clone()
        cache = binding.kv_cache_init(model, B, k, v, n_el * 2, k_init=k0, v_init=v0)
        lists = act[first:first + count]
        idx = torch.from_numpy(np.concatenate(lists)).cuda()
        off = torch.from_numpy(np.concatenate([[0], np.cumsum([len(a) for a in lists])]).astype(np.int32)).cuda()
        gen = torch.tensor(n_gen[first:first + count], dtype=torch.int32).cuda()
        total, a_max = int(off[-1]), max(len(a) for a in lists)
        wsb = binding.workspace_bytes(model, count, total)
        ws = torch.empty(wsb, dtype=torch.uint8).cuda()
        binding.marche_step_images(model, layers, cache, first, 0, L, count, x[first:first + count],
                                   idx, off, gen, total, a_max, max(n_gen[first:first + count]),
                                   None, -1, ws, wsb)
        torch.cuda.synchronize()
        return x, k.view(L, B, H, N, dh), v.view(L, B, H, N, dh)

    x_all, k_all, v_all = run(0, 4)
    x_part, k_part, v_part = run(2, 2)
    k_in, v_in = k0.view(L, B, H, N, dh), v0.view(L, B, H, N, dh)
    assert torch.equal(x_part[:2], x0[:2])
    assert torch.equal(k_part[:, :2], k_in[:, :2]) and torch.equal(v_part[:, :2], v_in[:, :2])
    assert torch.equal(x_part[2:], x_all[2:])
    assert torch.equal(k_part[:, 2:], k_all[:, 2:]) and torch.equal(v_part[:, 2:], v_all[:, 2:])
    assert not torch.equal(x_part[2:], x0[2:])  # the range was really computed
