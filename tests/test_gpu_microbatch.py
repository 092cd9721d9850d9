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
