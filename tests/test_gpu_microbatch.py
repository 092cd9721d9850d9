"""Micro-batched decoding: the batch split into micro-batches of consecutive
images, each on its own HIP stream, against one engine over the whole batch.

Images are independent and every kernel computes a row (or an image and head)
the same way whatever else shares the launch, so the KV cache and the
residual stream must match bit for bit over full and cache-aware steps."""
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
def test_micro_batches_match_the_whole_batch(whole, parts, overlap):
    cfg, ws, ref = whole
    say(f"micro-batches: {cfg.name} B={ref.B} parts={parts} overlap={overlap}")
    mb = driver.MicroBatchEngine(cfg, micro_batches=parts, weights=ws)
    mb.overlap = overlap
    assert sum(e.B for e in mb.engines) == ref.B
    assert all(e.params is mb.engines[0].params for e in mb.engines)
    for t in STEPS:
        mb.step(t)
    torch.cuda.synchronize()
    for e in mb.engines:
        sl = slice(e.first_image, e.first_image + e.B)
        assert torch.equal(e.x, ref.x[sl]), f"x of images {sl}"
        for l in range(cfg.n_layers):
            assert torch.equal(e.k_layer(l), ref.k_layer(l)[sl]), f"K of layer {l}, images {sl}"
            assert torch.equal(e.v_layer(l), ref.v_layer(l)[sl]), f"V of layer {l}, images {sl}"
