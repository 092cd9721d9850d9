"""Seeded synthetic inputs: determinism, per-layer independence and exact
storage-dtype rounding (CPU only)."""
import numpy as np
import torch

from paper_2506_12035_amd import workload


def test_bf16_rounding_matches_torch_rne():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.normal(size=10000).astype(np.float32),
                        np.array([0.0, -0.0, 1e-40, 3.4e38, -3.4e38, np.inf, -np.inf], np.float32)])
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(workload.round_to(a, "bf16"), ref)
    assert np.isnan(workload.round_to(np.array([np.nan], np.float32), "bf16")[0])


def test_weights_deterministic_and_layer_independent():
    cfg = workload.CONFIGS[2].with_(n_layers=3, d_model=64, n_heads=4, head_dim=16, d_mlp=256)
    w1 = workload.layer_weights(cfg, 1)
    w1b = workload.layer_weights(cfg, 1)
    w0 = workload.layer_weights(cfg, 0)
    for k in workload.LAYER_PARAM_NAMES:
        np.testing.assert_array_equal(w1[k], w1b[k])
        assert not np.array_equal(w1[k], w0[k])
        np.testing.assert_array_equal(workload.round_to(w1[k], "bf16"), w1[k])
    assert w1["w_qkv"].shape == (192, 64) and w1["w_2"].shape == (64, 256)
    assert abs(float(w1["w_qkv"].std()) - 0.02) < 0.002


def test_orders_and_single_block_case():
    cfg = workload.CONFIGS[1]
    o = workload.orders(cfg.with_(batch=3))
    assert all(sorted(r) == list(range(cfg.n_img)) for r in o)
    c = workload.single_block_case(cfg)
    assert c.x.shape == (1, 320, 768) and c.k_cache.shape == (1, 12, 320, 64)
    a = c.active[0]
    assert len(set(a.tolist())) == 32
    assert all(j >= cfg.n_buf for j in a[:16])


def test_config_shapes():
    for cid, c in workload.CONFIGS.items():
        assert c.d_model == c.n_heads * c.head_dim
        assert c.d_mlp == 4 * c.d_model
    assert workload.CONFIGS[5].n_tokens == 1088 and workload.CONFIGS[4].head_dim == 80


def test_image_ranges_are_slices_of_the_whole_batch():
    cfg = workload.CONFIGS[2].with_(batch=7, d_model=64, n_heads=4, head_dim=16, d_mlp=256)
    whole_e, whole_o = workload.embeddings(cfg), workload.orders(cfg)
    part_e, part_o = workload.embeddings(cfg, 3, first=2), workload.orders(cfg, 3, first=2)
    np.testing.assert_array_equal(part_o, whole_o[2:5])
    np.testing.assert_array_equal(part_e.cls, whole_e.cls[2:5])
    np.testing.assert_array_equal(part_e.value, whole_e.value[2:5])
    np.testing.assert_array_equal(part_e.pos, whole_e.pos)
    np.testing.assert_array_equal(part_e.mask, whole_e.mask)
    for bad in ((5, 3), (-1, 0)):
        with np.testing.assert_raises(ValueError):
            workload.orders(cfg, *bad)


def test_random_refresh_draws_per_image():
    cfg = workload.CONFIGS[2]
    rng = np.random.default_rng(3)
    cand = np.stack([np.sort(rng.choice(320, size=200, replace=False)) for _ in range(6)]).astype(np.int32)
    whole = workload.random_refresh(cfg, 4, cand, 20)
    np.testing.assert_array_equal(workload.random_refresh(cfg, 4, cand[2:5], 20, first=2), whole[2:5])
    for b in range(6):
        assert len(set(whole[b].tolist())) == 20 and set(whole[b].tolist()) <= set(cand[b].tolist())
        assert list(whole[b]) == sorted(whole[b])
    assert not np.array_equal(whole, workload.random_refresh(cfg, 5, cand, 20))


def test_engine_rejects_bad_range_sizes():
    """Explicit image counts per range are checked before any device work:
    empty, non-positive, or not summing to the batch."""
    import pytest
    from paper_2506_12035_amd import driver

    cfg = workload.CONFIGS[2]
    for sizes in ([], [0, 64], [10, 10], [-1, 65], [32, 33]):
        with pytest.raises(ValueError, match="range_sizes"):
            driver.Engine(cfg, device="cpu", range_sizes=sizes)
    with pytest.raises(ValueError, match="micro_batches"):
        driver.Engine(cfg, device="cpu", micro_batches=0)
