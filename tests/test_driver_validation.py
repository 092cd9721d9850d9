"""Host-side range checks of the decoding driver (CPU only).

A refresh count above the number of candidates would make the device
selection pad the active list with -1 entries, which the step then uses as
token indices.  The driver therefore refuses such budgets before touching the
device, and every step plan re-checks its count.
"""
import numpy as np
import pytest
import torch

from paper_2506_12035_amd import driver, schedule, workload

CFG = workload.CONFIGS[2].with_(n_layers=2, batch=3)


@pytest.mark.parametrize("policy,value", [("ratio", -1), ("ratio", 10001), ("ratio", 20000),
                                          ("fixed", -1), ("fixed", 321), ("bogus", 10)])
def test_check_budget_rejects(policy, value):
    with pytest.raises(ValueError):
        schedule.check_budget(policy, value, 320)


@pytest.mark.parametrize("policy,value", [("ratio", 0), ("ratio", 10000), ("fixed", 0),
                                          ("fixed", 64), ("fixed", 320)])
def test_check_budget_accepts_and_count_fits(policy, value):
    schedule.check_budget(policy, value, 320)
    for g, n in ((1, 0), (7, 6), (25, 25)):
        k = schedule.refresh_count(policy, value, 320, g, n)
        assert 0 <= k <= 320 - g - n


@pytest.mark.parametrize("kw", [dict(ratio_bp=20000), dict(ratio_bp=-5),
                                dict(policy="fixed", budget=400), dict(full_every=-1)])
def test_engine_rejects_before_touching_the_device(kw):
    # device "cpu": a check that ran after any device allocation would fail
    # differently (the library needs a GPU), so ValueError proves the order
    with pytest.raises(ValueError):
        driver.Engine(CFG, device="cpu", **kw)


def test_plan_rechecks_refresh_count():
    eng = object.__new__(driver.Engine)
    eng.cfg, eng.B, eng.device = CFG, CFG.batch, torch.device("cpu")
    eng.orders = workload.orders(CFG, CFG.batch)
    eng.full_every, eng.strategy, eng.first_image = 3, "marche", 0
    eng.ranges = [(0, CFG.batch)]
    eng.policy, eng.budget = "ratio", 1000
    p = eng._plan(1)
    assert p.k == schedule.refresh_count("ratio", 1000, CFG.n_tokens, p.g, p.n)
    eng.policy, eng.budget = "ratio", 30000    # bypasses check_budget on purpose
    with pytest.raises(ValueError, match="exceeds"):
        eng._plan(1)
