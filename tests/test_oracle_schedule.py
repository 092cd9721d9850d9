"""Pins of the oracle's decoding schedule (CPU only): Eq. 1-4's masked sets
shrink to empty and the generated sets partition the image tokens; golden
count sequences; the full-refresh rule of Section 4.3."""
import math
import os

import numpy as np
import pytest

from oracle import schedule

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "schedule_counts.txt")


def _golden():
    out = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        n, seq = line.split(":")
        out[int(n)] = [int(v) for v in seq.split()]
    return out


@pytest.mark.parametrize("n_img", [256, 1024])
def test_golden_counts(n_img):
    assert schedule.generated_counts(n_img, 64) == _golden()[n_img]


@pytest.mark.parametrize("n_img,T", [(256, 64), (1024, 64), (16, 8), (5, 5), (100, 7)])
def test_counts_partition(n_img, T):
    m = schedule.masked_counts(n_img, T)
    assert m[0] == n_img and m[-1] == 0 and len(m) == T + 1
    c = schedule.generated_counts(n_img, T)
    assert sum(c) == n_img and min(c) >= 1
    # m_t tracks the cosine curve N cos(pi t / 2T) from below, within the
    # one-token-per-step floor
    for t in range(1, T):
        assert m[t] <= max(1, math.floor(n_img * math.cos(math.pi * t / (2 * T))))


def test_sets_disjoint_cover_and_caching():
    rng = np.random.default_rng(3)
    n_buf, n_img, T = 4, 40, 9
    order = rng.permutation(n_img)
    seen = []
    for t in range(T):
        g = schedule.generating_tokens(order, n_buf, T, t)
        assert not set(g) & set(seen)
        assert set(schedule.known_before(order, n_buf, T, t)) == set(seen)
        n = schedule.caching_tokens(order, n_buf, T, t)
        assert n == ([] if t == 0 else schedule.generating_tokens(order, n_buf, T, t - 1))
        assert all(n_buf <= j < n_buf + n_img for j in g)
        seen += g
    assert sorted(seen) == list(range(n_buf, n_buf + n_img))
    # generation follows the order: step t takes the next |G^(t)| positions of pi
    assert seen == [n_buf + int(o) for o in order]


def test_full_steps():
    full = [t for t in range(64) if schedule.is_full_step(t, 3)]
    assert full[:4] == [0, 3, 6, 9] and len(full) == 22
    assert [t for t in range(64) if schedule.is_full_step(t, 0)] == [0]
