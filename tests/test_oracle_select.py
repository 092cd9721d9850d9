"""Pins of the oracle's refresh selection and budget (CPU only): brute force on
tiny inputs, exhaustive subset enumeration, and the worked budget example of
Section 4.3 (5 generating + 9 caching + 50 refreshing = 64 active tokens)."""
import itertools

import numpy as np
import pytest

from oracle import select

RNG = np.random.default_rng(7)


@pytest.mark.parametrize("trial", range(40))
def test_topk_matches_bruteforce_and_subset_enumeration(trial):
    n = int(RNG.integers(1, 13))
    # small integer scores force ties
    s = RNG.integers(0, 4, size=n).astype(float)
    n_ex = int(RNG.integers(0, n))
    excl = RNG.choice(n, n_ex, replace=False).tolist()
    n_cand = n - n_ex
    k = int(RNG.integers(0, n_cand + 1))
    got = select.select_topk(s, excl, k)
    assert got == select.select_topk_bruteforce(s, excl, k)
    assert got == sorted(got) and len(got) == k and not set(got) & set(excl)
    cand = [j for j in range(n) if j not in excl]
    best = max((sum(s[j] for j in c) for c in itertools.combinations(cand, k)), default=0.0)
    assert sum(s[j] for j in got) == best
    # among the maximal-sum subsets, ties go to the lower indices: the chosen set
    # is the lexicographically smallest maximal one
    maximal = [list(c) for c in itertools.combinations(cand, k) if sum(s[j] for j in c) == best]
    assert got == min(maximal)


def test_all_equal_scores_pick_lowest_candidates():
    s = np.full(20, 0.5)
    assert select.select_topk(s, [0, 2, 3], 4) == [1, 4, 5, 6]


def test_nan_ranks_last_and_distinct_scores():
    s = np.array([0.1, np.nan, 0.3, 0.2, np.nan, -5.0])
    assert select.select_topk(s, [], 3) == [0, 2, 3]
    assert select.select_topk(s, [], 5) == [0, 1, 2, 3, 5]
    assert select.select_topk_bruteforce(s, [], 5) == [0, 1, 2, 3, 5]


def test_too_many_requested():
    with pytest.raises(ValueError):
        select.select_topk([1.0, 2.0, 3.0], [0, 1], 2)


def test_budget_worked_example():
    # Section 4.3: budget 64, 5 generating, 9 caching -> 50 refreshing tokens.
    assert select.budget_fixed(64, 5, 9) == 50
    assert select.budget_fixed(64, 40, 30) == 0


def test_budget_ratio_special_cases():
    # 100% of the candidates: every token is active (full recompute)
    assert select.budget_ratio(10000, 320, 5, 9) == 320 - 14
    # 0%: no refreshing tokens, A = G u N
    assert select.budget_ratio(0, 320, 5, 9) == 0
    # 10% rounds half up: 0.1 * 305 = 30.5 -> 31; 0.1 * 304 = 30.4 -> 30
    assert select.budget_ratio(1000, 320, 6, 9) == 31
    assert select.budget_ratio(1000, 320, 7, 9) == 30


def test_total_scores_sums_heads():
    s = RNG.random((3, 9))
    np.testing.assert_allclose(select.total_scores(s), s[0] + s[1] + s[2], rtol=1e-15)


@pytest.mark.parametrize("trial", range(25))
def test_lowest_first_matches_bruteforce_and_enumeration(trial):
    # the low-attention ablation: the k candidates with the lowest scores
    rng = np.random.default_rng(100 + trial)
    n = int(rng.integers(1, 12))
    s = rng.integers(0, 4, size=n).astype(float)
    excl = rng.choice(n, int(rng.integers(0, n)), replace=False).tolist()
    cand = [j for j in range(n) if j not in excl]
    k = int(rng.integers(0, len(cand) + 1))
    got = select.select_topk(s, excl, k, lowest=True)
    assert got == select.select_topk_bruteforce(s, excl, k, lowest=True)
    best = min((sum(s[j] for j in c) for c in itertools.combinations(cand, k)), default=0.0)
    assert sum(s[j] for j in got) == best
    minimal = [list(c) for c in itertools.combinations(cand, k) if sum(s[j] for j in c) == best]
    assert got == min(minimal)
    # lowest-first on s equals highest-first on -s
    assert got == select.select_topk(-s, excl, k)


def test_lowest_first_nan_last():
    s = np.array([0.3, np.nan, 0.1, 0.2])
    assert select.select_topk(s, [], 3, lowest=True) == [0, 2, 3]
    assert select.select_topk(s, [], 4, lowest=True) == [0, 1, 2, 3]
