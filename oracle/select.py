"""fp64 oracle of refresh selection and the active-token budget (test infrastructure).

Section 4.2: the tokens with the highest relevance (the attention mass the
generating tokens put on them, summed over heads) become the refreshing
tokens.  Section 4.3: the refresh count fills a fixed active-token budget
(64 in the paper: 5 generating + 9 caching leaves 50 refresh tokens).

Readings where the paper is silent: the candidates are all tokens except the
generating and caching ones (buffer tokens included); equal scores go to the
lower token index; NaN ranks as -inf; the chosen set is returned in ascending
token order.  The ratio budget (a fraction of the candidates, in basis points,
rounded half up) is the workload's alternative to the fixed budget; 100% makes
every token active.

The low-attention selection (lowest scores first) is the refresh-strategy
ablation of Table 3.

Pins (tests/test_oracle_select.py): brute-force rank definition and exhaustive
subset enumeration on tiny inputs (both orders); the paper's 5 + 9 + 50 = 64
example.
"""
from __future__ import annotations

from typing import Iterable, List, Sequence

import numpy as np


def total_scores(scores_per_head: np.ndarray) -> np.ndarray:
    """Aggregate over heads: s_j = sum_h S_h[j] (Section 4.2)."""
    return np.asarray(scores_per_head, np.float64).sum(axis=0)


def _rank_key(s: float, lowest: bool = False) -> float:
    """Preference value: larger is preferred.  NaN is never preferred."""
    if np.isnan(s):
        return -np.inf
    return -float(s) if lowest else float(s)


def select_topk(scores: Sequence[float], excl: Iterable[int], k: int,
                lowest: bool = False) -> List[int]:
    """The k candidates with the highest score (or, with ``lowest``, the lowest:
    the low-attention ablation of Table 3); ties to the lower index; returned
    ascending.  Fewer than k candidates is an error."""
    excl = set(int(e) for e in excl)
    cand = [j for j in range(len(scores)) if j not in excl]
    if k > len(cand):
        raise ValueError("k exceeds the number of candidates")
    ranked = sorted(cand, key=lambda j: (-_rank_key(scores[j], lowest), j))
    return sorted(ranked[:k])


def select_topk_bruteforce(scores: Sequence[float], excl: Iterable[int], k: int,
                           lowest: bool = False) -> List[int]:
    """Rank definition: candidate j is chosen iff fewer than k candidates beat
    it, where l beats j when l is preferred (higher score, or lower with
    ``lowest``), or equally preferred and l < j."""
    excl = set(int(e) for e in excl)
    cand = [j for j in range(len(scores)) if j not in excl]
    out = []
    for j in cand:
        sj = _rank_key(scores[j], lowest)
        beaten_by = 0
        for l in cand:
            sl = _rank_key(scores[l], lowest)
            if sl > sj or (sl == sj and l < j):
                beaten_by += 1
        if beaten_by < k:
            out.append(j)
    return out


def budget_fixed(n_active: int, n_gen: int, n_cache: int) -> int:
    """Refresh count that fills a fixed active budget (Section 4.3)."""
    return max(0, n_active - n_gen - n_cache)


def budget_ratio(ratio_bp: int, n_tokens: int, n_gen: int, n_cache: int) -> int:
    """Refresh count as a fraction of the candidates, rounded half up:
    round(ratio * (N - |G| - |N|)) computed exactly in integers."""
    n_cand = n_tokens - n_gen - n_cache
    return (ratio_bp * n_cand + 5000) // 10000
