"""fp64 oracle of the decoding schedule (test infrastructure).

Section 3 (Eq. 1-4): positions are generated in a random order pi; at each
step a subset of the still-masked positions is predicted and leaves the masked
set, until none is left after T steps.  Section 4.3: the caching tokens of a
step are the tokens generated in the step before it; a step runs every layer
with full attention when it is the first step or when the periodic full
refresh falls on it (every third step).

The paper uses the default MAR schedule of 64 steps without stating its
formula.  Reading used here: a cosine schedule of the number of still-masked
image tokens,
    m_0 = N_img,  m_{t+1} = max(1, min(m_t - 1, floor(N_img cos(pi (t+1) / (2T))))),
    m_T = 0,
so step t generates the order positions [N_img - m_t, N_img - m_{t+1}).
Image tokens occupy token indices [n_buf, N); buffer tokens are never
generated.

Pins (tests/test_oracle_schedule.py): the counts partition N_img, every step
generates at least one token, the sets are disjoint and cover every image
token, golden count sequences under tests/golden/.
"""
from __future__ import annotations

import math
from typing import List

import numpy as np


def masked_counts(n_img: int, n_steps: int) -> List[int]:
    """m_0 .. m_T: how many image tokens are still masked before each step."""
    m = [n_img]
    for t in range(n_steps - 1):
        c = math.floor(n_img * math.cos(math.pi * (t + 1) / (2 * n_steps)))
        m.append(max(1, min(m[-1] - 1, c)))
    m.append(0)
    return m


def generated_counts(n_img: int, n_steps: int) -> List[int]:
    m = masked_counts(n_img, n_steps)
    return [m[t] - m[t + 1] for t in range(n_steps)]


def generating_tokens(order: np.ndarray, n_buf: int, n_steps: int, t: int) -> List[int]:
    """G^(t) of one image: token indices generated at step t (in order position)."""
    n_img = len(order)
    m = masked_counts(n_img, n_steps)
    lo, hi = n_img - m[t], n_img - m[t + 1]
    return [n_buf + int(order[r]) for r in range(lo, hi)]


def caching_tokens(order: np.ndarray, n_buf: int, n_steps: int, t: int) -> List[int]:
    """N^(t): the tokens generated at the previous step (none at step 0)."""
    return [] if t == 0 else generating_tokens(order, n_buf, n_steps, t - 1)


def known_before(order: np.ndarray, n_buf: int, n_steps: int, t: int) -> List[int]:
    """Image tokens generated before step t (the complement of M^(t))."""
    n_img = len(order)
    m = masked_counts(n_img, n_steps)
    return [n_buf + int(order[r]) for r in range(0, n_img - m[t])]


def is_full_step(t: int, full_every: int) -> bool:
    """Full attention in every layer on the first step and every full_every-th
    step (full_every = 0 disables the periodic refresh)."""
    return t == 0 or (full_every > 0 and t % full_every == 0)
