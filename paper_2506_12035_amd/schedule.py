"""Host-side decoding schedule of the driver (index bookkeeping only).

Section 3 (Eq. 1-4): positions are generated in a random order; each step
takes the next block of still-masked positions.  The block sizes follow a
cosine curve of the number of masked image tokens over T steps:
    m_0 = N_img,  m_{t+1} = max(1, min(m_t - 1, floor(N_img cos(pi (t+1) / (2T))))),  m_T = 0.
Section 4.3: the caching tokens of step t are those generated at step t-1;
the first step and every ``full_every``-th step run every layer with full
attention; the refresh count fills either a fixed active budget or a ratio of
the candidate tokens (rounded half up).
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List

import numpy as np


def masked_counts(n_img: int, n_steps: int) -> List[int]:
    out = [n_img]
    for t in range(1, n_steps):
        target = int(math.floor(n_img * math.cos(math.pi * t / (2.0 * n_steps))))
        out.append(max(1, min(out[-1] - 1, target)))
    out.append(0)
    return out


def full_step(t: int, full_every: int) -> bool:
    return t == 0 or (full_every > 0 and t % full_every == 0)


def check_budget(policy: str, value: int, n_tokens: int) -> None:
    """Reject budgets whose refresh count could exceed the candidates: a ratio
    outside [0, 10000] basis points, or a fixed active-set size outside
    [0, n_tokens].  The device selection would otherwise pad the active list
    with -1 entries, which the step would index the cache and x with."""
    if policy == "ratio":
        if not 0 <= value <= 10000:
            raise ValueError(f"refresh ratio {value} bp outside [0, 10000]")
    elif policy == "fixed":
        if not 0 <= value <= n_tokens:
            raise ValueError(f"fixed active budget {value} outside [0, n_tokens={n_tokens}]")
    else:
        raise ValueError(f"unknown budget policy {policy!r}")


def refresh_count(policy: str, value: int, n_tokens: int, n_gen: int, n_cache: int) -> int:
    if policy == "fixed":
        return max(0, value - n_gen - n_cache)
    if policy == "ratio":
        cand = n_tokens - n_gen - n_cache
        return (value * cand + 5000) // 10000
    raise ValueError(f"unknown budget policy {policy!r}")


@dataclass
class StepIndices:
    """Host index lists of one step for a batch of images (int32 arrays).

    ``gen`` [B][g] generating tokens, ``cache`` [B][n] caching tokens,
    ``full_order`` [B][N] every token with the generating ones first (the
    active list of full-attention layers), ``n_known`` image tokens generated
    before the step, ``k`` refresh count, ``full`` whether every layer is full.
    """

    t: int
    full: bool
    n_known: int
    k: int
    gen: np.ndarray
    cache: np.ndarray
    full_order: np.ndarray


def step_indices(orders: np.ndarray, n_buf: int, n_tokens: int, n_steps: int, t: int,
                 full_every: int, policy: str, budget: int) -> StepIndices:
    B, n_img = orders.shape
    m = masked_counts(n_img, n_steps)
    lo, hi = n_img - m[t], n_img - m[t + 1]
    gen = (orders[:, lo:hi] + n_buf).astype(np.int32)
    if t > 0:
        plo, phi = n_img - m[t - 1], n_img - m[t]
        cache = (orders[:, plo:phi] + n_buf).astype(np.int32)
    else:
        cache = np.zeros((B, 0), np.int32)
    full_order = np.empty((B, n_tokens), np.int32)
    for b in range(B):
        mark = np.zeros(n_tokens, bool)
        mark[gen[b]] = True
        full_order[b, :gen.shape[1]] = gen[b]
        full_order[b, gen.shape[1]:] = np.flatnonzero(~mark)
    k = refresh_count(policy, budget, n_tokens, gen.shape[1], cache.shape[1])
    return StepIndices(t, full_step(t, full_every), lo, k, gen, cache, full_order)
