"""fp64 oracle of one MARche decoding step over a stack of blocks (test infrastructure).

Per image (images never interact):

* a full step (the first step, and every periodic full refresh, Section 4.3)
  runs every layer with all tokens active;
* any other step runs the layers up to and including the selection layer
  with full attention (Section 4.2: the active set is not known yet there),
  sums the attention mass the generating tokens put on every key at the
  selection layer, picks the refreshing tokens R by top-k over the tokens
  that are neither generating nor caching, and runs every later layer the
  cache-aware way with A = G u N u R (Algorithm 1).

The step's output is the residual stream after the last layer at the
generating tokens: the context vectors z^(t) that Eq. 3's sampler consumes.
The synthetic decoder input stands in for Eq. 2's concatenation of encoder
features and mask embeddings: buffer tokens carry the image's class
embedding, already-generated image tokens their value embedding, masked
tokens the mask embedding; every token adds its positional embedding.

Pins (tests/test_oracle_step.py): at a 100% refresh ratio the step equals
full recomputation bit for bit; at 0% the active set is G u N; a full step
equals the stack of full layers.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from . import block, schedule, select

F64 = np.float64


def decoder_input(cls_emb: np.ndarray, value_emb: np.ndarray, mask_emb: np.ndarray,
                  pos_emb: np.ndarray, known: Sequence[int], n_buf: int) -> np.ndarray:
    """x_in [N][D] of one image (stand-in for Eq. 2's decoder input)."""
    pos = np.asarray(pos_emb, F64)
    N = pos.shape[0]
    x = np.empty_like(pos)
    known = set(int(j) for j in known)
    for j in range(N):
        if j < n_buf:
            base = np.asarray(cls_emb, F64)
        elif j in known:
            base = np.asarray(value_emb[j - n_buf], F64)
        else:
            base = np.asarray(mask_emb, F64)
        x[j] = base + pos[j]
    return x


@dataclass
class StepResult:
    x_out: np.ndarray
    k_caches: List[np.ndarray]
    v_caches: List[np.ndarray]
    gen: List[int]
    cache_tokens: List[int]
    refresh: Optional[List[int]]
    full: bool
    scores: Optional[np.ndarray] = None          # [H][N] at the selection layer
    layers: List[block.LayerResult] = field(default_factory=list)
    include_gen: bool = True                     # G part of the cache-aware active set

    @property
    def z(self) -> np.ndarray:
        return self.x_out[np.array(self.gen, dtype=np.int64)]

    @property
    def active(self) -> Optional[List[int]]:
        if self.refresh is None:
            return None
        g = list(self.gen) if self.include_gen else []
        return g + list(self.cache_tokens) + list(self.refresh)


def marche_step(params: Sequence[Dict[str, np.ndarray]], x_in: np.ndarray,
                k_caches: Sequence[np.ndarray], v_caches: Sequence[np.ndarray],
                gen: Sequence[int], cache_tokens: Sequence[int], *, n_heads: int,
                eps: float, sel_layer: int, full: bool, k_refresh: int,
                keep_layers: bool = False,
                refresh_override: Optional[Callable[[np.ndarray, List[int]], List[int]]] = None,
                layer_range: Optional[range] = None, select_lowest: bool = False,
                include_gen: bool = True) -> StepResult:
    """One decoding step of one image.

    ``sel_layer`` is 1-based; layers 1..sel_layer run with full attention in
    every step.  ``refresh_override`` (used by parity tests and by the random
    refresh ablation) receives the selection-layer scores and the oracle's own
    refresh set and returns the set to continue with.  ``layer_range``
    restricts the layers run (0-based).

    Ablations of the active-set construction (Tables 2-3): ``select_lowest``
    refreshes the tokens with the lowest attention mass; passing no caching
    tokens gives A = G u R; ``include_gen=False`` leaves the generating tokens
    out of the active set (A = N u R; they are still excluded from R and still
    provide the scores).
    """
    L = len(params)
    x = np.asarray(x_in, F64)
    kcs = [np.asarray(c, F64) for c in k_caches]
    vcs = [np.asarray(c, F64) for c in v_caches]
    gen = [int(g) for g in gen]
    cache_tokens = [int(c) for c in cache_tokens]
    N = x.shape[0]
    lr = range(L) if layer_range is None else layer_range

    refresh: Optional[List[int]] = None
    scores = None
    layers: List[block.LayerResult] = []
    active: Optional[List[int]] = None
    for l in lr:
        is_full_layer = full or l < sel_layer
        if is_full_layer:
            want_score = (not full) and l == sel_layer - 1
            res = block.full_layer(params[l], x, kcs[l], vcs[l], gen, n_heads, eps, score=want_score)
            if want_score:
                scores = res.scores
                refresh = select.select_topk(select.total_scores(scores), gen + cache_tokens,
                                             k_refresh, lowest=select_lowest)
                if refresh_override is not None:
                    refresh = list(refresh_override(scores, refresh))
                active = (gen if include_gen else []) + cache_tokens + refresh
        else:
            if active is None:
                raise ValueError("cache-aware layer reached before the selection layer")
            res = block.cache_aware_layer(params[l], x, kcs[l], vcs[l], active,
                                          gen if include_gen else [], n_heads, eps)
        x = res.x_out
        kcs[l], vcs[l] = res.k_cache, res.v_cache
        if keep_layers:
            layers.append(res)
    return StepResult(x, kcs, vcs, gen, cache_tokens, refresh, full, scores, layers, include_gen)


def refresh_count(policy: str, value: int, n_tokens: int, n_gen: int, n_cache: int) -> int:
    """``policy`` "ratio" (value in basis points) or "fixed" (value = active budget)."""
    if policy == "ratio":
        return select.budget_ratio(value, n_tokens, n_gen, n_cache)
    if policy == "fixed":
        return select.budget_fixed(value, n_gen, n_cache)
    raise ValueError(policy)


def run_generation(params: Sequence[Dict[str, np.ndarray]], cls_emb, value_emb, mask_emb, pos_emb,
                   order: np.ndarray, *, n_buf: int, n_steps: int, n_heads: int, eps: float,
                   sel_layer: int, full_every: int, policy: str = "ratio", budget: int = 1000,
                   steps: Optional[Sequence[int]] = None) -> List[StepResult]:
    """All decoding steps of one image from zero-filled caches (every cache row
    is written by the first, full, step before any read)."""
    N, D = np.asarray(pos_emb).shape
    H = n_heads
    dh = D // H
    kcs = [np.zeros((H, N, dh)) for _ in params]
    vcs = [np.zeros((H, N, dh)) for _ in params]
    out = []
    for t in range(n_steps):
        gen = schedule.generating_tokens(order, n_buf, n_steps, t)
        cache_toks = schedule.caching_tokens(order, n_buf, n_steps, t)
        known = schedule.known_before(order, n_buf, n_steps, t)
        x_in = decoder_input(cls_emb, value_emb, mask_emb, pos_emb, known, n_buf)
        full = schedule.is_full_step(t, full_every)
        k = refresh_count(policy, budget, N, len(gen), len(cache_toks))
        res = marche_step(params, x_in, kcs, vcs, gen, cache_toks, n_heads=H, eps=eps,
                          sel_layer=sel_layer, full=full, k_refresh=k)
        kcs, vcs = res.k_caches, res.v_caches
        if steps is None or t in steps:
            out.append(res)
    return out
