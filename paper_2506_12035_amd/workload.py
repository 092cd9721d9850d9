"""Seeded synthetic MAR-shaped workloads.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no layer norm, projection, attention, selection or mask
schedule).  Both the HIP path and the fp64 oracle take their inputs from here,
so the two sides see identical values.

The paper measures class-conditional ImageNet 256x256 generation with trained
MAR-B/L/H weights (Section 5.1).  Neither the dataset nor the weights exist
here, so seeded tensors with the same shapes stand in for them:

* token layout: ``n_buf`` buffer tokens at indices ``[0, n_buf)`` followed by
  the image tokens ``[n_buf, N)`` (16x16 = 256 image tokens, or 32x32 = 1024
  for the high-resolution stress shape);
* linear weights and biases ~ N(0, 0.02^2); LayerNorm gamma = 1 + N(0, 0.02^2),
  beta ~ N(0, 0.02^2); all rounded once to the storage dtype;
* embeddings (class embedding per image, one "generated value" embedding per
  image token, the mask embedding and the positional embedding) ~ N(0, 1);
* a random generation order per image (Section 3, the permutation pi).

Random streams: ``SeedSequence(seed)`` is spawned into four children
(weights, state, orders, planted); the weights child is spawned again, once per
layer, so any single layer can be regenerated without the others.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Dict, List, Optional

import numpy as np

SEED_BASE = 2506120350

STREAM_WEIGHTS, STREAM_STATE, STREAM_ORDERS, STREAM_PLANTED = range(4)

LAYER_PARAM_NAMES = (
    "ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
    "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2",
)


@dataclass(frozen=True)
class Config:
    """Shape and policy of one synthetic workload."""

    cid: int
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_mlp: int
    n_tokens: int
    n_buf: int
    batch: int
    dtype: str                 # storage / compute dtype of the path: "f32" or "bf16"
    n_steps: int = 64          # decoding steps of the mask schedule
    ratio_bp: int = 1000       # refresh budget: basis points of the candidate tokens
    sel_layer: int = 2         # 1-based layer whose attention feeds the refresh selection
    full_every: int = 3        # periodic full refresh period (0 = only the first step)
    ln_eps: float = 1e-6
    weight_std: float = 0.02
    seed: Optional[int] = None

    @property
    def n_img(self) -> int:
        return self.n_tokens - self.n_buf

    @property
    def seed_value(self) -> int:
        return SEED_BASE + self.cid if self.seed is None else self.seed

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)


# The five workload shapes.  Id 1 is the single-block fp32 case, ids 2-4 are
# MAR-B/L/H-shaped decoder stacks (the model scales of Table 1), id 5 is a
# 32x32-token high-resolution stress shape with long KV.
CONFIGS: Dict[int, Config] = {
    1: Config(1, "single-block-d768-fp32", 1, 768, 12, 64, 3072, 320, 64, 1, "f32",
              n_steps=1, ratio_bp=0, sel_layer=1, full_every=0),
    2: Config(2, "mar-b-d768-L24-B64", 24, 768, 12, 64, 3072, 320, 64, 64, "bf16"),
    3: Config(3, "mar-l-d1024-L32-B128", 32, 1024, 16, 64, 4096, 320, 64, 128, "bf16"),
    4: Config(4, "mar-h-d1280-L40-B256", 40, 1280, 16, 80, 5120, 320, 64, 256, "bf16"),
    5: Config(5, "hires-d1024-L32-N1088-B32", 32, 1024, 16, 64, 4096, 1088, 64, 32, "bf16"),
}

# Refresh ratios swept on the MAR-H shape (basis points; 10000 = full recompute).
MAR_H_RATIO_SWEEP_BP = (0, 500, 1000, 2500, 10000)


def streams(seed: int) -> List[np.random.Generator]:
    """The four child generators (weights, state, orders, planted)."""
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(4)]


def round_to(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 values once to the storage dtype (RNE), returned as float32.

    For "bf16" every returned value is exactly representable in bfloat16, so
    the GPU side converts it to bf16 exactly and the oracle to float64 exactly.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "f32":
        return a
    if dtype != "bf16":
        raise ValueError(f"unknown dtype {dtype!r}")
    u = a.view(np.uint32).astype(np.uint64)
    nan = np.isnan(a)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32).copy()
    out[nan] = np.nan
    return out


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    return rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std)


def layer_weights(cfg: Config, layer: int) -> Dict[str, np.ndarray]:
    """Parameters of one block, in torch ``nn.Linear`` layout ``[out][in]``.

    ``w_qkv`` is ``[3D][D]``: rows ``[0, D)`` project queries, ``[D, 2D)`` keys
    and ``[2D, 3D)`` values; inside each third, head ``h`` owns rows
    ``[h*d_h, (h+1)*d_h)``.
    """
    if not 0 <= layer < cfg.n_layers:
        raise IndexError(layer)
    root = np.random.SeedSequence(cfg.seed_value).spawn(4)[STREAM_WEIGHTS]
    ss = root.spawn(cfg.n_layers)[layer]
    rng = np.random.Generator(np.random.PCG64(ss))
    D, F, s = cfg.d_model, cfg.d_mlp, cfg.weight_std
    p = {
        "ln1_g": 1.0 + _normal(rng, (D,), s),
        "ln1_b": _normal(rng, (D,), s),
        "w_qkv": _normal(rng, (3 * D, D), s),
        "b_qkv": _normal(rng, (3 * D,), s),
        "w_o": _normal(rng, (D, D), s),
        "b_o": _normal(rng, (D,), s),
        "ln2_g": 1.0 + _normal(rng, (D,), s),
        "ln2_b": _normal(rng, (D,), s),
        "w_1": _normal(rng, (F, D), s),
        "b_1": _normal(rng, (F,), s),
        "w_2": _normal(rng, (D, F), s),
        "b_2": _normal(rng, (D,), s),
    }
    return {k: round_to(v, cfg.dtype) for k, v in p.items()}


def all_weights(cfg: Config) -> List[Dict[str, np.ndarray]]:
    return [layer_weights(cfg, l) for l in range(cfg.n_layers)]


@dataclass
class Embeddings:
    """Synthetic decoder-input embeddings (stand-in for Eq. 1-2's encoder output).

    ``cls``   [B][D]      class embedding per image, used at the buffer tokens;
    ``value`` [B][N_img][D] embedding of an image token once it is generated;
    ``mask``  [D]         the mask embedding;
    ``pos``   [N][D]      positional embedding.
    """

    cls: np.ndarray
    value: np.ndarray
    mask: np.ndarray
    pos: np.ndarray


def _image_range(cfg: Config, batch: Optional[int], first: int) -> slice:
    B = cfg.batch if batch is None else batch
    if first < 0 or B < 0 or first + B > cfg.batch:
        raise ValueError(f"images [{first}, {first + B}) outside the workload's {cfg.batch}")
    return slice(first, first + B)


def embeddings(cfg: Config, batch: Optional[int] = None, first: int = 0) -> Embeddings:
    """Images ``first .. first + batch - 1`` of the workload's batch."""
    sl = _image_range(cfg, batch, first)
    rng = streams(cfg.seed_value)[STREAM_STATE]
    D = cfg.d_model
    cls = rng.standard_normal((cfg.batch, D), dtype=np.float32)[sl]
    value = rng.standard_normal((cfg.batch, cfg.n_img, D), dtype=np.float32)[sl]
    mask = rng.standard_normal((D,), dtype=np.float32)
    pos = rng.standard_normal((cfg.n_tokens, D), dtype=np.float32)
    return Embeddings(np.ascontiguousarray(cls), np.ascontiguousarray(value), mask, pos)


def orders(cfg: Config, batch: Optional[int] = None, first: int = 0) -> np.ndarray:
    """Generation order per image: ``[B][N_img]``, a permutation of ``0..N_img-1``
    (image-local positions; token index = ``n_buf + position``), for images
    ``first .. first + batch - 1`` of the workload's batch."""
    sl = _image_range(cfg, batch, first)
    rng = streams(cfg.seed_value)[STREAM_ORDERS]
    out = np.empty((cfg.batch, cfg.n_img), dtype=np.int32)
    for b in range(cfg.batch):
        out[b] = rng.permutation(cfg.n_img)
    return out[sl].copy()


@dataclass
class SingleBlockCase:
    """Inputs of the single-block case: one cache-aware layer plus top-k.

    ``x`` [B][N][D], ``k_cache``/``v_cache`` [B][H][N][d_h] (all float32 values
    rounded to ``cfg.dtype``), ``active`` [B][n_a] int32 with the ``n_gen``
    generating tokens first, ``k_top`` the refresh-set size.
    """

    x: np.ndarray
    k_cache: np.ndarray
    v_cache: np.ndarray
    active: np.ndarray
    n_gen: int
    k_top: int


def single_block_case(cfg: Config, n_gen: int = 16, n_ref: int = 16, k_top: int = 16,
                      batch: Optional[int] = None) -> SingleBlockCase:
    """x and cached K/V ~ N(0, 1); generating tokens drawn without replacement
    from the image tokens, refresh tokens from the remaining tokens."""
    B = cfg.batch if batch is None else batch
    rng = streams(cfg.seed_value)[STREAM_STATE]
    N, D, H, dh = cfg.n_tokens, cfg.d_model, cfg.n_heads, cfg.head_dim
    x = rng.standard_normal((B, N, D), dtype=np.float32)
    kc = round_to(rng.standard_normal((B, H, N, dh), dtype=np.float32), cfg.dtype)
    vc = round_to(rng.standard_normal((B, H, N, dh), dtype=np.float32), cfg.dtype)
    act = np.empty((B, n_gen + n_ref), dtype=np.int32)
    for b in range(B):
        g = rng.choice(np.arange(cfg.n_buf, N), size=n_gen, replace=False)
        rest = np.setdiff1d(np.arange(N), g)
        r = rng.choice(rest, size=n_ref, replace=False)
        act[b, :n_gen] = g
        act[b, n_gen:] = r
    return SingleBlockCase(x, kc, vc, act, n_gen, k_top)


def planted_rows(cfg: Config, candidates: np.ndarray, k: int, batch: Optional[int] = None) -> np.ndarray:
    """Seeded choice of ``k`` candidate tokens per image for planted-structure
    variants (the caller decides how to make them stand out)."""
    B = cfg.batch if batch is None else batch
    rng = streams(cfg.seed_value)[STREAM_PLANTED]
    out = np.empty((B, k), dtype=np.int32)
    for b in range(B):
        c = candidates[b] if candidates.ndim == 2 else candidates
        out[b] = np.sort(rng.choice(c, size=k, replace=False))
    return out


def planted_stack_draw(cfg: Config, t: int, image: int, candidates: np.ndarray, k: int):
    """Seeded draw of a planted-structure stack case for step ``t`` of one
    image: ``k`` of the image's candidate tokens (ascending) and an anchor row
    ~ N(0, 1) of width d_model.  The caller turns these into the rows it
    plants; the generator depends only on (seed, step, image)."""
    ss = np.random.SeedSequence([cfg.seed_value, STREAM_PLANTED, 7000 + t, image])
    rng = np.random.Generator(np.random.PCG64(ss))
    rows = np.sort(rng.choice(np.asarray(candidates), size=k, replace=False)).astype(np.int32)
    anchor = rng.standard_normal(cfg.d_model, dtype=np.float32)
    return rows, anchor


def random_refresh(cfg: Config, t: int, candidates: np.ndarray, k: int,
                   first: int = 0) -> np.ndarray:
    """Seeded random refresh set of step ``t`` for the random-refresh ablation:
    ``candidates`` is [B][n_cand] per image (images ``first`` ..); returns
    [B][k] (ascending), drawn without replacement from each image's
    candidates with a generator of its own (seeded by step and image), so an
    image's draw does not depend on which other images share the call."""
    out = np.empty((candidates.shape[0], k), dtype=np.int32)
    for b in range(candidates.shape[0]):
        ss = np.random.SeedSequence([cfg.seed_value, STREAM_PLANTED, 1 + t, first + b])
        rng = np.random.Generator(np.random.PCG64(ss))
        out[b] = np.sort(rng.choice(candidates[b], size=k, replace=False))
    return out


@dataclass
class SegmentCase:
    """Inputs of the two-segment attention comparison (Appendix B): queries of
    the active rows and the keys/values of the active and cached segments.

    ``q`` [B][n_active][H*d_h]; ``k_a``/``v_a`` [B][H][n_active][d_h];
    ``k_c``/``v_c`` [B][H][n_cached][d_h]; all ~ N(0, 1) rounded to bf16.
    """

    q: np.ndarray
    k_a: np.ndarray
    v_a: np.ndarray
    k_c: np.ndarray
    v_c: np.ndarray


def segment_case(batch: int, n_heads: int, head_dim: int, n_active: int, n_cached: int,
                 seed: int = SEED_BASE + 100) -> SegmentCase:
    rng = streams(seed)[STREAM_STATE]
    D = n_heads * head_dim

    def draw(*shape):
        return round_to(rng.standard_normal(shape, dtype=np.float32), "bf16")

    return SegmentCase(draw(batch, n_active, D), draw(batch, n_heads, n_active, head_dim),
                       draw(batch, n_heads, n_active, head_dim),
                       draw(batch, n_heads, n_cached, head_dim),
                       draw(batch, n_heads, n_cached, head_dim))


# ------------------------------------------------------------------ the rest of a MAR step

@dataclass(frozen=True)
class MarConfig:
    """A whole MAR model around the cache-aware decoder (latency workloads):
    the encoder stack over the known tokens (Eq. 1), the decoder stack
    ``dec`` (Eq. 2, the cache-aware step), and the sampler head of Eq. 3
    (``head_blocks`` modulated residual MLP blocks of width ``head_width`` over
    ``c_tok``-channel token values, ``sample_steps`` DDPM steps)."""

    name: str
    dec: Config
    enc_layers: int
    head_width: int
    head_blocks: int
    c_tok: int = 16
    t_freq: int = 256
    sample_steps: int = 100
    temperature: float = 1.0
    head_eps: float = 1e-6
    head_std: float = 0.02

    @property
    def enc(self) -> Config:
        """The encoder stack: the decoder's block shape, its own depth and weights."""
        return self.dec.with_(n_layers=self.enc_layers, seed=self.dec.seed_value + 7919)


# MAR-L end to end (the scales the paper adopts from MAR: 16 encoder and 16
# decoder blocks of width 1024, a head of 8 blocks of width 1280, 16-channel
# tokens, 100 sampling steps), and a tiny case for parity tests.
MAR_CONFIGS: Dict[str, MarConfig] = {
    "mar-l-e2e": MarConfig("mar-l-e2e-enc16-dec16-head8x1280-B128",
                           CONFIGS[3].with_(n_layers=16, name="mar-l-dec16-B128"),
                           enc_layers=16, head_width=1280, head_blocks=8),
    "tiny": MarConfig("tiny-e2e", Config(90, "tiny-dec", 2, 256, 4, 64, 1024, 36, 4, 3, "bf16",
                                         n_steps=6),
                      enc_layers=2, head_width=256, head_blocks=2, sample_steps=8,
                      head_std=0.08),
}


def mar_embeddings(mc: MarConfig, batch: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Embeddings and the two LayerNorms around the stacks (float32; ``w_de``
    rounded to the model dtype): cls [B][D], w_z [D][C], b_z [D], pe_enc and
    pe_dec [N][D], enc_ln_g/b, w_de [D][D], b_de, mask [D], dec_ln_g/b,
    pe_diff [N_img][D]."""
    cfg = mc.dec
    B = cfg.batch if batch is None else batch
    ss = np.random.SeedSequence([cfg.seed_value, 31])
    rng = np.random.Generator(np.random.PCG64(ss))
    D, N, C = cfg.d_model, cfg.n_tokens, mc.c_tok
    s = cfg.weight_std
    out = {
        "cls": rng.standard_normal((cfg.batch, D), dtype=np.float32)[:B].copy(),
        "w_z": _normal(rng, (D, C), 0.25),
        "b_z": _normal(rng, (D,), s),
        "pe_enc": rng.standard_normal((N, D), dtype=np.float32),
        "enc_ln_g": 1.0 + _normal(rng, (D,), s),
        "enc_ln_b": _normal(rng, (D,), s),
        "w_de": round_to(_normal(rng, (D, D), s), cfg.dtype),
        "b_de": _normal(rng, (D,), s),
        "mask": rng.standard_normal((D,), dtype=np.float32),
        "pe_dec": rng.standard_normal((N, D), dtype=np.float32),
        "dec_ln_g": 1.0 + _normal(rng, (D,), s),
        "dec_ln_b": _normal(rng, (D,), s),
        "pe_diff": rng.standard_normal((cfg.n_img, D), dtype=np.float32),
    }
    return out


def head_weights(mc: MarConfig) -> Dict[str, np.ndarray]:
    """Sampler head parameters (nn.Linear layout): the GEMM weights w_t1, w_t2,
    w_c, w_ada [(3n+2)W][W], w_1 and w_2 [n][W][W] rounded to the model dtype;
    w_in [W][C], w_out [C][W] and all biases float32."""
    cfg = mc.dec
    ss = np.random.SeedSequence([cfg.seed_value, 37])
    rng = np.random.Generator(np.random.PCG64(ss))
    W, n, C, D, Ft, s = mc.head_width, mc.head_blocks, mc.c_tok, cfg.d_model, mc.t_freq, mc.head_std
    r = lambda a: round_to(a, cfg.dtype)
    return {
        "w_t1": r(_normal(rng, (W, Ft), s)), "b_t1": _normal(rng, (W,), s),
        "w_t2": r(_normal(rng, (W, W), s)), "b_t2": _normal(rng, (W,), s),
        "w_c": r(_normal(rng, (W, D), s)), "b_c": _normal(rng, (W,), s),
        "w_in": _normal(rng, (W, C), 0.25), "b_in": _normal(rng, (W,), s),
        "w_ada": r(_normal(rng, ((3 * n + 2) * W, W), s)), "b_ada": _normal(rng, ((3 * n + 2) * W,), s),
        "w_1": r(_normal(rng, (n, W, W), s)), "b_1": _normal(rng, (n, W), s),
        "w_2": r(_normal(rng, (n, W, W), s)), "b_2": _normal(rng, (n, W), s),
        "w_out": _normal(rng, (C, W), s), "b_out": _normal(rng, (C,), s),
    }


def head_noise(mc: MarConfig, t: int, n_rows: int) -> np.ndarray:
    """The sampler's draws for decoding step ``t``: [sample_steps + 1][n_rows][C]
    standard normal (index sample_steps is the initial x, index i the noise of
    sampling step i)."""
    ss = np.random.SeedSequence([mc.dec.seed_value, 41, t])
    rng = np.random.Generator(np.random.PCG64(ss))
    return rng.standard_normal((mc.sample_steps + 1, n_rows, mc.c_tok), dtype=np.float32)
