"""fp64 oracle of the rest of a MAR step around the decoder (test infrastructure).

The decoder step of ``step`` consumes Eq. 2's decoder input and produces the
context vectors z of Eq. 3.  This module holds the parts around it, per image
(or per row where rows are independent), in plain float64 numpy:

* ``encoder_input`` -- Eq. 1's input: the known tokens x_i + PE_i.  Known
  tokens enter through a linear token embedding; the n_buf buffer rows carry
  the image's class embedding (reading: MAR's buffer tokens).  Buffer rows
  come first, then the known tokens in the order given.
* ``encoder``       -- f_enc: a stack of full pre-LN blocks (``block.full_layer``)
  over those rows only.
* ``encoder_to_decoder`` -- Eq. 2: the encoder output after its final LayerNorm
  and a linear decoder embedding is put back at its positions; every masked
  position takes the mask embedding; all add the decoder's positional
  embedding.
* ``decoder_cond``  -- the condition of Eq. 3 for each generating token: the
  decoder output after a final LayerNorm plus a per-position embedding.
* ``denoiser`` / ``sample`` -- Eq. 3's sampler p_theta(x_i | z_i; tau).  The
  paper fixes only its inputs and the temperature.  Reading (the MAR head the
  paper adopts): a residual MLP over the token value whose every block is
  modulated (shift, scale, gate) by a condition c = time embedding + a linear
  map of z; DDPM ancestral sampling over T steps of a cosine noise schedule
  with the fixed posterior variance, tau scaling the injected noise, no
  guidance.  All random draws are inputs (``noise``).

Parity status: every function here is pinned (tests/test_oracle_mar.py):
library special cases of the denoiser (zero and unit modulation reduce to
torch's LayerNorm / Linear / SiLU), closed-form values of the time embedding,
the DDPM posterior mean in two independent forms and the posterior variance
from Gaussian conditioning, recovery of x0 from the true noise, permutation
equivariance of the encoder over the known tokens, and the row bookkeeping of
the decoder input.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Sequence

import numpy as np

from . import block

F64 = np.float64


def _f(a) -> np.ndarray:
    return np.asarray(a, F64)


def silu(z: np.ndarray) -> np.ndarray:
    """z * sigmoid(z)."""
    z = _f(z)
    return z / (1.0 + np.exp(-z))


def layer_norm_plain(x: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm without affine parameters (population variance, eps inside the root)."""
    x = _f(x)
    return block.layer_norm(x, np.ones(x.shape[-1]), np.zeros(x.shape[-1]), eps)


# ------------------------------------------------------------------ Eq. 1 and 2

def encoder_input(cls_emb, tok, w_z, b_z, pe_enc, known: Sequence[int], n_buf: int) -> np.ndarray:
    """Rows of f_enc's input for one image (Eq. 1).

    ``tok`` [n_img][C] token values, ``w_z`` [D][C] / ``b_z`` [D] the token
    embedding, ``pe_enc`` [N][D] positional embeddings indexed by sequence
    position (buffer rows 0..n_buf-1, image token p at n_buf + p), ``known``
    the sequence positions of the known tokens in the order they take as rows.
    Returns [n_buf + len(known)][D]."""
    pe = _f(pe_enc)
    rows = [ _f(cls_emb) + pe[j] for j in range(n_buf) ]
    for j in known:
        rows.append(block.linear(_f(tok)[j - n_buf], w_z, b_z) + pe[j])
    return np.stack(rows) if rows else np.zeros((0, pe.shape[1]))


def encoder(e: np.ndarray, params: Sequence[Dict[str, np.ndarray]], n_heads: int,
            eps: float) -> np.ndarray:
    """f_enc: full pre-LN blocks over the encoder rows only (bidirectional)."""
    x = _f(e)
    n = x.shape[0]
    for p in params:
        d = x.shape[1]
        kc = np.zeros((n_heads, n, d // n_heads))
        x = block.full_layer(p, x, kc, kc.copy(), n_heads=n_heads, eps=eps).x_out
    return x


def encoder_to_decoder(h_enc, ln_g, ln_b, eps: float, w_de, b_de, mask_emb, pe_dec,
                       known: Sequence[int], n_buf: int) -> np.ndarray:
    """Eq. 2's decoder input [N][D] for one image: LN + linear embedding of the
    encoder rows, scattered back to their sequence positions (buffer rows to
    0..n_buf-1, known rows to ``known`` in row order), the mask embedding at
    every other position, plus the decoder's positional embedding."""
    pe = _f(pe_dec)
    v = block.linear(block.layer_norm(h_enc, ln_g, ln_b, eps), w_de, b_de)
    x = pe + _f(mask_emb)
    targets = list(range(n_buf)) + [int(j) for j in known]
    for r, j in enumerate(targets):
        x[j] = v[r] + pe[j]
    return x


def decoder_cond(x_dec, ln_g, ln_b, eps: float, pe_diff, gen: Sequence[int], n_buf: int) -> np.ndarray:
    """z_i of Eq. 3 for the generating tokens ``gen`` (sequence positions):
    the decoder's final LayerNorm of row i plus the head's positional
    embedding of image token i - n_buf.  Returns [len(gen)][D]."""
    x = _f(x_dec)
    g = [int(i) for i in gen]
    return block.layer_norm(x[g], ln_g, ln_b, eps) + _f(pe_diff)[[i - n_buf for i in g]]


# ------------------------------------------------------------------ Eq. 3: denoiser

def timestep_embedding(t, dim: int, max_period: float = 10000.0) -> np.ndarray:
    """Sinusoidal embedding [cos(t f_0) .. cos(t f_{h-1}) | sin(t f_0) .. sin(t f_{h-1})]
    with f_i = max_period^(-i/h), h = dim / 2.  ``t`` scalar or [n]; returns [.., dim]."""
    half = dim // 2
    freqs = np.exp(-math.log(max_period) * np.arange(half, dtype=F64) / half)
    args = np.multiply.outer(_f(t), freqs)
    return np.concatenate([np.cos(args), np.sin(args)], axis=-1)


@dataclass(frozen=True)
class HeadShape:
    width: int       # W
    n_blocks: int
    c_tok: int       # C, token channels
    d_cond: int      # D, width of z
    t_freq: int = 256
    eps: float = 1e-6


def modulation_slices(hs: HeadShape, k: int):
    """Row ranges of the concatenated modulation weight: block k's shift, scale,
    gate (k < n_blocks) or the final layer's shift, scale (k == n_blocks)."""
    W = hs.width
    base = 3 * W * k
    if k < hs.n_blocks:
        return slice(base, base + W), slice(base + W, base + 2 * W), slice(base + 2 * W, base + 3 * W)
    return slice(base, base + W), slice(base + W, base + 2 * W)


def time_cond(t, head: Dict[str, np.ndarray], hs: HeadShape) -> np.ndarray:
    """Time embedding MLP: W_t2 SiLU(W_t1 sinus(t) + b_t1) + b_t2."""
    e = timestep_embedding(t, hs.t_freq)
    return block.linear(silu(block.linear(e, head["w_t1"], head["b_t1"])), head["w_t2"], head["b_t2"])


def denoiser(x, t, z, head: Dict[str, np.ndarray], hs: HeadShape) -> np.ndarray:
    """Predicted noise eps [M][C] for token values x [M][C] at timestep t given
    conditions z [M][D] (rows independent)."""
    c = time_cond(t, head, hs) + block.linear(z, head["w_c"], head["b_c"])
    sc = silu(c)
    mod = block.linear(sc, head["w_ada"], head["b_ada"])
    h = block.linear(x, head["w_in"], head["b_in"])
    for k in range(hs.n_blocks):
        sh, sc_, g = modulation_slices(hs, k)
        a = layer_norm_plain(h, hs.eps) * (1.0 + mod[:, sc_]) + mod[:, sh]
        y = block.linear(silu(block.linear(a, head["w_1"][k], head["b_1"][k])),
                         head["w_2"][k], head["b_2"][k])
        h = h + mod[:, g] * y
    sh, sc_ = modulation_slices(hs, hs.n_blocks)
    a = layer_norm_plain(h, hs.eps) * (1.0 + mod[:, sc_]) + mod[:, sh]
    return block.linear(a, head["w_out"], head["b_out"])


# ------------------------------------------------------------------ Eq. 3: sampler

@dataclass
class Schedule:
    betas: np.ndarray       # [T]
    alphas_bar: np.ndarray  # [T]

    @property
    def T(self) -> int:
        return len(self.betas)

    def alpha_bar_prev(self, i: int) -> float:
        return 1.0 if i == 0 else float(self.alphas_bar[i - 1])


def cosine_schedule(T: int, s: float = 0.008, max_beta: float = 0.999) -> Schedule:
    """beta_i = min(1 - g((i+1)/T) / g(i/T), max_beta), g(u) = cos^2((u + s)/(1 + s) pi/2);
    alpha_bar_i = prod_{j<=i} (1 - beta_j)."""
    g = lambda u: math.cos((u + s) / (1 + s) * math.pi / 2) ** 2
    betas = np.array([min(1 - g((i + 1) / T) / g(i / T), max_beta) for i in range(T)], F64)
    return Schedule(betas, np.cumprod(1.0 - betas))


def posterior(sch: Schedule, i: int):
    """Coefficients of q(x_{i-1} | x_i, x0): mean c1 x0 + c2 x_i, variance var."""
    ab, abp, b = float(sch.alphas_bar[i]), sch.alpha_bar_prev(i), float(sch.betas[i])
    c1 = b * math.sqrt(abp) / (1 - ab)
    c2 = (1 - abp) * math.sqrt(1 - b) / (1 - ab)
    var = b * (1 - abp) / (1 - ab)
    return c1, c2, var


def predict_x0(sch: Schedule, i: int, x, eps) -> np.ndarray:
    """x0 = (x_i - sqrt(1 - alpha_bar_i) eps) / sqrt(alpha_bar_i)."""
    ab = float(sch.alphas_bar[i])
    return (_f(x) - math.sqrt(1 - ab) * _f(eps)) / math.sqrt(ab)


def ddpm_step(sch: Schedule, i: int, x, eps, tau: float, noise) -> np.ndarray:
    """One ancestral step i -> i - 1: posterior mean from the predicted x0, plus
    tau * sqrt(var) * noise except at the last step (i == 0)."""
    c1, c2, var = posterior(sch, i)
    mean = c1 * predict_x0(sch, i, x, eps) + c2 * _f(x)
    if i == 0:
        return mean
    return mean + tau * math.sqrt(var) * _f(noise)


def sample(z, noise, T: int, tau: float, head: Dict[str, np.ndarray], hs: HeadShape) -> np.ndarray:
    """Eq. 3 for rows z [M][D]: x_T = noise[T]; for i = T-1 .. 0,
    x <- ddpm_step(x, denoiser(x, i, z), noise[i]).  ``noise`` [T+1][M][C]."""
    sch = cosine_schedule(T)
    nz = _f(noise)
    x = nz[T].copy()
    for i in range(T - 1, -1, -1):
        x = ddpm_step(sch, i, x, denoiser(x, i, z, head, hs), tau, nz[i])
    return x
