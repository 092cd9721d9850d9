"""Decoding-step driver: composes the C-ABI calls into MARche steps.

One step t of a batch of images (Section 4.2-4.3, Algorithm 1):

* build the decoder input x (marche_decoder_input);
* full step (the first step and every periodic full refresh): one
  marche_step over all layers with every token active;
* otherwise: marche_step over layers [0, sel_layer) with every token active
  and the generating tokens first, writing the selection layer's per-head
  attention mass; select_refresh picks R per image into the tail of the
  cache-aware active list [G | N | R]; marche_step over layers
  [sel_layer, L) on that list.  With micro_batches > 1 every step after
  the decoder input runs per range of consecutive images
  (marche_step_images), each range on its own stream.

All index lists of every step are built on the host once, before decoding,
and kept resident on the device; a step issues only kernel launches and
stream events (no host synchronisation, no host-device copies).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import binding, schedule, workload


def _dev_i32(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)


# Active-set constructions (the method and the ablations of Tables 2-3):
#   marche         A = G u N u R, R = highest attention mass (Section 4.2)
#   low-attention  A = G u N u R, R = lowest attention mass
#   random         A = G u N u R, R drawn at random (seeded) from the candidates
#   no-caching     A = G u R (caching tokens not forced in; they may be refreshed)
#   no-generating  A = N u R (generating tokens left out of the later layers)
STRATEGIES = ("marche", "low-attention", "random", "no-caching", "no-generating")


@dataclass
class StepPlan:
    t: int
    full: bool
    n_known: int
    g: int
    n: int
    k: int
    full_idx: torch.Tensor
    full_off: torch.Tensor
    n_gen: torch.Tensor
    a: int = 0                                # cache-aware active rows per image
    ca_idx: Optional[torch.Tensor] = None
    ca_off: Optional[torch.Tensor] = None
    ca_gen: Optional[torch.Tensor] = None     # generating rows leading the cache-aware list
    ca_gen_max: int = 0
    excl_idx: Optional[torch.Tensor] = None
    excl_off: Optional[torch.Tensor] = None
    out_off: Optional[torch.Tensor] = None
    device_select: bool = True                # R chosen on the device from the scores
    select_lowest: bool = False
    parts: Optional[list] = None              # per image range of a split step (RangePlan)


@dataclass
class RangePlan:
    """The lists of one range of consecutive images: views of the step's
    lists with offsets rebased to the range's first image (the cache-aware
    ones only in cache-aware steps)."""
    first: int
    count: int
    full_idx: torch.Tensor
    full_off: torch.Tensor
    n_gen: torch.Tensor
    ca_idx: Optional[torch.Tensor] = None
    ca_off: Optional[torch.Tensor] = None
    ca_gen: Optional[torch.Tensor] = None
    excl_idx: Optional[torch.Tensor] = None
    excl_off: Optional[torch.Tensor] = None
    out_off: Optional[torch.Tensor] = None


class Engine:
    """Device state and step composition for one workload configuration."""

    def __init__(self, cfg: workload.Config, device: str = "cuda", batch: Optional[int] = None,
                 n_layers: Optional[int] = None, ratio_bp: Optional[int] = None,
                 policy: str = "ratio", budget: Optional[int] = None,
                 full_every: Optional[int] = None, sel_layer: Optional[int] = None,
                 weights: Optional[Sequence[Dict[str, np.ndarray]]] = None,
                 strategy: str = "marche", first_image: int = 0, micro_batches: int = 1,
                 range_sizes: Optional[Sequence[int]] = None):
        """``batch`` images starting at image ``first_image`` of the workload's
        batch.  ``micro_batches`` > 1 runs every step (after the decoder input)
        as that many ranges of consecutive images, each enqueued on a HIP
        stream of its own (see ``step``); the ranges are as equal as possible
        unless ``range_sizes`` gives each range's image count (positive, summing
        to the batch; it overrides ``micro_batches``)."""
        if n_layers is not None:
            cfg = cfg.with_(n_layers=n_layers)
        self.cfg = cfg
        self.device = torch.device(device)
        self.B = cfg.batch if batch is None else batch
        if range_sizes is not None:
            sizes = [int(n) for n in range_sizes]
            if not sizes or min(sizes) < 1 or sum(sizes) != self.B:
                raise ValueError(f"range_sizes={list(range_sizes)} must be positive image "
                                 f"counts summing to batch={self.B}")
            S = len(sizes)
        else:
            S = micro_batches
            if not 1 <= S <= max(self.B, 1):
                raise ValueError(f"micro_batches={S} must lie in [1, batch={self.B}]")
            sizes = [self.B // S + (1 if i < self.B % S else 0) for i in range(S)]
        if strategy not in STRATEGIES:
            raise ValueError(f"strategy must be one of {STRATEGIES}")
        self.strategy = strategy
        self.policy = policy
        if budget is None:
            if policy != "ratio":
                raise ValueError("a fixed budget needs `budget` (the active-set size)")
            budget = cfg.ratio_bp if ratio_bp is None else ratio_bp
        schedule.check_budget(policy, budget, cfg.n_tokens)
        self.budget = budget
        self.full_every = cfg.full_every if full_every is None else full_every
        if self.full_every < 0:
            raise ValueError("full_every must be >= 0")
        self.sel = cfg.sel_layer if sel_layer is None else sel_layer
        if not 1 <= self.sel <= cfg.n_layers:
            raise ValueError("sel_layer must lie in [1, n_layers]")
        self.dt = binding.MARCHE_BF16 if cfg.dtype == "bf16" else binding.MARCHE_F32
        self.tdtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        L, D, H, N, dh, F = (cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_tokens, cfg.head_dim,
                             cfg.d_mlp)
        self.model = binding.make_model(L, D, H, dh, F, N, self.dt, cfg.ln_eps)

        ws = weights if weights is not None else [workload.layer_weights(cfg, l) for l in range(L)]
        self.params = [self._upload_layer(w) for w in ws]
        self.layers = binding.make_layers(self.params)

        es = 2 if cfg.dtype == "bf16" else 4
        n_el = L * self.B * H * N * dh
        self.k_cache = torch.empty(n_el, dtype=self.tdtype, device=self.device)
        self.v_cache = torch.empty(n_el, dtype=self.tdtype, device=self.device)
        self.cache = binding.kv_cache_init(self.model, self.B, self.k_cache, self.v_cache, n_el * es,
                                           stream=self.stream)
        self.x = torch.empty(self.B, N, D, dtype=torch.float32, device=self.device)
        self.scores = torch.empty(self.B, H, N, dtype=torch.float32, device=self.device)
        self.ranges = [(sum(sizes[:i]), sizes[i]) for i in range(S)]  # (first image, count)
        self.streams = [torch.cuda.Stream(device=self.device) for _ in range(S - 1)]
        # one workspace region per range, sized for the range with every token
        # active (a cache-aware step's range needs less and reuses it)
        self.ws_regions = []
        off = 0
        for _, n in self.ranges:
            nb = binding.workspace_bytes(self.model, n, n * N)
            self.ws_regions.append((off, nb))
            off += (nb + 255) // 256 * 256
        self.ws_bytes = off
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
        self.overlap = True  # False: the ranges one after another on the current stream

        self.first_image = first_image
        emb = workload.embeddings(cfg, self.B, first_image)
        self.orders = workload.orders(cfg, self.B, first_image)
        rank = np.empty_like(self.orders)
        for b in range(self.B):
            rank[b, self.orders[b]] = np.arange(cfg.n_img, dtype=np.int32)
        self.e_cls = torch.from_numpy(emb.cls).to(self.device)
        self.e_value = torch.from_numpy(emb.value).to(self.device)
        self.e_mask = torch.from_numpy(emb.mask).to(self.device)
        self.e_pos = torch.from_numpy(emb.pos).to(self.device)
        self.rank = _dev_i32(rank, self.device)
        self.set_schedule(self.full_every, self.policy, self.budget)

    def configure(self, sel_layer: Optional[int] = None, full_every: Optional[int] = None,
                  policy: Optional[str] = None, budget: Optional[int] = None,
                  strategy: Optional[str] = None) -> None:
        """Switch the decoding schedule (selection layer, refresh period, budget
        policy, active-set strategy) and rebuild the resident index lists."""
        if sel_layer is not None:
            if not 1 <= sel_layer <= self.cfg.n_layers:
                raise ValueError("sel_layer must lie in [1, n_layers]")
            self.sel = sel_layer
        if strategy is not None:
            if strategy not in STRATEGIES:
                raise ValueError(f"strategy must be one of {STRATEGIES}")
            self.strategy = strategy
        self.set_schedule(self.full_every if full_every is None else full_every,
                          self.policy if policy is None else policy,
                          self.budget if budget is None else budget)

    def set_schedule(self, full_every: int, policy: str, budget: int) -> None:
        """(Re)build the resident index lists of every step for a schedule:
        ``full_every`` = 1 with any budget is full recomputation."""
        schedule.check_budget(policy, budget, self.cfg.n_tokens)
        if full_every < 0:
            raise ValueError("full_every must be >= 0")
        self.full_every, self.policy, self.budget = full_every, policy, budget
        self.plans = [self._plan(t) for t in range(self.cfg.n_steps)]

    @property
    def stream(self):
        return torch.cuda.current_stream(self.device)

    # ------------------------------------------------------------------ setup

    def _upload_layer(self, w: Dict[str, np.ndarray]) -> Dict[str, torch.Tensor]:
        out = {}
        for name, a in w.items():
            t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
            if name.startswith("w_"):
                t = t.to(self.tdtype)
            out[name] = t.to(self.device).contiguous()
        return out

    def _plan(self, t: int) -> StepPlan:
        c = self.cfg
        si = schedule.step_indices(self.orders, c.n_buf, c.n_tokens, c.n_steps, t, self.full_every,
                                   self.policy, self.budget)
        B, N = self.B, c.n_tokens
        g, n = si.gen.shape[1], si.cache.shape[1]
        plan = StepPlan(t, si.full, si.n_known, g, n, si.k,
                        _dev_i32(si.full_order.reshape(-1), self.device),
                        _dev_i32(np.arange(B + 1) * N, self.device),
                        _dev_i32(np.full(B, g), self.device))
        if si.full:
            if len(self.ranges) > 1:
                plan.parts = self._range_plans(plan, 0, 0)
            return plan
        st = self.strategy
        forced_cache = si.cache if st != "no-caching" else si.cache[:, :0]
        if st == "no-caching":
            plan.k = schedule.refresh_count(self.policy, self.budget, N, g, 0)
        excl = np.concatenate([si.gen, forced_cache], axis=1)       # never refreshed
        if not 0 <= plan.k <= N - excl.shape[1]:
            # select_refresh would pad R with -1, which the step then indexes with
            raise ValueError(f"step {t}: refresh count {plan.k} exceeds the "
                             f"{N - excl.shape[1]} candidates")
        lead = forced_cache if st == "no-generating" else excl     # fixed head of A
        a = lead.shape[1] + plan.k
        ca = np.full((B, a), -1, np.int32)
        ca[:, :lead.shape[1]] = lead
        if st == "random":
            cand = np.stack([np.setdiff1d(np.arange(N), excl[b]) for b in range(B)])
            ca[:, lead.shape[1]:] = workload.random_refresh(c, t, cand, plan.k, self.first_image)
            plan.device_select = False
        plan.select_lowest = st == "low-attention"
        plan.a = a
        plan.ca_idx = _dev_i32(ca.reshape(-1), self.device)
        plan.ca_off = _dev_i32(np.arange(B + 1) * a, self.device)
        ca_g = 0 if st == "no-generating" else g
        plan.ca_gen = _dev_i32(np.full(B, ca_g), self.device)
        plan.ca_gen_max = ca_g
        plan.excl_idx = _dev_i32(excl.reshape(-1), self.device)
        plan.excl_off = _dev_i32(np.arange(B + 1) * excl.shape[1], self.device)
        plan.out_off = _dev_i32(np.arange(B) * a + lead.shape[1], self.device)
        if len(self.ranges) > 1:
            plan.parts = self._range_plans(plan, excl.shape[1], lead.shape[1])
        return plan

    def _range_plans(self, plan: StepPlan, n_excl: int, n_lead: int) -> List[RangePlan]:
        B, N, a = self.B, self.cfg.n_tokens, plan.a
        parts = []
        for first, n in self.ranges:
            sl = slice(first, first + n)
            r = RangePlan(first, n, plan.full_idx.view(B, N)[sl].reshape(-1),
                          _dev_i32(np.arange(n + 1) * N, self.device), plan.n_gen[sl])
            if not plan.full:
                r.ca_idx = plan.ca_idx.view(B, a)[sl].reshape(-1)
                r.ca_off = _dev_i32(np.arange(n + 1) * a, self.device)
                r.ca_gen = plan.ca_gen[sl]
                r.excl_idx = plan.excl_idx.view(B, n_excl)[sl].reshape(-1)
                r.excl_off = _dev_i32(np.arange(n + 1) * n_excl, self.device)
                r.out_off = _dev_i32(np.arange(n) * a + n_lead, self.device)
            parts.append(r)
        return parts

    # ------------------------------------------------------------------ step

    def decoder_input(self, t: int) -> None:
        c = self.cfg
        binding.decoder_input(self.x, self.e_cls, self.e_value, self.e_mask, self.e_pos, self.rank,
                              self.B, c.n_tokens, c.n_buf, c.d_model, self.plans[t].n_known,
                              stream=self.stream)

    def run_layers(self, begin: int, end: int, idx, off, a_total: int, a_max: int, g: int,
                   n_gen, score_layer: int = -1) -> None:
        binding.marche_step(self.model, self.layers, self.cache, begin, end, self.B, self.x, idx,
                            off, n_gen, a_total, a_max, g,
                            self.scores if score_layer >= 0 else None, score_layer,
                            self.workspace, self.ws_bytes, stream=self.stream)

    def select(self, p: StepPlan) -> None:
        if not p.device_select:
            return
        binding.select_refresh(self.scores, self.cfg.n_heads, p.excl_idx, p.excl_off, self.B,
                               self.cfg.n_tokens, p.k, p.ca_idx, p.out_off, stream=self.stream,
                               lowest=p.select_lowest)

    def step(self, t: int, build_input: bool = True) -> None:
        """One decoding step (all layers) of the whole batch, enqueued on the
        current stream (with image ranges: forked from and joined back into
        it)."""
        p = self.plans[t]
        c = self.cfg
        N, L, B = c.n_tokens, c.n_layers, self.B
        if build_input:
            self.decoder_input(t)
        if p.parts is None:
            if p.full:
                self.run_layers(0, L, p.full_idx, p.full_off, B * N, N, p.g, p.n_gen)
                return
            self.run_layers(0, self.sel, p.full_idx, p.full_off, B * N, N, p.g, p.n_gen,
                            score_layer=self.sel - 1 if p.device_select else -1)
            self.select(p)
            if p.a > 0:
                self.run_layers(self.sel, L, p.ca_idx, p.ca_off, B * p.a, p.a, p.ca_gen_max,
                                p.ca_gen)
            return
        # Image ranges: each range runs the whole step (every layer, the
        # selection) on its own stream between a fork from and a join back
        # into the current one, with its own workspace region.  Ranges share
        # no rows, so their kernels overlap on the GPU: one range's attention,
        # LayerNorm or partly filled last wave of tiles beside another's GEMMs.
        if not self.overlap:
            for i, r in enumerate(p.parts):
                self._range_step(p, r, i)
            return
        cur = self.stream
        fork = torch.cuda.Event()
        fork.record(cur)
        for i, r in enumerate(p.parts):
            s = cur if i == 0 else self.streams[i - 1]
            if i > 0:
                s.wait_event(fork)
            with torch.cuda.stream(s):
                self._range_step(p, r, i)
            if i > 0:
                done = torch.cuda.Event()
                done.record(s)
                cur.wait_event(done)

    def _range_step(self, p: StepPlan, r: RangePlan, i: int) -> None:
        c = self.cfg
        N, L, n = c.n_tokens, c.n_layers, r.count
        sl = slice(r.first, r.first + n)
        off, nb = self.ws_regions[i]
        ws = self.workspace[off:off + nb]

        def layers(begin, end, idx, a_off, gen, rows, a_max, gen_max, scores=None, score_layer=-1):
            binding.marche_step_images(self.model, self.layers, self.cache, r.first, begin, end, n,
                                       self.x[sl], idx, a_off, gen, rows, a_max, gen_max, scores,
                                       score_layer, ws, nb, stream=self.stream)

        if p.full:
            layers(0, L, r.full_idx, r.full_off, r.n_gen, n * N, N, p.g)
            return
        sel_scores = p.device_select
        layers(0, self.sel, r.full_idx, r.full_off, r.n_gen, n * N, N, p.g,
               self.scores[sl] if sel_scores else None, self.sel - 1 if sel_scores else -1)
        if p.device_select:
            binding.select_refresh(self.scores[sl], c.n_heads, r.excl_idx, r.excl_off, n, N, p.k,
                                   r.ca_idx, r.out_off, stream=self.stream,
                                   lowest=p.select_lowest)
        if p.a > 0:
            layers(self.sel, L, r.ca_idx, r.ca_off, r.ca_gen, n * p.a, p.a, p.ca_gen_max)

    def generate(self, steps: Optional[Sequence[int]] = None) -> None:
        for t in (range(self.cfg.n_steps) if steps is None else steps):
            self.step(t)

    # ------------------------------------------------------------------ readback (tests)

    def k_layer(self, l: int) -> torch.Tensor:
        c = self.cfg
        return self.k_cache.view(c.n_layers, self.B, c.n_heads, c.n_tokens, c.head_dim)[l]

    def v_layer(self, l: int) -> torch.Tensor:
        c = self.cfg
        return self.v_cache.view(c.n_layers, self.B, c.n_heads, c.n_tokens, c.head_dim)[l]

    def active_lists(self, t: int) -> Optional[np.ndarray]:
        """[B][|A|] cache-aware active list of step t as last computed."""
        p = self.plans[t]
        if p.full:
            return None
        return p.ca_idx.view(self.B, -1).cpu().numpy()

    def refresh_lists(self, t: int) -> Optional[np.ndarray]:
        """[B][k] refresh set of step t as last computed (ascending)."""
        p = self.plans[t]
        if p.full:
            return None
        lead = p.a - p.k
        return p.ca_idx.view(self.B, p.a)[:, lead:].cpu().numpy()


# ------------------------------------------------------------------ a whole MAR step

HEAD_GEMM_WEIGHTS = ("w_t1", "w_t2", "w_c", "w_ada", "w_1", "w_2")


class MarEngine:
    """A whole generation step of the masked autoregressive model around the
    cache-aware decoder: the encoder over the known tokens (Eq. 1), the
    decoder input built from its output (Eq. 2), the decoder step of
    ``Engine`` and the sampler that draws the generating tokens' values
    (Eq. 3), which become known tokens of the next step.

    The encoder runs as ``marche_step`` over its own stack with every row
    active; its row count n_buf + n_known changes with the step, so it has one
    model description per count and a scratch KV cache sized for all tokens.
    Every index list, the sampler's draws of every step and all weights are
    resident on the device before decoding; a step issues only kernel
    launches on one stream.
    """

    def __init__(self, mc: workload.MarConfig, device: str = "cuda", batch: Optional[int] = None,
                 steps: Optional[Sequence[int]] = None, **decoder_kw):
        self.mc = mc
        self.dec = Engine(mc.dec, device, batch, **decoder_kw)
        d = self.dec
        c = mc.dec
        self.device, self.B = d.device, d.B
        B, N, D, H, dh, C = self.B, c.n_tokens, c.d_model, c.n_heads, c.head_dim, mc.c_tok
        self.dt, self.tdtype = d.dt, d.tdtype

        # encoder stack and its scratch cache / workspace
        ec = mc.enc
        self.enc_params = [d._upload_layer(workload.layer_weights(ec, l)) for l in range(ec.n_layers)]
        self.enc_layers = binding.make_layers(self.enc_params)
        n_el = ec.n_layers * B * H * N * dh
        self.enc_k = torch.empty(n_el, dtype=self.tdtype, device=self.device)
        self.enc_v = torch.empty(n_el, dtype=self.tdtype, device=self.device)
        self.x_enc = torch.empty(B, N, D, dtype=torch.float32, device=self.device)
        big = self._enc_model(N)
        # one workspace region per image range of the decoder engine
        self.enc_regions, off = [], 0
        for _, n in d.ranges:
            nb = binding.workspace_bytes(big, n, n * N)
            self.enc_regions.append((off, nb))
            off += (nb + 255) // 256 * 256
        self.enc_ws_bytes = off
        self.enc_ws = torch.empty(self.enc_ws_bytes, dtype=torch.uint8, device=self.device)
        self.e2d_ws_bytes = max(256, binding.encoder_to_decoder_workspace_bytes(B, c.n_buf, c.n_img,
                                                                                D, self.dt))
        self.e2d_ws = torch.empty(self.e2d_ws_bytes, dtype=torch.uint8, device=self.device)

        emb = workload.mar_embeddings(mc, B)
        self.emb = {k: torch.from_numpy(np.ascontiguousarray(v, np.float32)).to(
            self.tdtype if k == "w_de" else torch.float32).to(self.device).contiguous()
            for k, v in emb.items()}

        # sampler head
        hw = workload.head_weights(mc)
        self.head_params = {k: torch.from_numpy(np.ascontiguousarray(v, np.float32)).to(
            self.tdtype if k in HEAD_GEMM_WEIGHTS else torch.float32).to(self.device).contiguous()
            for k, v in hw.items()}
        self.head = binding.make_head(mc.head_width, mc.head_blocks, C, D, mc.t_freq, self.dt,
                                      mc.head_eps)
        self.head_weights = binding.make_head_weights(self.head_params)
        self.tok = torch.zeros(B, c.n_img, C, dtype=torch.float32, device=self.device)

        # per-step resident lists and draws
        self.steps = list(range(c.n_steps)) if steps is None else list(steps)
        self.enc_lists: Dict[int, tuple] = {}
        self.known: Dict[int, Optional[torch.Tensor]] = {}
        self.gen_rows: Dict[int, tuple] = {}
        self.noise: Dict[int, torch.Tensor] = {}
        max_rows = 0
        for t in self.steps:
            p = d.plans[t]
            n_enc = c.n_buf + p.n_known
            if n_enc not in self.enc_lists:
                self.enc_lists[n_enc] = (
                    self._enc_model(n_enc),
                    _dev_i32(np.tile(np.arange(n_enc), B), self.device),
                    _dev_i32(np.arange(B + 1) * n_enc, self.device))
            known = np.sort(d.orders[:, :p.n_known], axis=1)
            self.known[t] = _dev_i32(known.reshape(-1), self.device) if p.n_known else None
            gen = np.stack(self._gen_tokens(t))  # [B][g] sequence positions
            b_idx = np.repeat(np.arange(B), gen.shape[1])
            pos = gen.reshape(-1) - c.n_buf
            rows = b_idx * N + c.n_buf + pos
            out_rows = b_idx * c.n_img + pos
            self.gen_rows[t] = (_dev_i32(rows, self.device), _dev_i32(out_rows, self.device),
                                int(rows.size))
            self.noise[t] = torch.from_numpy(workload.head_noise(mc, t, int(rows.size))).to(self.device)
            max_rows = max(max_rows, int(rows.size))
        self.head_ws_bytes = binding.diffusion_workspace_bytes(self.head, max_rows, mc.sample_steps)
        self.head_ws = torch.empty(self.head_ws_bytes, dtype=torch.uint8, device=self.device)

    def _enc_model(self, n_enc: int) -> binding.Model:
        c = self.mc.enc
        return binding.make_model(c.n_layers, c.d_model, c.n_heads, c.head_dim, c.d_mlp, n_enc,
                                  self.dt, c.ln_eps)

    def _gen_tokens(self, t: int) -> List[np.ndarray]:
        c = self.mc.dec
        m = schedule.masked_counts(c.n_img, c.n_steps)
        lo, hi = c.n_img - m[t], c.n_img - m[t + 1]
        return [c.n_buf + self.dec.orders[b, lo:hi] for b in range(self.B)]

    @property
    def stream(self):
        return self.dec.stream

    def encode(self, t: int) -> None:
        """Eq. 1 and 2: encoder over the known tokens, then the decoder input."""
        c, d, e = self.mc.dec, self.dec, self.emb
        p = d.plans[t]
        n_known = p.n_known
        n_enc = c.n_buf + n_known
        model, idx, off = self.enc_lists[n_enc]
        binding.encoder_input(self.x_enc, e["cls"], self.tok, e["w_z"], e["b_z"], e["pe_enc"],
                              self.known[t], self.B, c.n_buf, c.n_img, n_known, c.d_model,
                              self.mc.c_tok, stream=self.stream)
        ec = self.mc.enc
        cache = binding.KVCache(self.enc_k.data_ptr(), self.enc_v.data_ptr(), ec.n_layers, self.B,
                                ec.n_heads, n_enc, ec.head_dim, self.dt)
        # every image has the same encoder rows, so a range of n images takes
        # the first n lists; each range on its own stream, like the decoder's
        cur = self.stream
        fork = torch.cuda.Event()
        if len(d.ranges) > 1:
            fork.record(cur)
        for i, (first, n) in enumerate(d.ranges):
            s = cur if i == 0 else d.streams[i - 1]
            if i > 0:
                s.wait_event(fork)
            wo, wb = self.enc_regions[i]
            binding.marche_step_images(
                model, self.enc_layers, cache, first, 0, ec.n_layers, n,
                self.x_enc.view(-1)[first * n_enc * c.d_model:], idx[:n * n_enc], off[:n + 1],
                None, n * n_enc, n_enc, 0, None, -1, self.enc_ws[wo:wo + wb], wb, stream=s)
            if i > 0:
                done = torch.cuda.Event()
                done.record(s)
                cur.wait_event(done)
        binding.encoder_to_decoder(d.x, self.x_enc, e["enc_ln_g"], e["enc_ln_b"], c.ln_eps,
                                   e["w_de"], e["b_de"], e["mask"], e["pe_dec"], self.known[t],
                                   d.rank, self.B, c.n_buf, c.n_img, n_known, c.d_model, self.dt,
                                   self.e2d_ws, self.e2d_ws_bytes, stream=self.stream)

    def sample(self, t: int) -> None:
        """Eq. 3: draw the generating tokens' values from the decoder output."""
        c, e = self.mc.dec, self.emb
        rows, out_rows, n_rows = self.gen_rows[t]
        binding.diffusion_sample(self.head, self.head_weights, self.dec.x, c.n_tokens, c.n_buf,
                                 e["dec_ln_g"], e["dec_ln_b"], c.ln_eps, e["pe_diff"], rows,
                                 out_rows, n_rows, self.noise[t], self.mc.sample_steps,
                                 self.mc.temperature, self.tok, self.head_ws, self.head_ws_bytes,
                                 stream=self.stream)

    def step(self, t: int) -> None:
        self.encode(t)
        self.dec.step(t, build_input=False)
        self.sample(t)

    def generate(self) -> None:
        self.tok.zero_()
        for t in self.steps:
            self.step(t)
