"""Helpers for the GPU parity tests: upload seeded inputs, run one block through
the C ABI, and compare against the fp64 oracle."""
import sys

import numpy as np
import torch

from paper_2506_12035_amd import binding, workload

DEV = "cuda"
TOL = {"bf16": 2e-2, "f32": 1e-4}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel_err(gpu, ref) -> float:
    """Infinity-norm relative error max|g - r| / max|r|."""
    g = np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    den = np.abs(r).max()
    return float(np.abs(g - r).max() / (den if den > 0 else 1.0))


def tdtype(dtype: str):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def upload_params(p, dtype):
    out = {}
    for name, a in p.items():
        t = torch.from_numpy(np.ascontiguousarray(a, np.float32))
        if name.startswith("w_"):
            t = t.to(tdtype(dtype))
        out[name] = t.to(DEV).contiguous()
    return out


def f64(p):
    return {k: np.asarray(v, np.float64) for k, v in p.items()}


class SingleLayer:
    """One block run through marche_step for a batch of images with ragged
    active lists (generating tokens first in each list)."""

    def __init__(self, cfg: workload.Config, params, x, k_cache, v_cache):
        self.cfg = cfg
        c = cfg
        self.B = x.shape[0]
        self.dt = binding.MARCHE_BF16 if c.dtype == "bf16" else binding.MARCHE_F32
        self.model = binding.make_model(1, c.d_model, c.n_heads, c.head_dim, c.d_mlp, c.n_tokens,
                                        self.dt, c.ln_eps)
        self.p_dev = upload_params(params, c.dtype)
        self.layers = binding.make_layers([self.p_dev])
        td = tdtype(c.dtype)
        self.x = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(DEV)
        self.k = torch.from_numpy(np.ascontiguousarray(k_cache, np.float32)).to(td).to(DEV).contiguous()
        self.v = torch.from_numpy(np.ascontiguousarray(v_cache, np.float32)).to(td).to(DEV).contiguous()
        es = 2 if c.dtype == "bf16" else 4
        self.cache = binding.kv_cache_init(self.model, self.B, self.k, self.v, self.k.numel() * es,
                                           k_init=self.k.clone(), v_init=self.v.clone())
        # kv_cache_init copied from temporaries; keep the bound buffers as the state
        torch.cuda.synchronize()

    def run(self, active, n_gen, want_scores=True):
        c = self.cfg
        B = self.B
        idx = np.concatenate([np.asarray(a, np.int32) for a in active])
        off = np.zeros(B + 1, np.int32)
        off[1:] = np.cumsum([len(a) for a in active])
        a_total, a_max = int(off[-1]), max(len(a) for a in active)
        gen_max = max(n_gen)
        d_idx = torch.from_numpy(idx).to(DEV)
        d_off = torch.from_numpy(off).to(DEV)
        d_gen = torch.from_numpy(np.asarray(n_gen, np.int32)).to(DEV)
        ws_bytes = binding.workspace_bytes(self.model, B, a_total)
        ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=DEV)
        scores = torch.full((B, c.n_heads, c.n_tokens), float("nan"), device=DEV) if want_scores else None
        say(f"  marche_step: B={B} D={c.d_model} H={c.n_heads} dh={c.head_dim} N={c.n_tokens} "
            f"dtype={c.dtype} a_total={a_total} a_max={a_max}")
        binding.marche_step(self.model, self.layers, self.cache, 0, 1, B, self.x, d_idx, d_off, d_gen,
                            a_total, a_max, gen_max, scores, 0 if want_scores else -1, ws, ws_bytes)
        torch.cuda.synchronize()
        # attention output of the layer stays in the first activation buffer
        es = 2 if c.dtype == "bf16" else 4
        o_off = (a_total * 16 + 255) // 256 * 256
        o = ws[o_off:o_off + a_total * c.d_model * es].view(tdtype(c.dtype)).view(a_total, c.d_model)
        return {
            "x": self.x.cpu().numpy(),
            "k": self.k.float().cpu().numpy(),
            "v": self.v.float().cpu().numpy(),
            "o": o.float().cpu().numpy(),
            "scores": scores.cpu().numpy() if want_scores else None,
            "off": off,
        }


def record(kind: str, **fields) -> None:
    """Append one JSON line to the file named by MARCHE_PARITY_LOG, if set, so
    that a run's parity summary (worst errors, refresh-set counts) outlives
    pytest's output capture."""
    import json
    import os
    path = os.environ.get("MARCHE_PARITY_LOG")
    if not path:
        return
    d = os.path.dirname(path)
    if d:
        os.makedirs(d, exist_ok=True)
    with open(path, "a") as f:
        f.write(json.dumps({"kind": kind, **fields}, default=float) + "\n")


def check_refresh_set(got, s, excl, k, tol, lowest=False):
    """Gap rule for a GPU refresh set against the oracle's summed scores s.

    Returns "exact" when the oracle's relative gap at the k-th boundary
    exceeds tol (the set must then equal the oracle's), else "ambiguous"
    after checking that the set is valid on both sides of the boundary:
    every chosen token lies within tol of the k-th score, and every candidate
    clearly past it (beyond tol) is chosen."""
    from oracle import select as osel
    got = sorted(int(v) for v in got)
    excl = [int(e) for e in excl]
    cand = np.setdiff1d(np.arange(len(s)), excl)
    assert len(set(got)) == k and not set(got) & set(excl), "GPU refresh set invalid"
    assert set(got) <= set(cand.tolist()), "GPU refresh set holds a non-candidate"
    ordered = np.sort(s[cand])
    if not lowest:
        ordered = ordered[::-1]
    if k == 0:
        return "exact"
    sk = ordered[k - 1]
    gap = (abs(sk - ordered[k]) / max(abs(sk), abs(ordered[k])) if k < len(ordered) else np.inf)
    if gap > tol:
        want = osel.select_topk(s, excl, k, lowest=lowest)
        assert got == list(want), f"refresh set differs with gap {gap:.2e}"
        return "exact"
    if lowest:
        assert all(s[j] <= sk * (1 + tol) for j in got), "GPU refresh set outside tolerance"
        must = [int(j) for j in cand if s[j] < sk * (1 - tol)]
    else:
        assert all(s[j] >= sk * (1 - tol) for j in got), "GPU refresh set outside tolerance"
        must = [int(j) for j in cand if s[j] > sk * (1 + tol)]
    missing = sorted(set(must) - set(got))
    assert not missing, f"tokens clearly past the k-th score were not chosen: {missing[:8]}"
    return "ambiguous"
