"""Guard bands around every buffer the step and the selection write (GPU).

x, the K/V caches, the per-head scores, the workspace and the refresh output
are each placed between two 64 KB guard regions holding a canary pattern;
one cache-aware bf16 layer (ragged active sets: one token, a typical set,
every token; a key count that is not a multiple of the 64-key tile) and a
top-k selection then run through the C ABI.  Every guard byte must keep its
canary, and the results must be bitwise those of the same call on plain
buffers.  Rows outside the active sets are checked bitwise by the parity
tests; this catches writes past the ends of the buffers, which they cannot.
"""
import numpy as np
import pytest
import torch

from paper_2506_12035_amd import binding, workload
from tests.gpu_util import DEV, SingleLayer, say, upload_params

pytestmark = pytest.mark.gpu

GUARD = 64 * 1024  # bytes on each side
CANARY = 0x5A  # byte pattern of every guard


class Guarded:
    """A device buffer of `nbytes` between two canary-filled guard regions."""

    def __init__(self, nbytes):
        self.nbytes = nbytes
        self.raw = torch.full((GUARD + nbytes + GUARD,), CANARY, dtype=torch.uint8, device=DEV)

    def view(self, dtype, shape):
        inner = self.raw[GUARD:GUARD + self.nbytes]
        return inner.view(dtype).view(*shape)

    def check(self, name):
        lo = self.raw[:GUARD]
        hi = self.raw[GUARD + self.nbytes:]
        bad_lo = int((lo != CANARY).sum())
        bad_hi = int((hi != CANARY).sum())
        assert bad_lo == 0 and bad_hi == 0, f"{name}: {bad_lo} bytes before, {bad_hi} after changed"


def test_step_and_selection_stay_inside_their_buffers():
    cfg = workload.CONFIGS[3].with_(n_tokens=300, n_layers=1)
    N, D, H, dh = cfg.n_tokens, cfg.d_model, cfg.n_heads, cfg.head_dim
    rng = np.random.default_rng(31)
    sizes, gens = [1, 39, N], [1, 5, 7]
    B = len(sizes)
    x = rng.standard_normal((B, N, D), dtype=np.float32)
    kc = workload.round_to(rng.standard_normal((B, H, N, dh), dtype=np.float32), "bf16")
    vc = workload.round_to(rng.standard_normal((B, H, N, dh), dtype=np.float32), "bf16")
    active = [rng.permutation(N)[:s].astype(np.int32) for s in sizes]
    p = workload.layer_weights(cfg, 0)
    ref = SingleLayer(cfg, p, x, kc, vc).run(active, gens)

    model = binding.make_model(1, D, H, dh, cfg.d_mlp, N, binding.MARCHE_BF16, cfg.ln_eps)
    params = upload_params(p, "bf16")
    layers = binding.make_layers([params])
    gx = Guarded(B * N * D * 4)
    gk = Guarded(B * H * N * dh * 2)
    gv = Guarded(B * H * N * dh * 2)
    gs = Guarded(B * H * N * 4)
    xd = gx.view(torch.float32, (B, N, D))
    kd = gk.view(torch.bfloat16, (B * H * N * dh,))
    vd = gv.view(torch.bfloat16, (B * H * N * dh,))
    sd = gs.view(torch.float32, (B, H, N))
    # bind the cache first (without initial values it is zero-filled), then
    # write the cached rows
    cache = binding.kv_cache_init(model, B, kd, vd, kd.numel() * 2)
    xd.copy_(torch.from_numpy(x))
    kd.copy_(torch.from_numpy(kc.reshape(-1)).to(torch.bfloat16))
    vd.copy_(torch.from_numpy(vc.reshape(-1)).to(torch.bfloat16))
    idx = torch.from_numpy(np.concatenate(active)).to(DEV)
    off_np = np.zeros(B + 1, np.int32)
    off_np[1:] = np.cumsum(sizes)
    off = torch.from_numpy(off_np).to(DEV)
    gen = torch.tensor(gens, dtype=torch.int32, device=DEV)
    a_total = int(off_np[-1])
    wsb = binding.workspace_bytes(model, B, a_total)
    gw = Guarded((wsb + 255) // 256 * 256)
    wsd = gw.view(torch.uint8, (gw.nbytes,))
    say(f"  guarded step: B={B} N={N} a_total={a_total} workspace={wsb}")
    binding.marche_step(model, layers, cache, 0, 1, B, xd, idx, off, gen, a_total, max(sizes),
                        max(gens), sd, 0, wsd, wsb)
    torch.cuda.synchronize()
    for g, name in ((gx, "x"), (gk, "K cache"), (gv, "V cache"), (gs, "scores"), (gw, "workspace")):
        g.check(name)
    np.testing.assert_array_equal(xd.cpu().numpy(), ref["x"])
    np.testing.assert_array_equal(kd.float().cpu().numpy().reshape(ref["k"].shape), ref["k"])
    np.testing.assert_array_equal(vd.float().cpu().numpy().reshape(ref["v"].shape), ref["v"])
    np.testing.assert_array_equal(sd.cpu().numpy(), ref["scores"])

    # selection of k = 16 per image for the first two images (the third has
    # no candidates left), written at per-image offsets of a guarded list
    k = 16
    go = Guarded(2 * k * 4)
    od = go.view(torch.int32, (2 * k,))
    excl = torch.from_numpy(np.concatenate(active[:2])).to(DEV)
    eoff = torch.from_numpy(off_np[:3].copy()).to(DEV)
    ooff = torch.tensor([0, k], dtype=torch.int32, device=DEV)
    binding.select_refresh(sd[:2], H, excl, eoff, 2, N, k, od, ooff)
    torch.cuda.synchronize()
    go.check("refresh output")
    sel = od.cpu().numpy().reshape(2, k)
    for b in range(2):
        assert len(set(sel[b])) == k and not set(sel[b]) & set(active[b].tolist())
        assert list(sel[b]) == sorted(sel[b]) and sel[b].min() >= 0 and sel[b].max() < N
