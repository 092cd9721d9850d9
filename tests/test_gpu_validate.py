"""Debug-mode validation of the device-resident active lists (MARCHE_VALIDATE):
valid lists run unchanged; each kind of bad list is refused with
INVALID_ARG, naming the problem and the image, before any layer kernel is
launched (the check kernel reads only inside a_off[0..batch] and
a_idx[0..a_total), so a bad list is never dereferenced)."""
import numpy as np
import pytest
import torch

from paper_2506_12035_amd import binding, workload
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture
def setup(monkeypatch):
    monkeypatch.setenv("MARCHE_VALIDATE", "1")
    cfg = workload.CONFIGS[2].with_(n_layers=2, batch=3)
    B, N, D, H, dh, L = 3, cfg.n_tokens, cfg.d_model, cfg.n_heads, cfg.head_dim, 2
    rng = np.random.default_rng(9)
    model = binding.make_model(L, D, H, dh, cfg.d_mlp, N, binding.MARCHE_BF16, cfg.ln_eps)
    params = []
    for l in range(L):
        w = workload.layer_weights(cfg, l)
        params.append({k: torch.from_numpy(np.ascontiguousarray(v, np.float32)).to(
            torch.bfloat16 if k.startswith("w_") else torch.float32).cuda() for k, v in w.items()})
    layers = binding.make_layers(params)
    x0 = torch.from_numpy(rng.standard_normal((B, N, D)).astype(np.float32)).cuda()
    n_el = L * B * H * N * dh
    k0 = torch.from_numpy(rng.standard_normal(n_el).astype(np.float32)).to(torch.bfloat16).cuda()
    v0 = torch.from_numpy(rng.standard_normal(n_el).astype(np.float32)).to(torch.bfloat16).cuda()
    lists = [np.sort(rng.choice(N, size=a, replace=False)).astype(np.int32) for a in (30, 41, 25)]

    def run(lists, n_gen, a_off=None, a_max=None):
        x, k, v = x0.clone(), k0.clone(), v0.clone()
        cache = binding.kv_cache_init(model, B, k, v, n_el * 2, k_init=k0, v_init=v0)
        idx = torch.from_numpy(np.concatenate(lists)).cuda()
        total = int(idx.numel())
        off = np.concatenate([[0], np.cumsum([len(a) for a in lists])]).astype(np.int32)
        if a_off is not None:
            off = np.asarray(a_off, np.int32)
        a_max = max(len(a) for a in lists) if a_max is None else a_max
        wsb = binding.workspace_bytes(model, B, total)
        ws = torch.empty(wsb, dtype=torch.uint8).cuda()
        binding.marche_step(model, layers, cache, 0, L, B, x, idx, torch.from_numpy(off).cuda(),
                            torch.tensor(n_gen, dtype=torch.int32).cuda(), total, a_max,
                            max(n_gen), None, -1, ws, wsb)
        torch.cuda.synchronize()
        return x, k, v

    return run, lists, N


def test_valid_lists_run_unchanged(setup, monkeypatch):
    run, lists, N = setup
    say("validation: valid lists, with and without the check")
    checked = run(lists, [4, 6, 3])
    monkeypatch.setenv("MARCHE_VALIDATE", "0")
    plain = run(lists, [4, 6, 3])
    for a, b in zip(checked, plain):
        assert torch.equal(a, b)


@pytest.mark.parametrize("case,match", [
    ("duplicate", "listed twice .image 1"),
    ("range", "outside .0, n_tokens. .image 2"),
    ("offsets", "a_off inconsistent"),
    ("n_gen", "n_gen outside .*image 0"),
])
def test_bad_lists_are_refused(setup, case, match):
    run, lists, N = setup
    say(f"validation: {case}")
    lists = [a.copy() for a in lists]
    n_gen, a_off = [4, 6, 3], None
    if case == "duplicate":
        lists[1][5] = lists[1][6]
    elif case == "range":
        lists[2][0] = N
    elif case == "offsets":
        a_off = [0, 30, 71, 95]  # last entry != a_total = 96
    elif case == "n_gen":
        n_gen = [31, 6, 3]  # image 0 has 30 tokens
    with pytest.raises(RuntimeError, match=match):
        run(lists, n_gen, a_off=a_off)
