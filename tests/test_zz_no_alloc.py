"""marche_step_images_noalloc against marche_step_images (GPU).

The no-allocation entry point runs the same kernels as marche_step_images,
with the step's workspace in the library's own device array instead of the
caller's.  Two calls in a row (the second on fewer images and fewer active
rows, so it starts from the first call's leftovers in the array) must give
bit-identical x, K/V caches and scores to the caller-workspace entry point on
the same state.  The sizes are MAR-L's width and depth-2 stack, with ragged
active sets that span several GEMM and query tiles, full layers included.
"""
import numpy as np
import pytest
import torch

from paper_2506_12035_amd import binding, workload
from tests.gpu_util import DEV, say, upload_params

pytestmark = pytest.mark.gpu


class _State:
    """A 2-layer MAR-L-width stack on a batch of images: x, K/V caches."""

    def __init__(self, cfg, B, seed):
        rng = np.random.default_rng(seed)
        c = cfg
        self.model = binding.make_model(c.n_layers, c.d_model, c.n_heads, c.head_dim, c.d_mlp,
                                        c.n_tokens, binding.MARCHE_BF16, c.ln_eps)
        self.params = [upload_params(workload.layer_weights(c, l), "bf16") for l in range(c.n_layers)]
        self.layers = binding.make_layers(self.params)
        n_el = c.n_layers * B * c.n_heads * c.n_tokens * c.head_dim
        kv = rng.standard_normal((2, n_el), dtype=np.float32)
        self.k = torch.empty(n_el, dtype=torch.bfloat16, device=DEV)
        self.v = torch.empty(n_el, dtype=torch.bfloat16, device=DEV)
        # bound without initial values the cache is zero-filled: the cached
        # rows are written afterwards
        self.cache = binding.kv_cache_init(self.model, B, self.k, self.v, n_el * 2)
        self.k.copy_(torch.from_numpy(kv[0]).to(torch.bfloat16))
        self.v.copy_(torch.from_numpy(kv[1]).to(torch.bfloat16))
        self.x = torch.from_numpy(rng.standard_normal((B, c.n_tokens, c.d_model),
                                                      dtype=np.float32)).to(DEV)
        self.scores = torch.full((B, c.n_heads, c.n_tokens), float("nan"), device=DEV)
        torch.cuda.synchronize()

    def clone_from(self, other):
        self.k.copy_(other.k)
        self.v.copy_(other.v)
        self.x.copy_(other.x)
        self.scores.copy_(other.scores)
        torch.cuda.synchronize()


def _lists(cfg, sizes, gens, seed):
    rng = np.random.default_rng(seed)
    act = []
    for s, g in zip(sizes, gens):
        a = rng.permutation(cfg.n_tokens)[:s].astype(np.int32)
        act.append(a)
    idx = np.concatenate(act)
    off = np.zeros(len(sizes) + 1, np.int32)
    off[1:] = np.cumsum(sizes)
    return (torch.from_numpy(idx).to(DEV), torch.from_numpy(off).to(DEV),
            torch.from_numpy(np.asarray(gens, np.int32)).to(DEV), int(off[-1]), max(sizes), max(gens))


def _call(st, noalloc, first, n, lists, layer_begin, layer_end, score_layer):
    idx, off, gen, a_total, a_max, gen_max = lists
    x = st.x[first:first + n]
    scores = st.scores[first:first + n]
    args = (st.model, st.layers, st.cache, first, layer_begin, layer_end, n, x, idx, off, gen,
            a_total, a_max, gen_max, scores, score_layer)
    if noalloc:
        binding.marche_step_images_noalloc(*args)
    else:
        wsb = binding.workspace_bytes(st.model, n, a_total)
        ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
        binding.marche_step_images(*args, ws, wsb)
    torch.cuda.synchronize()


def test_noalloc_matches_caller_workspace_on_two_calls():
    cfg = workload.CONFIGS[3].with_(n_layers=2, batch=6)
    B = 6
    ref = _State(cfg, B, seed=41)
    got = _State(cfg, B, seed=41)
    got.clone_from(ref)
    calls = [
        # images 0..5: ragged sets (one token .. every token), scores at layer 1
        (0, 6, ([1, 39, 161, 320, 64, 250], [1, 5, 25, 7, 9, 3]), 0, 2, 1),
        # then a smaller call on images 2..3 of the same cache
        (2, 2, ([44, 17], [6, 2]), 0, 2, 0),
    ]
    for i, (first, n, (sizes, gens), lb, le, sl) in enumerate(calls):
        lists = _lists(cfg, sizes, gens, seed=100 + i)
        need = binding.workspace_bytes(ref.model, n, lists[3])
        say(f"  noalloc call {i}: images [{first}, {first + n}) a_total={lists[3]} "
            f"workspace {need / 2**20:.1f} MiB of {binding.SCRATCH_BYTES / 2**20:.0f}")
        assert need <= binding.SCRATCH_BYTES
        _call(ref, False, first, n, lists, lb, le, sl)
        _call(got, True, first, n, lists, lb, le, sl)
        assert torch.equal(got.x, ref.x), f"call {i}: x differs"
        assert torch.equal(got.k, ref.k), f"call {i}: K cache differs"
        assert torch.equal(got.v, ref.v), f"call {i}: V cache differs"
        sc = slice(first, first + n)
        assert torch.equal(got.scores[sc], ref.scores[sc]), f"call {i}: scores differ"
        assert torch.isfinite(got.x).all()


def test_noalloc_refuses_oversize_step():
    cfg = workload.CONFIGS[3].with_(n_layers=2, batch=20)
    st = _State(cfg, 20, seed=3)
    lists = _lists(cfg, [320] * 20, [1] * 20, seed=9)
    assert binding.workspace_bytes(st.model, 20, lists[3]) > binding.SCRATCH_BYTES
    with pytest.raises(binding.MarcheError) as e:
        binding.marche_step_images_noalloc(st.model, st.layers, st.cache, 0, 0, 2, 20, st.x,
                                           lists[0], lists[1], lists[2], lists[3], lists[4],
                                           lists[5], None, -1)
    assert e.value.status == binding.MARCHE_ERR_WORKSPACE
