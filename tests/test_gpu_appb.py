"""Parity of the stand-alone segment attention (Appendix B's comparison) on the
GPU: the two-segment pass and the concatenate-then-attend baseline, both
against the fp64 oracle's two-segment attention (Appendix A), element by
element, on the same seeded inputs."""
import numpy as np
import pytest

from oracle import block
from paper_2506_12035_amd import workload

from gpu_util import rel_err, say

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-2

# (batch, heads, head_dim, n_active, n_cached): the paper's 32 / 256 example,
# ragged tails in both segments, an empty cached segment, a long cached one,
# and the MAR-H head width.
CASES = [
    (4, 16, 64, 32, 256),
    (3, 4, 64, 45, 203),
    (2, 4, 64, 130, 0),
    (2, 2, 64, 7, 1500),
    (2, 4, 80, 70, 250),
]


def _dev(a, torch, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(dtype).contiguous()


@pytest.mark.parametrize("case", CASES, ids=lambda c: "b{}h{}d{}-a{}-c{}".format(*c))
@pytest.mark.parametrize("mode", ["two_segment", "concat"])
def test_segment_attention_parity(case, mode):
    import torch
    from paper_2506_12035_amd import binding

    B, H, dh, na, nc = case
    say(f"segment attention {mode} {case}")
    c = workload.segment_case(B, H, dh, na, nc)
    bf = torch.bfloat16
    q, ka, va = _dev(c.q, torch, bf), _dev(c.k_a, torch, bf), _dev(c.v_a, torch, bf)
    kc = _dev(c.k_c, torch, bf) if nc else None
    vc = _dev(c.v_c, torch, bf) if nc else None
    o = torch.full((B, na, H * dh), float("nan"), device="cuda", dtype=bf)
    m = binding.MARCHE_ATTN_TWO_SEGMENT if mode == "two_segment" else binding.MARCHE_ATTN_CONCAT
    wsb = binding.attention_workspace_bytes(B, H, dh, na, nc, binding.MARCHE_BF16, m)
    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device="cuda")
    binding.attention_segments(q, o, na, ka, va, na, kc, vc, nc, B, H, dh, binding.MARCHE_BF16, m,
                               ws if wsb else None, wsb)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy().reshape(B, na, H, dh)
    worst = 0.0
    for b in range(B):
        for h in range(H):
            ref = block.attention_two_segment(c.q[b, :, h * dh:(h + 1) * dh], c.k_a[b, h], c.v_a[b, h],
                                              c.k_c[b, h], c.v_c[b, h])
            worst = max(worst, rel_err(got[b, :, h], ref))
    say(f"  max rel err {worst:.2e}")
    assert np.isfinite(got).all()
    assert worst <= TOL_BF16


@pytest.mark.parametrize("n_a,n_c", [(0, 300), (300, 0)])
def test_single_segment_either_side(n_a, n_c):
    """Only one non-empty segment, with fewer queries than keys: the pass over
    one resident buffer (the layout of the decode step)."""
    import torch
    from paper_2506_12035_amd import binding

    B, H, dh, nq = 2, 4, 64, 40
    say(f"segment attention single segment n_a={n_a} n_c={n_c}")
    c = workload.segment_case(B, H, dh, nq, max(n_a, n_c))
    bf = torch.bfloat16
    q = _dev(c.q, torch, bf)
    kv = (_dev(c.k_c, torch, bf), _dev(c.v_c, torch, bf))
    o = torch.full((B, nq, H * dh), float("nan"), device="cuda", dtype=bf)
    a = kv if n_a else (None, None)
    cc = kv if n_c else (None, None)
    binding.attention_segments(q, o, nq, a[0], a[1], n_a, cc[0], cc[1], n_c, B, H, dh,
                               binding.MARCHE_BF16, binding.MARCHE_ATTN_TWO_SEGMENT)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy().reshape(B, nq, H, dh)
    worst = 0.0
    for b in range(B):
        for h in range(H):
            ref, _ = block.attention(c.q[b, :, h * dh:(h + 1) * dh], c.k_c[b, h], c.v_c[b, h])
            worst = max(worst, rel_err(got[b, :, h], ref))
    say(f"  max rel err {worst:.2e}")
    assert worst <= TOL_BF16
