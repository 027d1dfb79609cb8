"""GPU test of pp_attn_fwd_noalloc, the forward for callers that cannot
allocate device memory: through the C ABI it must give exactly what
pp_attn_fwd gives (same kernels, same plan; its metadata sits in the library's
static device scratch instead of a workspace), on two calls in a row, the
second with a smaller pack, so that the second runs on scratch that still holds
the first call's larger plan.  One case is also held to the oracle's bars."""
import numpy as np
import pytest
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import binding as pp
from paper_2602_24082_amd import workload as wl
from tolerances import lse_excess, o_excess

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _run(pack, hq, hkv, d, seed):
    print(f"case noalloc T={pack.total_tokens} hq={hq} hkv={hkv} d={d}", flush=True)
    q, k, v, _ = wl.qkv(pack, hq, hkv, d, seed, torch.bfloat16, device=DEV)
    o1, l1 = pp.pp_attn_fwd(pack, q, k, v)
    o2 = torch.full_like(q, float("nan"))
    l2 = torch.full((hq, pack.total_tokens), float("nan"), device=DEV)
    pp.pp_attn_fwd_noalloc(pack, q, k, v, out=o2, lse=l2)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    return q, k, v, o2, l2


def test_noalloc_forward_equals_workspace_forward():
    big = wl.config_pack(wl.LLAMA3_8B)  # the 8B-shaped batch, 10861 tokens
    _run(big, 32, 8, 128, 7)
    small = wl.make_pack([300, 0, 129, 5], [[70, 45], [33, 64], [1, 0, 200], [130]], pad=[3, 0, 0, 17])
    q, k, v, o, lse = _run(small, 8, 2, 128, 8)
    args = small.oracle_args()
    qn, kn, vn = (x.double().cpu().numpy() for x in (q, k, v))
    O, L = orc.attn_fwd(*args, qn, kn, vn)
    assert o_excess(o.double().cpu().numpy(), O, True) <= 0
    assert lse_excess(lse.double().cpu().numpy(), L) <= 0
    # d = 64 and a pack of a single short row on the same scratch
    _run(wl.make_pack([7], [[3]]), 4, 4, 64, 9)
