"""GPU check of the backward's central property (Sec. 1, Sec. 3.2): the prompt is
stored once, so the gradients of its keys and values gather the contributions
of all K responses, and the packed row gives the results of the unpacked
layout, where each (prompt, response_k) pair is its own causal sequence.

The packed row runs on the GPU.  The unpacked layout is the same tokens laid
out as K rows (prompt, response_k).  Its prompt query rows get dO * w_k with
w_k = 1/K (exact in bf16 for K = 2, 4), so the K unpacked losses add up to the
packed one.  Then, exactly:
  * O and dQ, dK, dV at every response position equal the unpacked row k's;
  * O at prompt positions equals any unpacked row's prompt O;
  * dQ, dK, dV at prompt positions equal the SUM over k of the unpacked rows'.
The packed GPU gradients are compared, per segment and at the gradient bar,
with those sums as the fp64 oracle computes them on the unpacked layout, and
with the same sums of the GPU's own unpacked run (the kernels then see every
response key tile and every prompt key tile in both layouts, so a prompt key
tile that stopped gathering after its first response, or a response key tile
that leaked into a sibling, fails one or the other).
"""
import numpy as np
import pytest
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import binding as pp
from paper_2602_24082_amd import workload as wl
from gradcheck import check_grad
from tolerances import lse_excess, o_excess

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _unpacked(P, lens):
    """The unpacked layout of one packed row and the packed token of each of its
    tokens: row k = prompt tokens 0..P-1, then response k's tokens."""
    K = len(lens)
    pack_u = wl.make_pack([P] * K, [[L] for L in lens])
    idx, is_prompt = [], []
    off = P
    for L in lens:
        idx += list(range(P)) + list(range(off, off + L))
        is_prompt += [True] * P + [False] * L
        off += L
    return pack_u, np.asarray(idx), np.asarray(is_prompt)


def _fold(pack_u, idx, is_prompt, x_u, T):
    """Packed-layout tensor from unpacked rows: response positions copied,
    prompt positions summed over the K rows."""
    out = np.zeros((T,) + x_u.shape[1:])
    np.add.at(out, idx[is_prompt], x_u[is_prompt])
    out[idx[~is_prompt]] = x_u[~is_prompt]
    return out


@pytest.mark.parametrize("P,lens,hq,hkv", [
    (300, [70, 1, 129, 64], 8, 2),      # a one-token response; responses straddle key tiles
    (700, [200, 33], 16, 2),            # G = 8, long prompt, K = 2
    (129, [128, 127, 1, 256], 4, 4),    # prompt one past a tile, MHA
])
def test_prompt_keys_gather_all_responses(P, lens, hq, hkv):
    d = 128
    K = len(lens)
    w = 1.0 / K
    pack = wl.make_pack([P], [lens])
    T = pack.total_tokens
    print(f"case gather P={P} lens={lens} hq={hq} hkv={hkv}", flush=True)
    q, k, v, do = wl.qkv(pack, hq, hkv, d, 5000 + P, torch.bfloat16, device="cpu")
    pack_u, idx, is_prompt = _unpacked(P, lens)
    qu, ku, vu = q[idx], k[idx], v[idx]
    scale_rows = torch.where(torch.from_numpy(is_prompt), torch.tensor(w), torch.tensor(1.0))
    dou = (do[idx].float() * scale_rows[:, None, None]).to(torch.bfloat16)  # exact: w is a power of 2
    assert torch.equal(dou[~torch.from_numpy(is_prompt)], do[idx][~torch.from_numpy(is_prompt)])

    # packed, on the GPU
    qg, kg, vg, dog = (x.to(DEV) for x in (q, k, v, do))
    o, lse = pp.pp_attn_fwd(pack, qg, kg, vg)
    dq, dk, dv = pp.pp_attn_bwd(pack, qg, kg, vg, o, lse, dog)
    # unpacked, on the GPU
    qug, kug, vug, doug = (x.to(DEV) for x in (qu, ku, vu, dou))
    ou, lseu = pp.pp_attn_fwd(pack_u, qug, kug, vug)
    dqu, dku, dvu = pp.pp_attn_bwd(pack_u, qug, kug, vug, ou, lseu, doug)
    torch.cuda.synchronize()
    npy = lambda t: t.double().cpu().numpy()

    # the oracle on the unpacked layout
    args_u = pack_u.oracle_args()
    qn, kn, vn, don = (x.double().numpy() for x in (qu, ku, vu, dou))
    O_u, L_u = orc.attn_fwd(*args_u, qn, kn, vn)
    dq_u, dk_u, dv_u = orc.attn_bwd(*args_u, qn, kn, vn, don)

    # forward: response positions are the unpacked rows'; the prompt rows of every
    # unpacked row agree with the packed prompt
    resp = idx[~is_prompt]
    o_c, l_c = npy(o), npy(lse)
    assert o_excess(o_c[resp], O_u[~is_prompt], True) <= 0
    assert lse_excess(l_c[:, resp], L_u[:, ~is_prompt]) <= 0
    for kk in range(K):
        rows = slice(kk * P + sum(lens[:kk]), kk * P + sum(lens[:kk]) + P)
        assert o_excess(o_c[:P], O_u[rows], True) <= 0
        assert lse_excess(l_c[:, :P], L_u[:, rows]) <= 0

    # backward: prompt gradients are the sums over the K unpacked rows
    for name, got, ref_u, gpu_u in (("dq", dq, dq_u, dqu), ("dk", dk, dk_u, dku), ("dv", dv, dv_u, dvu)):
        g = npy(got)
        want = _fold(pack_u, idx, is_prompt, ref_u, T)
        worst = check_grad(pack, name + " vs oracle (unpacked, folded)", g, want)
        want_gpu = _fold(pack_u, idx, is_prompt, npy(gpu_u), T)
        worst_gpu = check_grad(pack, name + " vs GPU (unpacked, folded)", g, want_gpu)
        print(f"  {name}: worst rel. Frobenius vs oracle {worst:.3e}, vs GPU unpacked {worst_gpu:.3e}",
              flush=True)
    # the prompt keys' gradients are not those of any single response: with the
    # other responses' contributions removed, they miss the bar by far
    dk_one = _fold(pack_u, idx[:P + lens[0]], is_prompt[:P + lens[0]], dk_u[:P + lens[0]], T)
    g = npy(dk)[:P]
    assert np.linalg.norm(g - dk_one[:P]) / np.linalg.norm(dk_one[:P]) > 0.1
