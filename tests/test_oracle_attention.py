"""Pins of the oracle's packed attention, forward and backward.

The paper's central claim (Sec. 3.2) is that the packed row gives exactly the
results of the unpacked layout, where each (prompt, response_k) pair is its own
causal sequence.  These tests check the oracle against that claim with an
independent textbook routine (torch's scaled-dot-product attention and autograd
in fp64 on the CPU), plus closed forms, finite differences and symmetries.
"""
import math

import numpy as np
import pytest
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import workload as wl


def _causal_sdpa(q, k, v, G, scale):
    """Textbook causal attention over one sequence: q [T,Hq,d], k,v [T,Hkv,d]."""
    kk = k.repeat_interleave(G, dim=1)
    vv = v.repeat_interleave(G, dim=1)
    o = torch.nn.functional.scaled_dot_product_attention(
        q.transpose(0, 1), kk.transpose(0, 1), vv.transpose(0, 1), is_causal=True, scale=scale)
    return o.transpose(0, 1)


def _causal_lse(q, k, G, scale):
    kk = k.repeat_interleave(G, dim=1)
    s = torch.einsum("thd,uhd->htu", q, kk) * scale
    T = q.shape[0]
    s = s.masked_fill(~torch.tril(torch.ones(T, T, dtype=torch.bool)), -math.inf)
    return torch.logsumexp(s, dim=-1)


def _rand(shape, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(*shape, generator=g, dtype=torch.float64)


def _pack(P, lens, pad=0):
    return wl.make_pack([P], [lens], pad=[pad])


@pytest.mark.parametrize("P,lens,hq,hkv", [(5, [3, 4], 2, 1), (4, [1, 6, 2], 4, 2), (7, [2], 2, 2),
                                           (3, [0, 5], 2, 1), (6, [4, 4, 4, 4], 2, 2)])
def test_packed_equals_unpacked_fwd_and_grads(P, lens, hq, hkv):
    """Fact (a): packed == unpacked per (prompt, response_k), fwd and grads.

    The unpacked prompt rows of sequence k get dO * w_k with sum_k w_k = 1, so
    the sum of the unpacked losses equals the packed loss; then the packed
    prompt gradients equal the sums of the unpacked prompt gradients and the
    response gradients equal the unpacked ones, exactly (fp64)."""
    d = 8
    G = hq // hkv
    scale = 1.0 / math.sqrt(d)
    pack = _pack(P, lens)
    T = pack.total_tokens
    q, k, v, do = (_rand((T, hq, d), 1), _rand((T, hkv, d), 2), _rand((T, hkv, d), 3),
                   _rand((T, hq, d), 4))
    args = pack.oracle_args()
    O, LSE = orc.attn_fwd(*args, q.numpy(), k.numpy(), v.numpy())
    dq, dk, dv = orc.attn_bwd(*args, q.numpy(), k.numpy(), v.numpy(), do.numpy())

    K = len(lens)
    w = np.full(K, 1.0 / K) if K else np.zeros(0)
    gq = torch.zeros_like(q)
    gk = torch.zeros_like(k)
    gv = torch.zeros_like(v)
    offs = pack.resp_off[0].tolist()
    for kk, (o, L) in enumerate(zip(offs, lens)):
        idx = list(range(P)) + list(range(o, o + L))
        qs = q[idx].clone().requires_grad_(True)
        ks = k[idx].clone().requires_grad_(True)
        vs = v[idx].clone().requires_grad_(True)
        out = _causal_sdpa(qs, ks, vs, G, scale)
        lse = _causal_lse(qs.detach(), ks.detach(), G, scale)
        # forward: prompt rows and this response's rows
        assert np.abs(out.detach().numpy() - O[idx]).max() < 1e-12
        assert np.abs(lse.numpy() - LSE[:, idx]).max() < 1e-12
        wt = torch.ones(len(idx), 1, 1, dtype=torch.float64)
        wt[:P] = w[kk]
        (out * do[idx] * wt).sum().backward()
        gq[idx] += qs.grad
        gk[idx] += ks.grad
        gv[idx] += vs.grad
    if K == 0:
        pytest.skip("no response")
    # every token belongs to the prompt or exactly one response here
    assert np.abs(gq.numpy() - dq).max() < 1e-12
    assert np.abs(gk.numpy() - dk).max() < 1e-12
    assert np.abs(gv.numpy() - dv).max() < 1e-12


def test_single_response_is_plain_causal():
    """Fact (b): K = 1 reduces to plain causal attention over P + L tokens."""
    pack = _pack(9, [7])
    T = pack.total_tokens
    q, k, v = _rand((T, 4, 16), 10), _rand((T, 2, 16), 11), _rand((T, 2, 16), 12)
    O, LSE = orc.attn_fwd(*pack.oracle_args(), q.numpy(), k.numpy(), v.numpy())
    ref = _causal_sdpa(q, k, v, 2, 0.25)
    assert np.abs(ref.numpy() - O).max() < 1e-12
    assert np.abs(_causal_lse(q, k, 2, 0.25).numpy() - LSE).max() < 1e-12


def test_zero_prompt_is_independent_documents():
    """P = 0: each response is its own causal document."""
    lens = [4, 6, 3]
    pack = _pack(0, lens)
    T = pack.total_tokens
    q, k, v = _rand((T, 2, 8), 20), _rand((T, 2, 8), 21), _rand((T, 2, 8), 22)
    O, _ = orc.attn_fwd(*pack.oracle_args(), q.numpy(), k.numpy(), v.numpy())
    o = 0
    for L in lens:
        ref = _causal_sdpa(q[o:o + L], k[o:o + L], v[o:o + L], 1, 1 / math.sqrt(8))
        assert np.abs(ref.numpy() - O[o:o + L]).max() < 1e-12
        o += L


def test_softmax_rows_sum_to_one_and_padding_rows_zero():
    """Fact (c): every non-padding softmax row sums to 1; padding rows are 0."""
    pack = _pack(5, [3, 2], pad=3)
    T = pack.total_tokens
    q, k = _rand((T, 2, 8), 30), _rand((T, 1, 8), 31)
    for h in range(2):
        Pm, M = orc.attn_probs(*pack.oracle_args(), q.numpy(), k.numpy(), 0, h)
        sums = Pm.sum(axis=1)
        assert np.abs(sums[:10] - 1.0).max() < 1e-13
        assert (sums[10:] == 0).all()
        assert (Pm[~M] == 0).all()


def test_zero_queries_closed_form():
    """Q = 0 makes every visible score equal: O_i is the mean of the visible V
    rows and LSE_i = ln |vis(i)|, with |vis(i)| = i + 1 in the prompt and
    P + (i - o_k) + 1 in response k.  This pins the mask apart from the softmax."""
    P, lens = 6, [3, 5]
    pack = _pack(P, lens, pad=2)
    T = pack.total_tokens
    q = np.zeros((T, 2, 4))
    k = _rand((T, 1, 4), 40).numpy()
    v = _rand((T, 1, 4), 41).numpy()
    O, LSE = orc.attn_fwd(*pack.oracle_args(), q, k, v)
    offs = [6, 9]
    for i in range(T):
        if i < P:
            vis = list(range(i + 1))
        elif i < 9:
            vis = list(range(P)) + list(range(6, i + 1))
        elif i < 14:
            vis = list(range(P)) + list(range(9, i + 1))
        else:
            vis = []
        for h in range(2):
            if vis:
                assert np.abs(O[i, h] - v[vis, 0].mean(axis=0)).max() < 1e-13
                assert abs(LSE[h, i] - math.log(len(vis))) < 1e-13
            else:
                assert (O[i, h] == 0).all() and LSE[h, i] == 0


def test_gradients_finite_differences():
    """Central differences of sum(dO * O) in fp64 (relative error <= 1e-6)."""
    pack = wl.make_pack([3, 2], [[2, 3], [1]], pad=[1, 0])
    T = pack.total_tokens
    rng = np.random.default_rng(0)
    q = rng.standard_normal((T, 2, 4))
    k = rng.standard_normal((T, 1, 4))
    v = rng.standard_normal((T, 1, 4))
    do = rng.standard_normal((T, 2, 4))
    args = pack.oracle_args()
    dq, dk, dv = orc.attn_bwd(*args, q, k, v, do)

    def f(q_, k_, v_):
        O, _ = orc.attn_fwd(*args, q_, k_, v_)
        return float((O * do).sum())

    eps = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        for idx in np.ndindex(*x.shape):
            xp = x.copy(); xp[idx] += eps
            xm = x.copy(); xm[idx] -= eps
            a = (q, k, v)
            sel = {"q": 0, "k": 1, "v": 2}[name]
            ap = list(a); ap[sel] = xp
            am = list(a); am[sel] = xm
            num[idx] = (f(*ap) - f(*am)) / (2 * eps)
        err = np.linalg.norm(num - g) / max(np.linalg.norm(g), 1e-30)
        assert err < 1e-6, (name, err)
        # padding token (row 0, position 8) gets no gradient
        assert np.abs(g[8]).max() == 0.0


def test_permuting_responses_permutes_outputs():
    """Reordering the responses of a row reorders the outputs and changes
    nothing else (a response never sees a sibling)."""
    P, lens = 4, [3, 5, 2]
    pack = _pack(P, lens)
    T = pack.total_tokens
    q, k, v, do = (_rand((T, 2, 8), 50).numpy(), _rand((T, 1, 8), 51).numpy(),
                   _rand((T, 1, 8), 52).numpy(), _rand((T, 2, 8), 53).numpy())
    perm = [2, 0, 1]
    offs = pack.resp_off[0].tolist()
    idx = list(range(P))
    for p in perm:
        idx += list(range(offs[p], offs[p] + lens[p]))
    pack2 = _pack(P, [lens[p] for p in perm])
    args, args2 = pack.oracle_args(), pack2.oracle_args()
    O, L = orc.attn_fwd(*args, q, k, v)
    O2, L2 = orc.attn_fwd(*args2, q[idx], k[idx], v[idx])
    assert np.abs(O[idx] - O2).max() < 1e-13
    assert np.abs(L[:, idx] - L2).max() < 1e-13
    g = orc.attn_bwd(*args, q, k, v, do)
    g2 = orc.attn_bwd(*args2, q[idx], k[idx], v[idx], do[idx])
    for a, b in zip(g, g2):
        assert np.abs(a[idx] - b).max() < 1e-12


def test_rows_are_independent():
    """Two rows packed side by side give each row's results alone."""
    p1 = _pack(4, [2, 3])
    p2 = _pack(3, [5])
    both = wl.make_pack([4, 3], [[2, 3], [5]])
    T1 = p1.total_tokens
    T = both.total_tokens
    q, k, v = _rand((T, 2, 8), 60).numpy(), _rand((T, 2, 8), 61).numpy(), _rand((T, 2, 8), 62).numpy()
    O, L = orc.attn_fwd(*both.oracle_args(), q, k, v)
    Oa, La = orc.attn_fwd(*p1.oracle_args(), q[:T1], k[:T1], v[:T1])
    Ob, Lb = orc.attn_fwd(*p2.oracle_args(), q[T1:], k[T1:], v[T1:])
    assert np.abs(O[:T1] - Oa).max() == 0 and np.abs(O[T1:] - Ob).max() == 0
    assert np.abs(L[:, :T1] - La).max() == 0 and np.abs(L[:, T1:] - Lb).max() == 0
