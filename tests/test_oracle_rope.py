"""Pins of the oracle's rotary position embedding on packed position IDs (R19).

The paper requires that packed tokens keep the position IDs they have in the
unpacked layout (Sec. 3.2).  With rotary embeddings that decides every score,
so the strongest pin is again the unpacked equivalence: packed attention of
rotated queries/keys equals each (prompt, response_k) sequence rotated with its
own positions 0..P+L-1 and run through torch's causal attention.  The rotation
itself is pinned by the geometry of a plane rotation (d = 2, d = 4 written out),
by the complex-number form of the same map (an independent formulation through
torch's complex arithmetic), by the relative-position property of the scores,
and by finite differences of the gradients.
"""
import math

import numpy as np
import pytest
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import workload as wl


def _rand(shape, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(*shape, generator=g, dtype=torch.float64)


def test_d2_is_a_counter_clockwise_plane_rotation_by_the_position():
    """d = 2 has one frequency (w_0 = 1): the unit vector e_0 at position p goes
    to (cos p, sin p) and e_1 to (-sin p, cos p)."""
    for p in (0, 1, 2, 7, 1000):
        y0 = orc.rope(np.array([[[1.0, 0.0]]]), [p], 10000.0)[0, 0]
        y1 = orc.rope(np.array([[[0.0, 1.0]]]), [p], 10000.0)[0, 0]
        assert np.allclose(y0, [math.cos(p), math.sin(p)], atol=1e-12)
        assert np.allclose(y1, [-math.sin(p), math.cos(p)], atol=1e-12)


def test_d4_pairs_halves_with_the_stated_frequencies():
    """d = 4: pair 0 is (x0, x2) at frequency 1, pair 1 is (x1, x3) at frequency
    base^(-1/2); the interleaved pairing (x0, x1) would fail this."""
    base, p = 400.0, 3
    w1 = 1.0 / math.sqrt(base)
    y = orc.rope(np.array([[[0.0, 1.0, 0.0, 0.0]]]), [p], base)[0, 0]
    assert np.allclose(y, [0.0, math.cos(p * w1), 0.0, math.sin(p * w1)], atol=1e-12)
    y = orc.rope(np.array([[[1.0, 0.0, 0.0, 0.0]]]), [p], base)[0, 0]
    assert np.allclose(y, [math.cos(p), 0.0, math.sin(p), 0.0], atol=1e-12)


def test_matches_complex_multiplication():
    """Pair j as the complex number x_j + i x_{j+d/2}, multiplied by
    exp(i p w_j) (torch complex arithmetic, an independent formulation)."""
    n, H, d, base = 9, 3, 16, 10000.0
    x = _rand((n, H, d), 1)
    pos = torch.tensor([0, 1, 5, 17, 100, 4095, 4096, 8191, 123456], dtype=torch.float64)
    w = torch.tensor([base ** (-2.0 * j / d) for j in range(d // 2)], dtype=torch.float64)
    z = torch.complex(x[..., : d // 2], x[..., d // 2:])
    rot = torch.polar(torch.ones(n, 1, d // 2, dtype=torch.float64), (pos[:, None] * w[None, :])[:, None, :])
    zz = z * rot
    ref = torch.cat([zz.real, zz.imag], dim=-1).numpy()
    assert np.abs(orc.rope(x.numpy(), pos.numpy(), base) - ref).max() < 1e-12


def test_inverse_undoes_and_norms_are_kept():
    x = _rand((6, 2, 8), 2).numpy()
    pos = np.array([0, 3, 9, 50, 511, 7000])
    y = orc.rope(x, pos, 500000.0)
    assert np.abs(orc.rope(y, pos, 500000.0, inverse=True) - x).max() < 1e-12
    # each pair keeps its length
    n1 = x[..., :4] ** 2 + x[..., 4:] ** 2
    n2 = y[..., :4] ** 2 + y[..., 4:] ** 2
    assert np.abs(n1 - n2).max() < 1e-12
    # position 0 is the identity
    assert np.abs(orc.rope(x, np.zeros(6, int), 10.0) - x).max() == 0.0


def test_scores_depend_only_on_relative_position():
    """<rope(q, m), rope(k, n)> is unchanged when m and n shift together."""
    q = _rand((1, 1, 32), 3).numpy()
    k = _rand((1, 1, 32), 4).numpy()
    base = 10000.0
    for m, n in ((5, 2), (100, 37), (4000, 10)):
        ref = float((orc.rope(q, [m], base) * orc.rope(k, [n], base)).sum())
        for s in (1, 17, 1000):
            got = float((orc.rope(q, [m + s], base) * orc.rope(k, [n + s], base)).sum())
            assert abs(got - ref) < 1e-9 * max(1.0, abs(ref))


def _causal_sdpa(q, k, v, G, scale):
    kk = k.repeat_interleave(G, dim=1)
    vv = v.repeat_interleave(G, dim=1)
    o = torch.nn.functional.scaled_dot_product_attention(
        q.transpose(0, 1), kk.transpose(0, 1), vv.transpose(0, 1), is_causal=True, scale=scale)
    return o.transpose(0, 1)


def _torch_rope(x, pos, base):
    """RoPE in torch (complex form) for the unpacked reference sequences."""
    d = x.shape[-1]
    w = torch.tensor([base ** (-2.0 * j / d) for j in range(d // 2)], dtype=torch.float64)
    ang = pos.to(torch.float64)[:, None] * w[None, :]
    z = torch.complex(x[..., : d // 2], x[..., d // 2:]) * torch.polar(torch.ones_like(ang), ang)[:, None, :]
    return torch.cat([z.real, z.imag], dim=-1)


@pytest.mark.parametrize("P,lens,hq,hkv", [(5, [3, 4], 2, 1), (4, [1, 6, 2], 4, 2), (6, [0, 3], 2, 2)])
def test_packed_rope_equals_unpacked_rope_fwd_and_grads(P, lens, hq, hkv):
    """Fact (a) with rotary embeddings: each unpacked (prompt, response_k)
    sequence uses its own positions 0..P+L-1, rotated in torch (complex form),
    and torch's causal attention; gradients flow back to the un-rotated q, k."""
    d, base = 8, 50.0
    G = hq // hkv
    scale = 1.0 / math.sqrt(d)
    pack = wl.make_pack([P], [lens])
    T = pack.total_tokens
    q, k, v, do = (_rand((T, hq, d), 11), _rand((T, hkv, d), 12), _rand((T, hkv, d), 13),
                   _rand((T, hq, d), 14))
    args = pack.oracle_args()
    O, LSE, qr, kr = orc.attn_fwd_rope(*args, q.numpy(), k.numpy(), v.numpy(), base)
    dq, dk, dv = orc.attn_bwd_rope(*args, q.numpy(), k.numpy(), v.numpy(), do.numpy(), base)
    K = len(lens)
    gq, gk, gv = torch.zeros_like(q), torch.zeros_like(k), torch.zeros_like(v)
    offs = pack.resp_off[0].tolist()
    for kk, (o, L) in enumerate(zip(offs, lens)):
        idx = list(range(P)) + list(range(o, o + L))
        pos = torch.arange(P + L)
        qs = q[idx].clone().requires_grad_(True)
        ks = k[idx].clone().requires_grad_(True)
        vs = v[idx].clone().requires_grad_(True)
        out = _causal_sdpa(_torch_rope(qs, pos, base), _torch_rope(ks, pos, base), vs, G, scale)
        assert np.abs(out.detach().numpy() - O[idx]).max() < 1e-12
        wt = torch.ones(len(idx), 1, 1, dtype=torch.float64)
        wt[:P] = 1.0 / K
        (out * do[idx] * wt).sum().backward()
        gq[idx] += qs.grad
        gk[idx] += ks.grad
        gv[idx] += vs.grad
    assert np.abs(gq.numpy() - dq).max() < 1e-12
    assert np.abs(gk.numpy() - dk).max() < 1e-12
    assert np.abs(gv.numpy() - dv).max() < 1e-12


def test_rope_gradients_by_finite_differences():
    """Central differences of sum(dO * O) through the rotation (d = 4, padding)."""
    pack = wl.make_pack([3], [[2, 3]], pad=[1])
    T = pack.total_tokens
    args = pack.oracle_args()
    q, k, v, do = (_rand((T, 2, 4), 21).numpy(), _rand((T, 1, 4), 22).numpy(), _rand((T, 1, 4), 23).numpy(),
                   _rand((T, 2, 4), 24).numpy())
    base = 7.0
    dq, dk, _ = orc.attn_bwd_rope(*args, q, k, v, do, base)

    def f(qq, kk):
        return float((orc.attn_fwd_rope(*args, qq, kk, v, base)[0] * do).sum())

    eps = 1e-6
    for arr, grad, which in ((q, dq, 0), (k, dk, 1)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            a, b = arr.copy(), arr.copy()
            a[idx] += eps
            b[idx] -= eps
            fa = f(a, k) if which == 0 else f(q, a)
            fb = f(b, k) if which == 0 else f(q, b)
            num[idx] = (fa - fb) / (2 * eps)
        assert np.linalg.norm(num - grad) <= 1e-6 * max(1.0, np.linalg.norm(grad))
