"""GPU parity of the rotary position embedding on packed position IDs (R19).

pp_rope (standalone) against the oracle's fp64 rotation, and the fused
pp_attn_fwd_rope / pp_attn_bwd_rope against the oracle's attention composed
with the rotation (attn_fwd_rope / attn_bwd_rope) on the inputs the kernels see.

Tolerances:
  rotated values  |y - y_ref| <= 2^-8 |y_ref| + 4e-6 max|x|   (bf16: one rounding
                  of the fp32 result, 2^-9 relative, plus fp32 products and
                  sine/cosine good to ~1e-7)
                  |y - y_ref| <= 4e-6 max|x|                  (fp32 outputs)
  O, LSE, dQ, dK, dV  the attention tolerances (tolerances.py, gradcheck.py: O max-abs
                  <= 1e-2 beyond its bf16 rounding, LSE within 2e-4 + 2^-16 |LSE|,
                  gradients relative Frobenius <= 2e-2 on the whole tensor and on every
                  prompt and response); dq and dk are w.r.t. the un-rotated q, k

The rotated queries and keys are bf16 activations, as in a bf16 model: the
kernels attend with the rotation rounded to bf16.  As for every bf16 input, the
oracle's attention runs on the values the kernels see -- the oracle's fp64
rotation rounded to bf16 (for fp32 callers: of the bf16-rounded q, since
attention inputs are rounded first) -- and its gradients are carried back
through the exact inverse rotation.  The rotated tensors themselves are checked
against the exact fp64 rotation.
"""
import numpy as np
import pytest
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import binding as pp
from paper_2602_24082_amd import workload as wl
from gradcheck import check_grad
from tolerances import lse_excess, o_excess, rope_lse_slack

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _rel_fro(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30)


def _check_rot(got, ref, x_absmax, bf16):
    got = got.double().cpu().numpy()
    err = np.abs(got - ref)
    bound = (2.0 ** -8 * np.abs(ref) if bf16 else 0.0) + 4e-6 * x_absmax
    assert np.isfinite(got).all()
    assert (err <= bound).all(), float((err - bound).max())


PACKS = [
    ("ragged", lambda: wl.make_pack([300, 0, 129, 5], [[70, 45], [33, 64], [1, 0, 200], [130]], pad=[3, 0, 0, 17])),
    ("long_prefix", lambda: wl.make_pack([6000, 2100], [[200, 64], [256, 1, 90]], pad=[0, 11])),
]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("name,mk", PACKS)
@pytest.mark.parametrize("d,base", [(128, 500000.0), (64, 10000.0)])
def test_rope_standalone(dtype, name, mk, d, base):
    pack = mk()
    # heads go through the kernel four at a time: 9 = two groups and one left over
    H = 9 if d == 128 else 3
    print(f"case rope {name} T={pack.total_tokens} H={H} d={d} base={base} {dtype}", flush=True)
    x = wl.randn((pack.total_tokens, H, d), 4321, dtype, "cpu")
    xn = x.double().numpy()
    args = pack.oracle_args()
    ref = orc.pack_rope(*args, xn, base)
    y = pp.pp_rope(pack, x.to(DEV), base)
    _check_rot(y, ref, np.abs(xn).max(), dtype == torch.bfloat16)
    # inverse, in place, on the rotated output
    back = y.clone()
    pp.pp_rope(pack, back, base, inverse=True, out=back)
    ref_back = orc.pack_rope(*args, y.double().cpu().numpy(), base, inverse=True)
    _check_rot(back, ref_back, np.abs(xn).max(), dtype == torch.bfloat16)


def _check_fused(pack, hq, hkv, d, base, dtype, seed, store_ds=False):
    print(f"case attn_rope T={pack.total_tokens} hq={hq} hkv={hkv} d={d} base={base} {dtype} seed={seed}"
          f" store_ds={store_ds}", flush=True)
    q, k, v, do = wl.qkv(pack, hq, hkv, d, seed, dtype, device="cpu")
    qg, kg, vg, dog = (x.to(DEV) for x in (q, k, v, do))
    o, lse, q_rot, k_rot = pp.pp_attn_fwd_rope(pack, qg, kg, vg, base)
    args = pack.oracle_args()
    # the kernels attend with bf16 q (fp32 callers are rounded first), as in the plain path
    qn = q.to(torch.bfloat16).double().numpy() if dtype == torch.float32 else q.double().numpy()
    kn, vn, don = (x.double().numpy() for x in (k, v, do))
    qr_ref = orc.pack_rope(*args, qn, base)
    kr_ref = orc.pack_rope(*args, kn, base)
    to_bf = lambda a: torch.from_numpy(a).to(torch.bfloat16).double().numpy()
    qr_b, kr_b = to_bf(qr_ref), to_bf(kr_ref)
    O_ref, L_ref = orc.attn_fwd(*args, qr_b, kr_b, vn)
    o_c, l_c = o.double().cpu().numpy(), lse.double().cpu().numpy()
    assert np.isfinite(o_c).all() and np.isfinite(l_c).all()
    assert o_excess(o_c, O_ref, dtype == torch.bfloat16) <= 0, np.abs(o_c - O_ref).max()
    slack = rope_lse_slack(pack, qr_ref, kr_ref, 4e-6 * np.abs(qn).max(), 4e-6 * np.abs(kn).max())
    assert lse_excess(l_c, L_ref, slack) <= 0, np.abs(l_c - L_ref).max()
    bf = dtype == torch.bfloat16
    _check_rot(q_rot, qr_ref, np.abs(qn).max(), bf)
    _check_rot(k_rot, kr_ref, np.abs(kn).max(), bf)
    dq, dk, dv = pp.pp_attn_bwd_rope(pack, q_rot, k_rot, vg, o, lse, dog, base, store_ds=store_ds)
    dqr, dkr, dv_r = orc.attn_bwd(*args, qr_b, kr_b, vn, don)
    dq_r = orc.pack_rope(*args, dqr, base, inverse=True)
    dk_r = orc.pack_rope(*args, dkr, base, inverse=True)
    for nm, got, ref in (("dq", dq, dq_r), ("dk", dk, dk_r), ("dv", dv, dv_r)):
        g = got.double().cpu().numpy()
        assert np.isfinite(g).all(), nm
        check_grad(pack, nm, g, ref)
    return (qg, kg, vg, dog), (o, lse, q_rot, k_rot), (dq, dk, dv)


@pytest.mark.parametrize("store_ds", [False, True])
@pytest.mark.parametrize("d,hq,hkv", [(128, 8, 2), (64, 4, 4)])
def test_fused_rope_attention_matches_oracle(d, hq, hkv, store_ds):
    """Both backward modes: the stored-dS dQ pass rotates its gradient back too."""
    pack = wl.make_pack([300, 0, 129, 5, 64], [[70, 45], [33, 64], [1, 0, 200], [130], [64, 64]],
                        pad=[3, 0, 0, 17, 0])
    _check_fused(pack, hq, hkv, d, 500000.0, torch.bfloat16, 77, store_ds=store_ds)


def test_fused_rope_attention_fp32_tiny_config():
    cfg = wl.TINY_FP32
    pack = wl.config_pack(cfg)
    _check_fused(pack, cfg.hq, cfg.hkv, cfg.head_dim, 10000.0, torch.float32, 78)


def test_fused_rope_long_positions():
    """Positions past 6000 (long shared prefix): the fp64 angle reduction keeps
    the rotation exact enough for the attention tolerances."""
    pack = wl.make_pack([6144, 2048], [[200, 64], [256, 90]])
    _check_fused(pack, 2, 1, 128, 1000000.0, torch.bfloat16, 79)


def test_fused_equals_rope_then_attention():
    """The fused forward attends exactly like pp_rope followed by pp_attn_fwd
    (same rotated bf16 queries and keys), and the fused backward's dq, dk equal
    pp_attn_bwd's gradients rotated back by pp_rope(inverse)."""
    pack = wl.make_pack([500, 77], [[100, 28, 300], [64, 64]], pad=[0, 5])
    base = 500000.0
    (qg, kg, vg, dog), (o, lse, q_rot, k_rot), (dq, dk, dv) = _check_fused(pack, 8, 2, 128, base,
                                                                          torch.bfloat16, 80)
    qr2 = pp.pp_rope(pack, qg, base)
    kr2 = pp.pp_rope(pack, kg, base)
    assert (qr2.float() - q_rot.float()).abs().max().item() <= 2.0 ** -7 * qr2.float().abs().max().item()
    assert torch.equal(kr2, k_rot)
    o2, lse2 = pp.pp_attn_fwd(pack, qr2, kr2, vg)
    assert (o2.float() - o.float()).abs().max().item() <= 1e-2
    dq2, dk2, dv2 = pp.pp_attn_bwd(pack, q_rot, k_rot, vg, o, lse, dog)
    assert torch.equal(dv2, dv)
    dq2 = pp.pp_rope(pack, dq2, base, inverse=True)
    dk2 = pp.pp_rope(pack, dk2, base, inverse=True)
    for a, b in ((dq, dq2), (dk, dk2)):
        assert _rel_fro(a.double().cpu().numpy(), b.double().cpu().numpy()) <= 1e-2
