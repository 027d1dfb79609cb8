"""CPU checks of the forward-output bar (tests/tolerances.py).

The bar's helper is checked against torch's bf16 rounding, and the reason for
the bar is shown on the CPU: on the seeded random pack where the GPU reached
0.0113, attention computed exactly as the kernels do it -- probabilities rounded
to bf16 before the PV product, fp32-exact sums, O rounded to bf16 -- is itself
more than 1e-2 from the fp64 oracle, and within the bar.
"""
import numpy as np
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import workload as wl
from tolerances import O_BAR, bf16_half_ulp, o_excess


def _bf16(a):
    # float32 first: one rounding to bf16 of a value that float32 holds exactly
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).double().numpy()


def test_half_ulp_bounds_bf16_rounding():
    x = (np.random.default_rng(5).standard_normal(100000) * 6).astype(np.float32)
    err = np.abs(_bf16(x) - x)
    hu = bf16_half_ulp(x)
    assert (err <= hu).all()
    assert (err / hu).max() > 0.99  # and it is reached
    assert bf16_half_ulp(2.57) == 2.0 ** -7 and bf16_half_ulp(1.0) == 2.0 ** -8 and bf16_half_ulp(0.0) == 0


def test_bf16_arithmetic_needs_the_rounding_allowance():
    # the seeded random pack of the GPU sweep (seed 6): 3 rows, 16/2 heads, d 128
    pack = wl.make_pack([240, 95, 162], [[50], [103], [64, 87, 122]], pad=[14, 11, 1])
    hq, hkv, d = 16, 2, 128
    G = hq // hkv
    q, k, v, _ = wl.qkv(pack, hq, hkv, d, 2006, torch.bfloat16, device="cpu")
    args = pack.oracle_args()
    qn, kn, vn = (x.double().numpy() for x in (q, k, v))
    O, _ = orc.attn_fwd(*args, qn, kn, vn)
    emul = np.zeros_like(O)
    tau = 1.0 / np.sqrt(d)
    for b in range(pack.num_rows):
        r0, T = int(pack.row_start[b]), int(pack.row_start[b + 1] - pack.row_start[b])
        K = int(pack.num_resp[b])
        M = orc.row_mask(T, int(pack.prompt_len[b]), pack.resp_off[b, :K], pack.resp_len[b, :K])
        for h in range(hq):
            S = np.where(M, tau * qn[r0:r0 + T, h] @ kn[r0:r0 + T, h // G].T, -np.inf)
            m = S.max(axis=1, keepdims=True)
            m[~np.isfinite(m)] = 0.0
            P = np.exp(S - m)
            l = P.sum(axis=1, keepdims=True)
            l[l == 0] = 1.0
            emul[r0:r0 + T, h] = _bf16((_bf16(P) @ vn[r0:r0 + T, h // G]) / l)
    worst = np.abs(emul - O).max()
    assert worst > O_BAR                   # a flat 1e-2 fails the prescribed arithmetic
    assert o_excess(emul, O, True) <= 0    # the bar of R21 holds
