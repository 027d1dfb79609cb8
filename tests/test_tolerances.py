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


def test_fp32_lse_within_the_lse_bar():
    """The LSE bar (tolerances.py) holds for log-sum-exp computed in fp32 from the
    bf16 inputs -- scores summed in fp32, the exponentials in fp32 and summed in
    fp32 in key order -- on a seeded pack with an 1100-token row, and is not so
    loose that an error of one part in 1e3 would pass."""
    from tolerances import lse_excess
    pack = wl.make_pack([900, 60], [[150, 64], [33, 40, 17]])
    hq, hkv, d = 4, 2, 128
    G = hq // hkv
    q, k, _, _ = wl.qkv(pack, hq, hkv, d, 2077, torch.bfloat16, device="cpu")
    args = pack.oracle_args()
    qn, kn = q.double().numpy(), k.double().numpy()
    _, L = orc.attn_fwd(*args, qn, kn, kn)
    q32, k32 = q.float().numpy(), k.float().numpy()
    emul = np.zeros_like(L)
    tau = np.float32(1.0 / np.sqrt(d))
    for b in range(pack.num_rows):
        r0, T = int(pack.row_start[b]), int(pack.row_start[b + 1] - pack.row_start[b])
        K = int(pack.num_resp[b])
        M = orc.row_mask(T, int(pack.prompt_len[b]), pack.resp_off[b, :K], pack.resp_len[b, :K])
        for h in range(hq):
            S = (q32[r0:r0 + T, h] @ k32[r0:r0 + T, h // G].T) * tau
            S = np.where(M, S, np.float32(-np.inf)).astype(np.float32)
            m = S.max(axis=1)
            E = np.exp(S - m[:, None]).astype(np.float32)
            l = np.cumsum(E, axis=1, dtype=np.float32)[:, -1]
            emul[h, r0:r0 + T] = (m + np.log(l)).astype(np.float32)
    assert lse_excess(emul, L) <= 0
    assert lse_excess(L + 1e-3 * np.abs(L).max(), L) > 0


def test_rope_lse_slack_covers_rounding_flips():
    """Attention on the bf16 rounding of a rotation that is off by up to `err`
    (as an fp32 rotation is) against attention on the rounding of the exact
    rotation: the LSE difference exceeds the plain bar and stays inside the bar
    widened by rope_lse_slack."""
    from tolerances import bf16_rounding_ambiguity, lse_excess, rope_lse_slack
    pack = wl.make_pack([300, 77], [[100, 28, 60], [64, 64]], pad=[0, 5])
    hq, hkv, d, base = 4, 2, 64, 500000.0
    q, k, _, _ = wl.qkv(pack, hq, hkv, d, 4040, torch.bfloat16, device="cpu")
    args = pack.oracle_args()
    qr = orc.pack_rope(*args, q.double().numpy(), base)
    kr = orc.pack_rope(*args, k.double().numpy(), base)
    eq, ek = 4e-6 * np.abs(qr).max(), 4e-6 * np.abs(kr).max()
    rng = np.random.default_rng(9)
    qp = qr + rng.uniform(-eq, eq, qr.shape)
    kp = kr + rng.uniform(-ek, ek, kr.shape)
    to_bf = lambda a: torch.from_numpy(a).to(torch.bfloat16).double().numpy()
    assert (to_bf(qp) != to_bf(qr)).any() and (to_bf(kp) != to_bf(kr)).any()
    assert bf16_rounding_ambiguity(qr, eq).any()
    _, L_exact = orc.attn_fwd(*args, to_bf(qr), to_bf(kr), to_bf(kr))
    _, L_pert = orc.attn_fwd(*args, to_bf(qp), to_bf(kp), to_bf(kr))
    slack = rope_lse_slack(pack, qr, kr, eq, ek)
    assert lse_excess(L_pert, L_exact) > 0          # the flips do exceed the plain bar
    assert lse_excess(L_pert, L_exact, slack) <= 0  # and the slack covers them


def test_fp32_lse_slack_covers_input_rounding():
    """fp32 q, k rounded to bf16 (as the kernels do for fp32 callers): the LSE
    change exceeds the plain bar on the tiny fp32 workload and stays inside the
    bar widened by fp32_lse_slack."""
    from tolerances import fp32_lse_slack, lse_excess
    cfg = wl.TINY_FP32
    pack = wl.config_pack(cfg)
    q, k, _, _ = wl.qkv(pack, cfg.hq, cfg.hkv, cfg.head_dim, 11, torch.float32, device="cpu")
    args = pack.oracle_args()
    qn, kn = q.double().numpy(), k.double().numpy()
    _, L = orc.attn_fwd(*args, qn, kn, kn)
    _, L_b = orc.attn_fwd(*args, _bf16(qn), _bf16(kn), kn)
    assert lse_excess(L_b, L) > 0
    assert lse_excess(L_b, L, fp32_lse_slack(pack, qn, kn)) <= 0
