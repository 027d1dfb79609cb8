"""The forward-output and log-sum-exp bars shared by the GPU parity tests.

O must lie within 1e-2 (max-abs) of the fp64 oracle.  A bf16 output cannot do
better than its own rounding, half a bf16 ulp of the exact value: bf16 keeps 8
significant bits, so its spacing at |O| in [2^e, 2^(e+1)) is 2^(e-7) and half of
it is 2^(e-8) -- 2^-7 at |O| in [2, 4), 2^-6 in [4, 8).  For bf16 outputs the bar
therefore sits on top of that rounding: at |O| in [4, 8) it is 1e-2 + 2^-6 =
0.0256.  The rest of the budget covers the bf16 probabilities of the PV product
(2^-9 relative per weight).  fp32 outputs keep the flat 1e-2.

LSE is computed in fp32 from bf16 q and k, so its error is set by fp32
arithmetic, not by bf16 rounding:
  * a score is a d-term dot product of exact bf16 products summed in fp32:
    at most d * 2^-24 * scale * sum_c |q_c k_c| (5.5e-5 for N(0,1) inputs at
    d = 128), and a few fp32 roundings of the score itself (2^-24 relative
    each, which matters only when scores are large);
  * each lane sums its share of exp2 terms in fp32 through at most ~16
    additions per key tile plus one per tile: below 1e-5 relative for the
    8192-key rows here, i.e. 1e-5 absolute on LSE;
  * exp2 and log2 on the transcendental unit are good to a few ulps.
The bar is 2e-4 absolute (about twice the worst case of the first two items at
unit-variance inputs) plus 2^-16 |LSE_ref| (256 fp32 ulps of the result, which
covers the rounding of large scores: the rising-score case reaches |LSE| ~ 1e3).

Where the kernels attend with inputs that differ from the oracle's, the bar
is widened by the first-order effect of that difference on LSE, computed from
the oracle's own inputs and probabilities (`lse_input_slack`): with dLSE_i/dq_ic
= scale sum_j P_ij k_jc and dLSE_i/dk_jc = scale P_ij q_ic, twice
scale sum_j P_ij sum_c (|dq_ic| |k_jc| + |q_ic| |dk_jc|).  Two cases:
  * fp32 callers: the kernels round q and k to bf16, the oracle takes them as
    given, so dq, dk are exactly bf16(x) - x (`fp32_lse_slack`);
  * the fused rotary path: the kernels attend with their own bf16 rounding of
    an fp32 rotation, the oracle with the bf16 rounding of its fp64 rotation.
    The two agree except for elements that lie within the rotation's error of
    a bf16 rounding boundary, where they may differ by one bf16 ulp
    (`rope_lse_slack`).
"""
import numpy as np
import torch

O_BAR = 1e-2
LSE_ABS = 2e-4
LSE_REL = 2.0 ** -16


def bf16_half_ulp(x):
    """Half the spacing of bfloat16 numbers (8 significant bits) at |x|: the most a
    correctly rounded bf16 value can differ from x."""
    a = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.exp2(e - 8), 0.0)


def o_excess(got, ref, bf16_out):
    """Largest amount by which |got - ref| exceeds the bar (<= 0 passes)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.size == 0:
        return 0.0
    allow = O_BAR + (bf16_half_ulp(ref) if bf16_out else 0.0)
    return float((np.abs(got - ref) - allow).max())


def lse_excess(got, ref, extra=0.0):
    """Largest amount by which |got - ref| exceeds the LSE bar (<= 0 passes);
    `extra` (scalar or per element) widens it."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.size == 0:
        return 0.0
    return float((np.abs(got - ref) - (LSE_ABS + LSE_REL * np.abs(ref)) - extra).max())


def _to_bf16(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64)).to(torch.bfloat16).double().numpy()


def bf16_rounding_ambiguity(x, err):
    """Per element: 0 where every value within `err` of x rounds to the same
    bf16 number, else the distance between the two candidates (one ulp)."""
    x = np.asarray(x, dtype=np.float64)
    return np.abs(_to_bf16(x + err) - _to_bf16(x - err))


def lse_input_slack(pack, q, k, dq, dk, scale=None):
    """Widening of the LSE bar [Hq, sumT] when the kernels attend with inputs
    that differ from the oracle's q, k ([sumT, H, d]) by at most dq, dk per
    element (see the module docstring)."""
    from oracle import pp_oracle as orc
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    d = q.shape[2]
    Hq, Hkv = q.shape[1], k.shape[1]
    G = Hq // Hkv
    tau = 1.0 / np.sqrt(d) if scale is None else scale
    args = pack.oracle_args()
    slack = np.zeros((Hq, pack.total_tokens))
    for b in range(pack.num_rows):
        r0, r1 = int(pack.row_start[b]), int(pack.row_start[b + 1])
        if r1 == r0:
            continue
        for h in range(Hq):
            if not (dq[r0:r1, h].any() or dk[r0:r1, h // G].any()):
                continue
            Pm, _ = orc.attn_probs(*args, q, k, b, h, scale=tau)
            kg, qh = np.abs(k[r0:r1, h // G]), np.abs(q[r0:r1, h])
            t_q = (dq[r0:r1, h] * (Pm @ kg)).sum(axis=1)
            t_k = (Pm * (qh @ dk[r0:r1, h // G].T)).sum(axis=1)
            slack[h, r0:r1] = 2.0 * tau * (t_q + t_k)
    return slack


def fp32_lse_slack(pack, q, k, scale=None):
    """LSE bar widening for fp32 q, k that the kernels round to bf16."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    return lse_input_slack(pack, q, k, np.abs(_to_bf16(q) - q), np.abs(_to_bf16(k) - k), scale)


def rope_lse_slack(pack, q_rot, k_rot, q_err, k_err, scale=None):
    """LSE bar widening for attention on bf16 roundings of rotated q, k whose
    exact values are q_rot, k_rot (fp64) and whose computed rotation may be off
    by q_err, k_err (absolute); the oracle attends with bf16(q_rot), bf16(k_rot)."""
    return lse_input_slack(pack, _to_bf16(q_rot), _to_bf16(k_rot), bf16_rounding_ambiguity(q_rot, q_err),
                           bf16_rounding_ambiguity(k_rot, k_err), scale)
