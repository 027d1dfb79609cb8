"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Tolerances (attention in bf16 MFMA with fp32 accumulation):
  O            max |O - O_ref| <= 1e-2 (+ half a bf16 ulp of O_ref for bf16 O; tolerances.py)
  LSE          max |lse - lse_ref| <= 2e-4 + 2^-16 |lse_ref|  (fp32 arithmetic; tolerances.py)
  dQ, dK, dV   ||g - g_ref||_F / ||g_ref||_F <= 2e-2, each, over the whole tensor AND
               over every prompt's and every response's rows (gradcheck.py)
  seq log-prob |s - s_ref| / |s_ref|                    <= 1e-4
  loss, dlogp  relative                                 <= 1e-4
The oracle runs on the inputs the kernels see: bf16 inputs as rounded, fp32
inputs as given (the kernels round them to bf16 at load, which the bf16
tolerances cover).
"""
import math

import numpy as np
import pytest
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import binding as pp
from paper_2602_24082_amd import workload as wl
from gradcheck import check_grad
from tolerances import fp32_lse_slack, lse_excess, o_excess

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
LP_TOL = 1e-4


def _inputs(pack, hq, hkv, d, dtype, seed):
    q, k, v, do = wl.qkv(pack, hq, hkv, d, seed, dtype, device="cpu")
    return q, k, v, do


def _poisoned_like(t):
    return torch.full_like(t, float("nan"))


def _check_attention(pack, hq, hkv, d, dtype, seed, check_bwd=True, inputs=None, grads=("dq", "dk", "dv"),
                     store_ds=False):
    """Forward and backward against the oracle; store_ds selects the backward
    mode whose dQ pass reads the dS stored by the key-major pass instead of
    recomputing S and dP."""
    print(f"case rows={pack.num_rows} T={pack.total_tokens} hq={hq} hkv={hkv} d={d} {dtype} seed={seed}"
          f" store_ds={store_ds}", flush=True)
    q, k, v, do = _inputs(pack, hq, hkv, d, dtype, seed) if inputs is None else inputs
    qg, kg, vg, dog = (x.to(DEV) for x in (q, k, v, do))
    T = pack.total_tokens
    o = _poisoned_like(qg)
    lse = torch.full((hq, T), float("nan"), device=DEV)
    pp.pp_attn_fwd(pack, qg, kg, vg, out=o, lse=lse)
    args = pack.oracle_args()
    qn, kn, vn, don = (x.double().numpy() for x in (q, k, v, do))
    O_ref, L_ref = orc.attn_fwd(*args, qn, kn, vn)
    o_c = o.double().cpu().numpy()
    l_c = lse.double().cpu().numpy()
    assert np.isfinite(o_c).all() and np.isfinite(l_c).all(), "unwritten output"
    assert o_excess(o_c, O_ref, dtype == torch.bfloat16) <= 0, np.abs(o_c - O_ref).max()
    # fp32 callers: the kernels attend with q, k rounded to bf16 (R11)
    slack = fp32_lse_slack(pack, qn, kn) if dtype == torch.float32 else 0.0
    assert lse_excess(l_c, L_ref, slack) <= 0, np.abs(l_c - L_ref).max()
    print(f"  max|dO| {np.abs(o_c - O_ref).max():.3e}  max|dLSE| {np.abs(l_c - L_ref).max():.3e}", flush=True)
    if not check_bwd:
        return
    dq, dk, dv = _poisoned_like(qg), _poisoned_like(kg), _poisoned_like(vg)
    pp.pp_attn_bwd(pack, qg, kg, vg, o, lse, dog, dq=dq, dk=dk, dv=dv, store_ds=store_ds)
    dq_r, dk_r, dv_r = orc.attn_bwd(*args, qn, kn, vn, don)
    out = {}
    for name, got, ref in (("dq", dq, dq_r), ("dk", dk, dk_r), ("dv", dv, dv_r)):
        g = got.double().cpu().numpy()
        out[name] = (g, ref)
        assert np.isfinite(g).all(), f"unwritten {name}"
        if name in grads:
            worst = check_grad(pack, name, g, ref)
            print(f"  {name}: worst whole/segment rel. Frobenius {worst:.3e}", flush=True)
    # padding rows are exactly zero
    seg = orc.pack_segment_ids(*args)
    pad = seg < 0
    if pad.any():
        assert (o_c[pad] == 0).all() and (l_c[:, pad] == 0).all()
        assert (dq.cpu().double().numpy()[pad] == 0).all()
        assert (dk.cpu().double().numpy()[pad] == 0).all()
        assert (dv.cpu().double().numpy()[pad] == 0).all()
    return out


@pytest.mark.parametrize("store_ds", [False, True])
def test_tiny_fp32_config(store_ds):
    """4 rows, 4 heads (MHA), d 64, fp32 inputs, K=2 (the tiny check config)."""
    cfg = wl.TINY_FP32
    _check_attention(wl.config_pack(cfg), cfg.hq, cfg.hkv, cfg.head_dim, torch.float32, 11, store_ds=store_ds)


@pytest.mark.parametrize("store_ds", [False, True])
@pytest.mark.parametrize("d", [64, 128])
def test_bf16_gqa_ragged(d, store_ds):
    """Several tiles per row, unaligned boundaries, padding, GQA 8/2."""
    pack = wl.make_pack([300, 0, 129, 5, 64], [[70, 45], [33, 64], [1, 0, 200], [130], [64, 64]],
                        pad=[3, 0, 0, 17, 0])
    _check_attention(pack, 8, 2, d, torch.bfloat16, 21 + d, store_ds=store_ds)


def test_bf16_k4_mha():
    pack = wl.make_pack([200, 57], [[31, 64, 1, 97], [128, 2, 300, 9]], pad=[0, 40])
    _check_attention(pack, 4, 4, 128, torch.bfloat16, 31)


@pytest.mark.parametrize("store_ds", [False, True])
def test_edge_cases(store_ds):
    """Single response (plain causal), empty prompt (document masking), one-token
    rows, empty rows, all-padding rows, rows shorter than one tile."""
    pack = wl.make_pack([0, 1, 7, 0, 129, 3, 0],
                        [[1], [], [0, 0], [], [], [1, 1, 1], [5, 6]],
                        pad=[0, 0, 0, 0, 0, 2, 0])
    _check_attention(pack, 4, 1, 64, torch.bfloat16, 41, store_ds=store_ds)
    pack = wl.make_pack([5, 0], [[], []], pad=[0, 9])  # all-padding second row
    _check_attention(pack, 2, 2, 128, torch.bfloat16, 42, store_ds=store_ds)


@pytest.mark.parametrize("seed", range(8))
def test_random_pack_sweep(seed):
    """Seeded random packs: prompt lengths 0-400 (the first row has none on two
    seeds: its responses are then separate documents), 0-4 responses of 0-260
    tokens, 0-20 padding tokens, GQA ratios 1, 2, 4 and 8, d 64 or 128; forward
    and all three gradients against the oracle (odd seeds: the stored-dS
    backward)."""
    rng = np.random.default_rng(1000 + seed)
    B = int(rng.integers(1, 5))
    P, L, pad = [], [], []
    for _ in range(B):
        k = int(rng.integers(0, 5))
        lens = [int(x) for x in rng.integers(0, 261, size=k)]
        p0 = int(rng.integers(0, 401))
        P.append(p0)
        L.append(lens)
        pad.append(int(rng.integers(0, 21)))
    if seed % 4 == 3:
        P[0], L[0] = 0, [17, 40]
    pack = wl.make_pack(P, L, pad=pad)
    hkv = int(rng.choice([1, 2, 4]))
    G = int(rng.choice([1, 2, 4, 8]))
    d = int(rng.choice([64, 128]))
    _check_attention(pack, hkv * G, hkv, d, torch.bfloat16, 2000 + seed, store_ds=bool(seed % 2))


def test_large_scores():
    """Scores with standard deviation 16 (q, k ~ N(0, 2) per element, d = 128):
    nearly one-hot softmax rows whose maximum jumps between key tiles, so the
    forward's lazily raised reference maximum is raised often.  V is halved so
    that the bf16 rounding of one dominant P (2^-9 relative) stays inside the
    1e-2 bound on O."""
    pack = wl.make_pack([300, 90], [[70, 45], [33, 64, 10]], pad=[3, 0])
    hq, hkv, d = 4, 2, 128
    q, k, v, do = _inputs(pack, hq, hkv, d, torch.bfloat16, 61)
    q = (q.float() * 2).to(torch.bfloat16)
    k = (k.float() * 2).to(torch.bfloat16)
    v = (v.float() * 0.5).to(torch.bfloat16)
    _check_attention(pack, hq, hkv, d, torch.bfloat16, 61, inputs=(q, k, v, do))


def test_scores_rising_along_the_row():
    """Every query's score grows by 0.2 per key position (plus small noise), so
    the running maximum rises by more than the rescale slack on every key tile
    and the softmax mass sits on each query's latest visible keys: the rescale
    branch runs on nearly every tile of the forward.

    O, LSE, dK and dV are held to the usual bars.  dQ is split by component.
    Components 1..d-1 are held to the usual bar.  Component 0 is the one every
    key shares with a value of up to ~1000: dQ_i0 = scale sum_j dS_ij k_j0 sums
    near-one-hot dS_ij (whose row sums are exactly 0) against those large k_j0,
    so the rounding of dS (2^-9 relative when it is rounded to bf16 for the
    MFMA, plus P times the 2^-9 rounding of O inside delta) is amplified far
    past a relative bar on the small result.  That component is held, element
    by element, to twice the bound this rounding gives:
        |err_i0| <= 2 scale sum_j 2^-9 (|dS_ij| + P_ij sum_c |dO_ic O_ic|) |k_j0|."""
    pack = wl.make_pack([300, 200], [[100, 130], [64, 97, 40]], pad=[0, 7])
    hq, hkv, d = 4, 2, 128
    q, k, v, do = _inputs(pack, hq, hkv, d, torch.bfloat16, 62)
    T = pack.total_tokens
    pos = torch.zeros(T)
    rs = np.asarray(pack.row_start)
    for b in range(pack.num_rows):
        pos[rs[b]:rs[b + 1]] = torch.arange(rs[b + 1] - rs[b], dtype=torch.float32)
    scale = 1.0 / math.sqrt(d)
    qf = q.float() * 0.05
    kf = k.float() * 0.05
    qf[:, :, 0] = 1.0
    kf[:, :, 0] = (0.2 / scale) * pos[:, None]
    q, k = qf.to(torch.bfloat16), kf.to(torch.bfloat16)
    v = (v.float() * 0.5).to(torch.bfloat16)
    res = _check_attention(pack, hq, hkv, d, torch.bfloat16, 62, inputs=(q, k, v, do), grads=("dk", "dv"))
    dq_g, dq_r = res["dq"]
    check_grad(pack, "dq[..., 1:]", dq_g[..., 1:], dq_r[..., 1:])
    args = pack.oracle_args()
    qn, kn, vn, don = (x.double().numpy() for x in (q, k, v, do))
    O, _ = orc.attn_fwd(*args, qn, kn, vn)
    G = hq // hkv
    worst = 0.0
    for b in range(pack.num_rows):
        r0, r1 = int(rs[b]), int(rs[b + 1])
        for h in range(hq):
            Pm, M = orc.attn_probs(*args, qn, kn, b, h)
            Vg, Kg = vn[r0:r1, h // G], kn[r0:r1, h // G]
            dOh, Oh = don[r0:r1, h], O[r0:r1, h]
            dS = Pm * (dOh @ Vg.T - (dOh * Oh).sum(axis=1)[:, None])
            rnd = 2.0 ** -9 * (np.abs(dS) + Pm * np.abs(dOh * Oh).sum(axis=1)[:, None])
            bound = 2 * scale * rnd @ np.abs(Kg[:, 0])
            err = np.abs(dq_g[r0:r1, h, 0] - dq_r[r0:r1, h, 0])
            assert (err <= bound + 1e-6).all(), (b, h, float((err - bound).max()))
            worst = max(worst, float((err / (bound + 1e-6)).max()))
    print(f"  dq[..., 0]: worst error / rounding bound {worst:.3f}", flush=True)


def test_g8_long_prefix_small():
    """64/8-style grouping (G=8) with a long prefix and short responses."""
    pack = wl.make_pack([700, 450], [[64, 100], [256, 70]])
    _check_attention(pack, 16, 2, 128, torch.bfloat16, 51)


@pytest.mark.parametrize("store_ds", [False, True])
def test_backward_is_deterministic(store_ds):
    pack = wl.make_pack([400, 150], [[100, 61], [33, 270]])
    q, k, v, do = (x.to(DEV) for x in _inputs(pack, 8, 2, 128, torch.bfloat16, 61))
    o, lse = pp.pp_attn_fwd(pack, q, k, v)
    g1 = pp.pp_attn_bwd(pack, q, k, v, o, lse, do, store_ds=store_ds)
    g2 = pp.pp_attn_bwd(pack, q, k, v, o, lse, do, store_ds=store_ds)
    o2, lse2 = pp.pp_attn_fwd(pack, q, k, v)
    assert torch.equal(o, o2) and torch.equal(lse, lse2)
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)


def test_stored_and_recompute_backward_agree():
    """The two backward modes take the same inputs to the same gradients: dV
    (which does not use delta) bit for bit, dQ and dK up to the rounding of
    delta's fp32 sum and of dS to bf16 (each mode forms dS in its own pass)."""
    pack = wl.make_pack([333, 90, 0], [[129, 64, 1, 40], [300], [65, 31]], pad=[5, 0, 11])
    q, k, v, do = (x.to(DEV) for x in _inputs(pack, 8, 2, 128, torch.bfloat16, 71))
    o, lse = pp.pp_attn_fwd(pack, q, k, v)
    s = pp.pp_attn_bwd(pack, q, k, v, o, lse, do, store_ds=True)
    r = pp.pp_attn_bwd(pack, q, k, v, o, lse, do)
    assert torch.equal(s[2], r[2])
    for a, b in zip(s[:2], r[:2]):
        a, b = a.double(), b.double()
        assert torch.isfinite(a).all()
        assert ((a - b).norm() / b.norm()).item() < 4e-3


# ---------------------------------------------------------------- log-prob / loss


def _check_logprob(pack, V, dtype, sigma, seed):
    print(f"logprob rows={pack.num_rows} T={pack.total_tokens} V={V} {dtype}", flush=True)
    T = pack.total_tokens
    logits = wl.randn((T, V), seed, dtype, "cpu", sigma=sigma)
    tokens = wl.randint((T,), V, seed + 1, "cpu")
    seq = torch.full((pack.num_rows, pack.max_resp), float("nan"), device=DEV)
    tok = torch.full((T,), float("nan"), device=DEV)
    pp.pp_seq_logprob(pack, logits.to(DEV), tokens.to(DEV), want_tok=True, seq=seq, tok=tok)
    ref_seq, ref_tok = orc.seq_logprob(*pack.oracle_args(), logits.double().numpy(), tokens.numpy())
    s = seq.double().cpu().numpy()
    t = tok.double().cpu().numpy()
    assert np.isfinite(s).all() and np.isfinite(t).all()
    nz = np.abs(ref_seq) > 0
    assert (s[~nz] == 0).all()
    rel = np.abs(s[nz] - ref_seq[nz]) / np.abs(ref_seq[nz])
    assert rel.max() <= LP_TOL, rel.max()
    assert np.abs(t - ref_tok).max() <= 1e-4 * max(1.0, np.abs(ref_tok).max())
    return s


def _random_logprob_pack(rng):
    B = int(rng.integers(1, 5))
    P, L, pad = [], [], []
    for _ in range(B):
        P.append(int(rng.integers(1, 200)))
        L.append([int(x) for x in rng.integers(0, 120, size=int(rng.integers(0, 5)))])
        pad.append(int(rng.integers(0, 9)))
    return wl.make_pack(P, L, pad=pad)


@pytest.mark.parametrize("seed", range(4))
def test_logprob_random_sweep(seed):
    """Seeded random packs and vocabularies (rows 16-byte aligned or not), bf16
    and fp32 logits, against the oracle's per-response log-probabilities."""
    rng = np.random.default_rng(3000 + seed)
    pack = _random_logprob_pack(rng)
    V = int(rng.choice([1000, 4099, 32000, 50257]))
    dtype = torch.bfloat16 if seed % 2 == 0 else torch.float32
    _check_logprob(pack, V, dtype, 3.0, 3100 + seed)


def test_logprob_tiny_fp32():
    cfg = wl.TINY_FP32
    _check_logprob(wl.config_pack(cfg), 1000, torch.float32, 2.0, 71)


def test_logprob_bf16_odd_vocab_and_edges():
    # vocab 4099: rows are not 16-byte aligned -> element path; empty responses
    pack = wl.make_pack([5, 1, 9], [[3, 0, 7], [1], [12, 40]], pad=[2, 0, 1])
    _check_logprob(pack, 4099, torch.bfloat16, 3.0, 72)
    _check_logprob(pack, 4096, torch.bfloat16, 3.0, 73)


def test_logprob_bf16_llama_vocab():
    pack = wl.make_pack([40, 17], [[9, 30, 2, 11], [25, 1, 0, 8]])
    _check_logprob(pack, 128256, torch.bfloat16, 3.0, 74)


def test_logprob_out_of_range_label_poisons_response():
    pack = wl.make_pack([4], [[3, 3]])
    V = 64
    logits = wl.randn((10, V), 80, torch.float32, "cpu")
    tokens = wl.randint((10,), V, 81, "cpu")
    tokens[5] = V + 3  # inside response 0
    seq = pp.pp_seq_logprob(pack, logits.to(DEV), tokens.to(DEV)).cpu()
    assert math.isnan(seq[0, 0]) and math.isfinite(seq[0, 1])


def _check_loss(num, pol, ref, beta):
    polg = torch.tensor(pol, dtype=torch.float32, device=DEV)
    refg = None if ref is None else torch.tensor(ref, dtype=torch.float32, device=DEV)
    loss, rows, grad = pp.pp_dpo_loss(num, polg, refg, beta)
    want, want_rows, want_g = orc.pair_loss(num, np.asarray(pol, np.float32).astype(np.float64),
                                            None if ref is None else np.asarray(ref, np.float32).astype(np.float64),
                                            beta)
    assert abs(float(loss) - want) <= LP_TOL * abs(want)
    assert np.allclose(rows.cpu().numpy(), want_rows, rtol=LP_TOL, atol=1e-7)
    assert np.allclose(grad.cpu().numpy(), want_g, rtol=LP_TOL, atol=1e-8)


def test_dpo_loss_and_bt_loss():
    rng = np.random.default_rng(90)
    _check_loss([2, 2, 2, 2], rng.standard_normal((4, 2)) * 30, rng.standard_normal((4, 2)) * 30, 0.1)
    _check_loss([4, 3, 1, 4, 0, 2], rng.standard_normal((6, 4)) * 10, None, 1.0)
    B = 700  # more rows than threads
    _check_loss(list(rng.integers(0, 5, B)), rng.standard_normal((B, 4)) * 5, rng.standard_normal((B, 4)) * 5, 0.5)
    for B in (256, 257):  # the last row count passed in the launch arguments, the first one staged
        _check_loss(list(rng.integers(0, 5, B)), rng.standard_normal((B, 4)) * 5, rng.standard_normal((B, 4)) * 5,
                    0.3)


def test_full_chain_tiny_config():
    """Tiny config end to end: policy and reference log-probs, then DPO at beta 0.1."""
    cfg = wl.TINY_FP32
    pack = wl.config_pack(cfg)
    s_pol = _check_logprob(pack, cfg.vocab, torch.float32, cfg.logit_sigma, 100)
    s_ref = _check_logprob(pack, cfg.vocab, torch.float32, cfg.logit_sigma, 200)
    _check_loss(pack.num_resp.tolist(), s_pol, s_ref, cfg.beta)
