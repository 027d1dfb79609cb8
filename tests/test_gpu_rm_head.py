"""GPU parity of the reward-model head (pp_rm_scores / pp_rm_scores_bwd) against
the fp64 oracle (reading R17).

Tolerances from the arithmetic: a score is an fp32 dot product of H products
of exact inputs, so its error is bounded by ~H * 2^-24 * sum|h_i w_i| (held to
1e-5 * sum|h_i w_i|); dw sums one product per slot in fp32 (same bound over the
slots); dhidden is one fp32 product per element, rounded to the output dtype
(fp32: rtol 1e-6; bf16: rtol 2^-8).  Rows no slot reads must be exactly 0.
"""
import numpy as np
import pytest
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import binding as pp
from paper_2602_24082_amd import workload as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _inputs(pack, H, dtype, seed):
    hidden = wl.randn((pack.total_tokens, H), seed, dtype, "cpu")
    w = wl.randn((H,), seed + 1, dtype, "cpu", sigma=0.05)
    dsc = wl.randn((pack.num_rows, pack.max_resp), seed + 2, torch.float32, "cpu")
    return hidden, w, dsc


def _check(pack, H, dtype, seed, bias=0.5):
    print(f"rm head rows={pack.num_rows} T={pack.total_tokens} H={H} {dtype}", flush=True)
    hidden, w, dsc = _inputs(pack, H, dtype, seed)
    args = pack.oracle_args()
    hn, wn, gn = hidden.double().numpy(), w.double().numpy(), dsc.double().numpy()
    s = pp.pp_rm_scores(pack, hidden.to(DEV), w.to(DEV), bias).cpu().double().numpy()
    want = orc.rm_scores(*args, hn, wn, bias)
    rows = orc.rm_score_rows(*args)
    scale = np.zeros_like(want)
    for idx in np.ndindex(*rows.shape):
        if rows[idx] >= 0:
            scale[idx] = np.abs(hn[rows[idx]] * wn).sum() + abs(bias)
    assert (np.abs(s - want) <= 1e-5 * scale).all()
    dh, dw, db = pp.pp_rm_scores_bwd(pack, hidden.to(DEV), w.to(DEV), dsc.to(DEV))
    dh_r, dw_r, db_r = orc.rm_scores_grad(*args, hn, wn, gn)
    rt = 1e-6 if dtype == torch.float32 else 2.0 ** -8
    dh_c = dh.double().cpu().numpy()
    assert (np.abs(dh_c - dh_r) <= rt * np.abs(dh_r)).all()
    read = set(int(r) for r in rows.ravel() if r >= 0)
    unread = [r for r in range(pack.total_tokens) if r not in read]
    assert (dh_c[unread] == 0).all()
    dw_scale = sum(np.abs(gn[idx] * hn[rows[idx]]) for idx in np.ndindex(*rows.shape) if rows[idx] >= 0)
    assert (np.abs(dw.cpu().double().numpy() - dw_r) <= 1e-5 * dw_scale + 1e-30).all()
    assert abs(float(db) - db_r) <= 1e-5 * np.abs(gn).sum()


def test_rm_head_fp32_edges():
    # empty responses (read the last prompt token), a row with no prompt and an
    # empty response (no token: score 0), padding rows, hidden size not a
    # multiple of the workgroup
    pack = wl.make_pack([4, 0, 3, 1], [[2, 0, 3], [0, 2], [5], [0]], pad=[1, 2, 0, 3])
    _check(pack, 96, torch.float32, 301)


def test_rm_head_bf16_k4_full_size():
    cfg = wl.RM_K4
    _check(wl.config_pack(cfg), 4096, torch.bfloat16, 302)


def test_rm_head_bradley_terry_chain():
    # scores -> Bradley-Terry loss over all ranked pairs -> head gradients
    cfg = wl.RM_K4
    pack = wl.config_pack(cfg)
    hidden, w, _ = _inputs(pack, 1024, torch.float32, 303)
    hg, wg = hidden.to(DEV), w.to(DEV)
    s = pp.pp_rm_scores(pack, hg, wg, 0.0)
    loss, _, g = pp.pp_dpo_loss(pack.num_resp.tolist(), s, None, 1.0)
    dh, dw, db = pp.pp_rm_scores_bwd(pack, hg, wg, g)
    args = pack.oracle_args()
    s_r = orc.rm_scores(*args, hidden.double().numpy(), w.double().numpy())
    want, _, g_r = orc.pair_loss(pack.num_resp.tolist(), s_r, None, 1.0)
    assert abs(float(loss) - want) <= 1e-4 * abs(want)
    dh_r, dw_r, _ = orc.rm_scores_grad(*args, hidden.double().numpy(), w.double().numpy(), g_r)
    assert np.allclose(dw.cpu().double().numpy(), dw_r, rtol=1e-3, atol=1e-6 * np.abs(dw_r).max())
    assert np.allclose(dh.cpu().double().numpy(), dh_r, rtol=1e-3, atol=1e-6 * np.abs(dh_r).max())
