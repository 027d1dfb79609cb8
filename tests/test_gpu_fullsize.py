"""Full-size GPU parity on sampled outputs.

The kernels run on whole batches of the benchmarked workloads, in the launch
configuration the benchmark times; the fp64 oracle then recomputes a sample
it can afford -- one row (rows are independent) and one kv-head group (heads
are independent), or single responses for the log-probabilities -- and the
two are compared element by element with the same tolerances as the small
parity tests, gradients also per prompt and per response (gradcheck.py).

Attention is sampled on the longest row of the 8B-shaped, reward-model and
DPO-chain batches (the longest prompt key ranges: their key tiles walk the most
query steps and gather the most responses) and on the shortest; on the
long-prefix batch, whose longest row (6348 tokens) would hold the oracle for
minutes, on the row of median length and the shortest.
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


def _row_pack(pack, b):
    K = int(pack.num_resp[b])
    return wl.make_pack([int(pack.prompt_len[b])], [pack.resp_len[b, :K].tolist()],
                        pad=[int(pack.row_lengths()[b]) - int(pack.prompt_len[b]) - int(pack.resp_len[b, :K].sum())])


def _pick_row(pack, which):
    n = pack.row_lengths()
    if which == "shortest":
        return int(np.argmin(n))
    if which == "longest":
        return int(np.argmax(n))
    return int(np.argsort(n, kind="stable")[len(n) // 2])  # median length


def _attention_sample(cfg, group, which, store_ds=False):
    pack = wl.config_pack(cfg)
    seed = wl.tensor_seed(cfg.index, 0)
    q, k, v, do = wl.qkv(pack, cfg.hq, cfg.hkv, cfg.head_dim, seed, torch.bfloat16, DEV)
    o, lse = pp.pp_attn_fwd(pack, q, k, v)
    dq, dk, dv = pp.pp_attn_bwd(pack, q, k, v, o, lse, do, store_ds=store_ds)
    torch.cuda.synchronize()
    b = _pick_row(pack, which)
    r0, r1 = int(pack.row_start[b]), int(pack.row_start[b + 1])
    G = cfg.hq // cfg.hkv
    hs = slice(group * G, (group + 1) * G)
    gs = slice(group, group + 1)
    print(f"{cfg.name}: {which} row {b} T={r1 - r0}, q-heads {hs.start}..{hs.stop - 1}, kv-head {group}"
          f" store_ds={store_ds}", flush=True)
    sub = lambda x, s: x[r0:r1, s].double().cpu().numpy()
    row = _row_pack(pack, b)
    args = row.oracle_args()
    O_ref, L_ref = orc.attn_fwd(*args, sub(q, hs), sub(k, gs), sub(v, gs))
    dq_r, dk_r, dv_r = orc.attn_bwd(*args, sub(q, hs), sub(k, gs), sub(v, gs), sub(do, hs))
    o_c = sub(o, hs)
    l_c = lse[hs, r0:r1].double().cpu().numpy()
    assert o_excess(o_c, O_ref, True) <= 0, np.abs(o_c - O_ref).max()
    assert lse_excess(l_c, L_ref) <= 0, np.abs(l_c - L_ref).max()
    print(f"  max|dO| {np.abs(o_c - O_ref).max():.3e}  max|dLSE| {np.abs(l_c - L_ref).max():.3e}", flush=True)
    for name, got, ref in (("dq", sub(dq, hs), dq_r), ("dk", sub(dk, gs), dk_r), ("dv", sub(dv, gs), dv_r)):
        worst = check_grad(row, name, got, ref)
        print(f"  {name}: worst whole/segment rel. Frobenius {worst:.3e}", flush=True)
    # nothing left unwritten anywhere in the batch
    for t in (o, lse, dq, dk, dv):
        assert torch.isfinite(t).all()


@pytest.mark.parametrize("which", ["longest", "shortest"])
def test_fullsize_llama3_8b_attention(which):
    _attention_sample(wl.LLAMA3_8B, group=3, which=which)


@pytest.mark.parametrize("which", ["longest", "shortest"])
def test_fullsize_rm_k4_attention(which):
    _attention_sample(wl.RM_K4, group=5, which=which)


@pytest.mark.parametrize("which", ["median", "shortest"])
def test_fullsize_long_prefix_attention(which):
    _attention_sample(wl.LONG_PREFIX, group=7, which=which)


@pytest.mark.parametrize("which", ["longest", "shortest"])
def test_fullsize_dpo_chain_attention(which):
    _attention_sample(wl.DPO_CHAIN, group=0, which=which)


@pytest.mark.parametrize("name,group,which", [("llama3_8b_gqa32x8_d128_k2", 6, "longest"),
                                              ("long_prefix_qwen72b_gqa64x8_d128", 2, "median"),
                                              ("dpo_chain_qwen72b_gqa64x8_d128_v152064", 5, "longest")])
def test_fullsize_attention_stored_ds(name, group, which):
    """The stored-dS backward on whole benchmarked batches (0.45 to 12 GB of dS)."""
    _attention_sample(wl.BY_NAME[name], group=group, which=which, store_ds=True)


def _attention_rope_sample(cfg, group, base):
    """The fused rotary path on a whole benchmarked batch; the oracle recomputes
    one row and one kv-head group on the bf16-rounded rotations the kernels
    attend with, and carries the gradients back through the exact rotation."""
    pack = wl.config_pack(cfg)
    seed = wl.tensor_seed(cfg.index, 0)
    q, k, v, do = wl.qkv(pack, cfg.hq, cfg.hkv, cfg.head_dim, seed, torch.bfloat16, DEV)
    o, lse, q_rot, k_rot = pp.pp_attn_fwd_rope(pack, q, k, v, base)
    dq, dk, dv = pp.pp_attn_bwd_rope(pack, q_rot, k_rot, v, o, lse, do, base)
    torch.cuda.synchronize()
    b = _pick_row(pack, "shortest")
    r0, r1 = int(pack.row_start[b]), int(pack.row_start[b + 1])
    G = cfg.hq // cfg.hkv
    hs = slice(group * G, (group + 1) * G)
    gs = slice(group, group + 1)
    print(f"{cfg.name} rope base {base}: row {b} T={r1 - r0}, kv-head {group}", flush=True)
    sub = lambda x, s: x[r0:r1, s].double().cpu().numpy()
    row = _row_pack(pack, b)
    args = row.oracle_args()
    qr = orc.pack_rope(*args, sub(q, hs), base)
    kr = orc.pack_rope(*args, sub(k, gs), base)
    for got, ref in ((sub(q_rot, hs), qr), (sub(k_rot, gs), kr)):
        assert (np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 4e-6 * np.abs(ref).max()).all()
    to_bf = lambda a: torch.from_numpy(a).to(torch.bfloat16).double().numpy()
    qb, kb = to_bf(qr), to_bf(kr)
    O_ref, L_ref = orc.attn_fwd(*args, qb, kb, sub(v, gs))
    dqr, dkr, dv_r = orc.attn_bwd(*args, qb, kb, sub(v, gs), sub(do, hs))
    assert o_excess(sub(o, hs), O_ref, True) <= 0, np.abs(sub(o, hs) - O_ref).max()
    slack = rope_lse_slack(row, qr, kr, 4e-6 * np.abs(sub(q, hs)).max(), 4e-6 * np.abs(sub(k, gs)).max())
    assert lse_excess(lse[hs, r0:r1].double().cpu().numpy(), L_ref, slack) <= 0
    for name, got, ref in (("dq", sub(dq, hs), orc.pack_rope(*args, dqr, base, inverse=True)),
                           ("dk", sub(dk, gs), orc.pack_rope(*args, dkr, base, inverse=True)),
                           ("dv", sub(dv, gs), dv_r)):
        check_grad(row, name, got, ref)
    for t in (o, lse, dq, dk, dv, q_rot, k_rot):
        assert torch.isfinite(t).all()


def test_fullsize_llama3_8b_attention_rope():
    _attention_rope_sample(wl.LLAMA3_8B, group=2, base=500000.0)


def test_fullsize_long_prefix_attention_rope():
    _attention_rope_sample(wl.LONG_PREFIX, group=4, base=1000000.0)


def _compact_response(pack, b, k, logits, tokens):
    """One response as its own pack: the predicting row P-1 then the rows that
    predict tokens 2..L, with the response's labels (the oracle's index rule
    maps the compact pack onto exactly these rows)."""
    r0 = int(pack.row_start[b])
    P = int(pack.prompt_len[b])
    o, L = int(pack.resp_off[b, k]), int(pack.resp_len[b, k])
    rows = [r0 + P - 1] + [r0 + o + j - 1 for j in range(1, L)]
    lg = logits[rows].double().cpu().numpy()
    lab = np.zeros(1 + L, np.int64)
    lab[1:] = tokens[r0 + o:r0 + o + L].cpu().numpy()
    # compact layout: prompt of 1 token (row 0 = the last prompt position), then the
    # response; row 1 + j - 1 predicts token 1 + j
    lg_full = np.zeros((1 + L, lg.shape[1]))
    lg_full[0] = lg[0]
    lg_full[1:L] = lg[1:]
    cp = wl.make_pack([1], [[L]])
    seq, _ = orc.seq_logprob(*cp.oracle_args(), lg_full, lab)
    return seq[0, 0]


def _logprob_sample(cfg, stream, n_samples=6):
    pack = wl.config_pack(cfg)
    seed = wl.tensor_seed(cfg.index, 0)
    T = pack.total_tokens
    logits = wl.randn_rows(T, cfg.vocab, seed + stream, torch.bfloat16, DEV, cfg.logit_sigma)
    tokens = wl.randint((T,), cfg.vocab, seed + wl.STREAM_TOKENS, DEV)
    seq, tok = pp.pp_seq_logprob(pack, logits, tokens, want_tok=True)
    torch.cuda.synchronize()
    seq_c = seq.double().cpu().numpy()
    tok_c = tok.double().cpu().numpy()
    rng = np.random.default_rng(cfg.index)
    picks = [(int(b), int(rng.integers(0, int(pack.num_resp[b])))) for b in rng.integers(0, pack.num_rows, n_samples)]
    for b, k in picks:
        want = _compact_response(pack, b, k, logits, tokens)
        assert abs(seq_c[b, k] - want) <= 1e-4 * abs(want), (b, k, seq_c[b, k], want)
    # every response's sum equals the sum of its per-token values (fp64 on host)
    for b in range(pack.num_rows):
        r0 = int(pack.row_start[b])
        for k in range(int(pack.num_resp[b])):
            o, L = int(pack.resp_off[b, k]), int(pack.resp_len[b, k])
            s = tok_c[r0 + o:r0 + o + L].sum()
            assert abs(seq_c[b, k] - s) <= 1e-5 * max(1.0, abs(s))
    return pack, seq


def test_fullsize_rm_k4_logprob_and_bt_loss():
    pack, seq = _logprob_sample(wl.RM_K4, wl.STREAM_LOGITS_POL)
    cfg = wl.RM_K4
    loss, rows, grad = pp.pp_dpo_loss(pack.num_resp.tolist(), seq, None, cfg.beta)
    want, want_rows, want_g = orc.pair_loss(pack.num_resp.tolist(), seq.double().cpu().numpy(), None, cfg.beta)
    assert abs(float(loss) - want) <= 1e-4 * abs(want)
    assert np.allclose(grad.cpu().numpy(), want_g, rtol=1e-4, atol=1e-7)


def test_fullsize_dpo_chain_logprob_and_loss():
    pack, s_pol = _logprob_sample(wl.DPO_CHAIN, wl.STREAM_LOGITS_POL, n_samples=4)
    _, s_ref = _logprob_sample(wl.DPO_CHAIN, wl.STREAM_LOGITS_REF, n_samples=4)
    cfg = wl.DPO_CHAIN
    loss, rows, grad = pp.pp_dpo_loss(pack.num_resp.tolist(), s_pol, s_ref, cfg.beta)
    want, want_rows, want_g = orc.pair_loss(pack.num_resp.tolist(), s_pol.double().cpu().numpy(),
                                            s_ref.double().cpu().numpy(), cfg.beta)
    assert abs(float(loss) - want) <= 1e-4 * abs(want)
    assert np.allclose(rows.cpu().numpy(), want_rows, rtol=1e-4, atol=1e-7)
