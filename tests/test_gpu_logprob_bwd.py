"""GPU parity of the log-prob backward (pp_seq_logprob_bwd, and
pp_seq_logprob_bwd_rows, which writes only the rows that predict a response
token) against the fp64 oracle's seq_logprob_grad, element by element.  The
gathered rows must come back in the order of the oracle's
logprob_predicting_rows, with those row indices (bit-exact), and equal the
dense output's rows bit for bit.

Tolerances, derived from the arithmetic: the kernel forms softmax in fp32 from
a logsumexp accumulated in fp32 (relative error a few 1e-6 for vocabularies up
to ~1e5), so fp32 outputs are held to rtol 2e-5; bf16 outputs add the final
rounding to bf16 (relative 2^-9), held to rtol 5e-3.  Both get an absolute
floor of 1e-6 times the largest |dseq| for entries that are tiny multiples of
it.  Rows that predict no response token must be exactly 0.
"""

import numpy as np
import pytest
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import binding as pp
from paper_2602_24082_amd import workload as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
RTOL = {torch.float32: 2e-5, torch.bfloat16: 5e-3}


def _needed_rows(pack):
    rows = set()
    for b in range(pack.num_rows):
        r0, P = int(pack.row_start[b]), int(pack.prompt_len[b])
        for k in range(int(pack.num_resp[b])):
            o, L = int(pack.resp_off[b, k]), int(pack.resp_len[b, k])
            if L > 0:
                rows.add(r0 + P - 1)
            rows.update(r0 + o + j - 1 for j in range(1, L))
    return sorted(rows)


def _check_bwd(pack, V, dtype, sigma, seed, dseq=None):
    print(f"logprob_bwd rows={pack.num_rows} T={pack.total_tokens} V={V} {dtype}", flush=True)
    T = pack.total_tokens
    logits = wl.randn((T, V), seed, dtype, "cpu", sigma=sigma)
    tokens = wl.randint((T,), V, seed + 1, "cpu")
    if dseq is None:
        dseq = wl.randn((pack.num_rows, pack.max_resp), seed + 2, torch.float32, "cpu")
    dl = torch.full((T, V), float("nan"), dtype=dtype, device=DEV)
    pp.pp_seq_logprob_bwd(pack, logits.to(DEV), tokens.to(DEV), dseq.to(DEV), dlogits=dl)
    ref = orc.seq_logprob_grad(*pack.oracle_args(), logits.double().numpy(), tokens.numpy(),
                               dseq.double().numpy())
    got = dl.double().cpu().numpy()
    need = _needed_rows(pack)
    unused = np.ones(T, bool)
    unused[need] = False
    assert (got[unused] == 0).all()
    gmax = float(np.abs(dseq.numpy()).max())
    assert np.isfinite(got).all()
    err = np.abs(got - ref) - RTOL[dtype] * np.abs(ref)
    assert err.max() <= 1e-6 * gmax, err.max()
    # the gathered form: the same rows, compact, with their indices
    rows_want = orc.logprob_predicting_rows(*pack.oracle_args())
    assert pp.pp_logprob_row_count(pack) == len(rows_want)
    if rows_want:
        dr = torch.full((len(rows_want), V), float("nan"), dtype=dtype, device=DEV)
        ri = torch.full((len(rows_want),), -7, dtype=torch.int32, device=DEV)
        pp.pp_seq_logprob_bwd_rows(pack, logits.to(DEV), tokens.to(DEV), dseq.to(DEV), dlogits_rows=dr,
                                   row_index=ri)
        assert ri.cpu().tolist() == rows_want
        assert torch.equal(dr, dl[torch.tensor(rows_want, device=DEV).long()])
        g_rows = dr.double().cpu().numpy()
        err = np.abs(g_rows - ref[rows_want]) - RTOL[dtype] * np.abs(ref[rows_want])
        assert err.max() <= 1e-6 * gmax, err.max()
    return got


def test_logprob_bwd_tiny_fp32():
    _check_bwd(wl.config_pack(wl.TINY_FP32), 1000, torch.float32, 2.0, 171)


def test_logprob_bwd_bf16_odd_vocab_and_edges():
    # vocab 4099: rows are not 16-byte aligned -> element path; empty and one-token
    # responses, a one-token prompt, padding rows
    pack = wl.make_pack([5, 1, 9], [[3, 0, 7], [1], [12, 40]], pad=[2, 0, 1])
    _check_bwd(pack, 4099, torch.bfloat16, 3.0, 172)
    _check_bwd(pack, 4096, torch.bfloat16, 3.0, 173)
    _check_bwd(pack, 4096, torch.float32, 3.0, 174)


def test_logprob_bwd_llama_vocab_k4():
    pack = wl.make_pack([40, 17], [[9, 30, 2, 11], [25, 1, 0, 8]])
    _check_bwd(pack, 128256, torch.bfloat16, 3.0, 175)


def test_logprob_bwd_register_row_limit():
    # fp32 rows of exactly 1024 threads x 19 vectors x 4 values (held in
    # registers, read once) and one 16-byte vector longer (the two-read kernel)
    pack = wl.make_pack([6, 3], [[5, 2], [4, 1, 3]], pad=[1, 0])
    _check_bwd(pack, 77824, torch.float32, 3.0, 185)
    _check_bwd(pack, 77828, torch.float32, 3.0, 186)


def test_logprob_bwd_qwen_vocab():
    # a 152064-entry bf16 vocabulary (the 72B-shaped workloads): register rows
    pack = wl.make_pack([33, 8], [[12, 1], [20, 5, 3]], pad=[0, 2])
    _check_bwd(pack, 152064, torch.bfloat16, 3.0, 187)


def _random_logprob_pack(rng):
    B = int(rng.integers(1, 5))
    P, L, pad = [], [], []
    for _ in range(B):
        P.append(int(rng.integers(1, 200)))
        L.append([int(x) for x in rng.integers(0, 120, size=int(rng.integers(0, 5)))])
        pad.append(int(rng.integers(0, 9)))
    return wl.make_pack(P, L, pad=pad)


@pytest.mark.parametrize("seed", range(4))
def test_logprob_bwd_random_sweep(seed):
    """Seeded random packs and vocabularies (the register-row and the two-read
    kernel, aligned and unaligned rows), bf16 and fp32."""
    rng = np.random.default_rng(4000 + seed)
    pack = _random_logprob_pack(rng)
    V = int(rng.choice([1000, 4099, 32000, 50257, 70000]))
    dtype = torch.bfloat16 if seed % 2 == 0 else torch.float32
    _check_bwd(pack, V, dtype, 3.0, 4100 + seed)


def test_logprob_bwd_takes_the_loss_gradient():
    # the DPO chain: forward scores, loss gradient, then logits gradient
    pack = wl.make_pack([30, 12, 20], [[10, 14], [7, 9], [5, 6]])
    V, T = 2048, pack.total_tokens
    lp = wl.randn((T, V), 176, torch.float32, DEV, sigma=2.0)
    lr = wl.randn((T, V), 177, torch.float32, DEV, sigma=2.0)
    tokens = wl.randint((T,), V, 178, DEV)
    s_pol = pp.pp_seq_logprob(pack, lp, tokens)
    s_ref = pp.pp_seq_logprob(pack, lr, tokens)
    _, _, g = pp.pp_dpo_loss(pack.num_resp.tolist(), s_pol, s_ref, 0.1)
    dl = pp.pp_seq_logprob_bwd(pack, lp, tokens, g)
    ref = orc.seq_logprob_grad(*pack.oracle_args(), lp.double().cpu().numpy(), tokens.cpu().numpy(),
                               g.double().cpu().numpy())
    got = dl.double().cpu().numpy()
    gmax = float(g.abs().max())
    assert (np.abs(got - ref) - RTOL[torch.float32] * np.abs(ref)).max() <= 1e-6 * gmax


def test_logprob_bwd_out_of_range_label_poisons_its_row():
    pack = wl.make_pack([4], [[3, 3]])
    V = 64
    logits = wl.randn((10, V), 180, torch.float32, DEV)
    tokens = wl.randint((10,), V, 181, "cpu")
    tokens[5] = V + 3  # second token of response 0 (positions 4..6), predicted by row 4
    dseq = torch.ones(1, 2, device=DEV)
    dl = pp.pp_seq_logprob_bwd(pack, logits, tokens.to(DEV), dseq).cpu()
    assert torch.isnan(dl[4]).all()
    assert torch.isfinite(dl[torch.arange(10) != 4]).all()
    # gathered: rows 3 (first tokens), 4, 5, 7, 8 -- only row 4's copy is NaN
    dr, ri = pp.pp_seq_logprob_bwd_rows(pack, logits, tokens.to(DEV), dseq)
    assert ri.cpu().tolist() == [3, 4, 5, 7, 8]
    dr = dr.cpu()
    assert torch.isnan(dr[1]).all() and torch.isfinite(dr[[0, 2, 3, 4]]).all()


def test_logprob_bwd_fullsize_rm_k4_sampled():
    # the reward-model batch at full size (17.7k rows x 128256, bf16); the oracle
    # recomputes sampled rows from compact packs: single-label rows of sampled
    # responses, and every row's last prompt position (all K first tokens)
    cfg = wl.RM_K4
    pack = wl.config_pack(cfg)
    T, V = pack.total_tokens, cfg.vocab
    seed = wl.tensor_seed(cfg.index, 0)
    logits = wl.randn_rows(T, V, seed + wl.STREAM_LOGITS_POL, torch.bfloat16, DEV, cfg.logit_sigma)
    tokens = wl.randint((T,), V, seed + wl.STREAM_TOKENS, DEV)
    dseq = wl.randn((pack.num_rows, pack.max_resp), seed + 5, torch.float32, DEV)
    dl = pp.pp_seq_logprob_bwd(pack, logits, tokens, dseq)
    # the gathered form at full size: the oracle's rows, each equal to the dense row
    dr, ri = pp.pp_seq_logprob_bwd_rows(pack, logits, tokens, dseq)
    rows_want = orc.logprob_predicting_rows(*pack.oracle_args())
    assert ri.cpu().tolist() == rows_want
    assert torch.equal(dr, dl[ri.long()])
    del dr
    torch.cuda.synchronize()
    tok = tokens.cpu().numpy()
    g = dseq.double().cpu().numpy()
    gmax = float(np.abs(g).max())
    rng = np.random.default_rng(2)
    checked = 0
    for b in rng.choice(pack.num_rows, 3, replace=False):
        b = int(b)
        r0, P, K = int(pack.row_start[b]), int(pack.prompt_len[b]), int(pack.num_resp[b])
        lens = [int(x) for x in pack.resp_len[b, :K]]
        # last prompt row: a compact pack of 1 prompt token and the K first tokens
        cp = wl.make_pack([1], [[1 if L > 0 else 0 for L in lens]])
        labels = np.zeros(cp.total_tokens, np.int64)
        pos = 1
        for k, L in enumerate(lens):
            if L > 0:
                labels[pos] = tok[r0 + int(pack.resp_off[b, k])]
                pos += 1
        x = np.zeros((cp.total_tokens, V))
        x[0] = logits[r0 + P - 1].double().cpu().numpy()
        gg = np.zeros((1, cp.max_resp))
        gg[0, :K] = g[b, :K]
        want = orc.seq_logprob_grad(*cp.oracle_args(), x, labels, gg)[0]
        got = dl[r0 + P - 1].double().cpu().numpy()
        assert (np.abs(got - want) - RTOL[torch.bfloat16] * np.abs(want)).max() <= 1e-6 * gmax
        checked += 1
        # a few single-label rows of one response
        k = int(np.argmax(lens))
        o = int(pack.resp_off[b, k])
        for j in rng.choice(np.arange(1, lens[k]), 3, replace=False):
            r = r0 + o + int(j) - 1
            cp1 = wl.make_pack([1], [[1]])
            x1 = np.zeros((2, V))
            x1[0] = logits[r].double().cpu().numpy()
            want = orc.seq_logprob_grad(*cp1.oracle_args(), x1, np.array([0, tok[r + 1]]),
                                        np.array([[g[b, k]]]))[0]
            got = dl[r].double().cpu().numpy()
            assert (np.abs(got - want) - RTOL[torch.bfloat16] * np.abs(want)).max() <= 1e-6 * gmax
            checked += 1
        # prompt rows before P-1 predict nothing
        if P >= 2:
            assert (dl[r0:r0 + P - 1] == 0).all()
    assert checked >= 6
    assert torch.isfinite(dl).all()
