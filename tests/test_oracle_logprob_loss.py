"""Pins of the oracle's per-response log-probabilities and the ranked-pair
DPO / Bradley-Terry loss (Sec. 2.1, Sec. 3.1, Sec. 3.2)."""
import itertools
import math

import numpy as np
import pytest
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import workload as wl


def _unpacked_logprob(P, resp_tokens, prompt_tokens, prompt_logits, resp_logits):
    """Textbook causal-LM score of one unpacked (prompt, response) sequence:
    sum over response tokens of log_softmax(logits[t-1])[token t]."""
    toks = torch.tensor(list(prompt_tokens) + list(resp_tokens))
    logits = torch.cat([prompt_logits, resp_logits], dim=0)
    lsm = torch.log_softmax(logits, dim=-1)
    s = 0.0
    for t in range(P, P + len(resp_tokens)):
        s += float(lsm[t - 1, toks[t]])
    return s


def test_packed_logprob_equals_unpacked():
    """Each response's packed score equals the unpacked sequence's score when
    the logits at the packed positions are those the unpacked sequence would
    produce (the equivalence of Sec. 3.2)."""
    pack = wl.make_pack([5, 3, 1], [[2, 4], [1, 1, 3], [6]], pad=[2, 0, 1])
    T = pack.total_tokens
    V = 11
    g = torch.Generator().manual_seed(3)
    logits = torch.randn(T, V, generator=g, dtype=torch.float64) * 2
    tokens = torch.randint(0, V, (T,), generator=g)
    seq, tok = orc.seq_logprob(*pack.oracle_args(), logits.numpy(), tokens.numpy())
    for b in range(pack.num_rows):
        r0 = int(pack.row_start[b])
        P = int(pack.prompt_len[b])
        for k in range(int(pack.num_resp[b])):
            o, L = int(pack.resp_off[b, k]), int(pack.resp_len[b, k])
            want = _unpacked_logprob(P, tokens[r0 + o:r0 + o + L].tolist(),
                                     tokens[r0:r0 + P].tolist(), logits[r0:r0 + P],
                                     logits[r0 + o:r0 + o + L])
            assert abs(seq[b, k] - want) < 1e-12
            assert abs(tok[r0 + o:r0 + o + L].sum() - want) < 1e-12
    # empty slots and non-response positions are 0
    assert seq[0, 2] == 0.0 and seq[2, 1] == 0.0
    assert (tok[:5] == 0).all()


def test_zero_logits_give_minus_L_log_V():
    pack = wl.make_pack([4, 2], [[3, 0, 5], [7]])
    V = 37
    T = pack.total_tokens
    logits = np.zeros((T, V))
    tokens = np.arange(T) % V
    seq, _ = orc.seq_logprob(*pack.oracle_args(), logits, tokens)
    assert seq[0].tolist() == pytest.approx([-3 * math.log(V), 0.0, -5 * math.log(V)], abs=1e-12)
    assert seq[1, 0] == pytest.approx(-7 * math.log(V), abs=1e-12)


def test_confident_logits_give_zero_score():
    """A logit row with +60 at its label scores ~0 (log-prob of ~1)."""
    pack = wl.make_pack([3], [[4]])
    V = 9
    T = pack.total_tokens
    tokens = np.array([1, 2, 3, 4, 5, 6, 7])
    logits = np.zeros((T, V))
    for t in range(3, 7):
        src = 2 if t == 3 else t - 1
        logits[src, tokens[t]] = 60.0
    seq, _ = orc.seq_logprob(*pack.oracle_args(), logits, tokens)
    # each token: 60 - ln(e^60 + 8) = -ln(1 + 8 e^-60) ~ -8 e^-60
    assert seq[0, 0] == pytest.approx(-4 * 8 * math.exp(-60), rel=1e-9)


def test_out_of_range_label_poisons_only_its_response():
    pack = wl.make_pack([3], [[2, 2]])
    V = 5
    tokens = np.array([0, 1, 2, 3, 9, 1, 2])
    logits = np.random.default_rng(1).standard_normal((7, V))
    seq, _ = orc.seq_logprob(*pack.oracle_args(), logits, tokens)
    assert math.isnan(seq[0, 0]) and not math.isnan(seq[0, 1])


def test_logsumexp_against_library():
    x = np.random.default_rng(2).standard_normal(1000) * 30
    assert abs(orc.logsumexp_row(x) - float(torch.logsumexp(torch.tensor(x), 0))) < 1e-12


# ------------------------------------------------------------------------ loss


def test_policy_equal_reference_gives_log2():
    rng = np.random.default_rng(0)
    for K in (2, 3, 4, 6):
        s = rng.standard_normal((3, K)) * 10
        loss, rows, _ = orc.pair_loss([K, K, K], s, s.copy(), 0.1)
        assert loss == pytest.approx(math.log(2), abs=1e-14)
        assert rows == pytest.approx([math.log(2)] * 3, abs=1e-14)


def test_two_responses_is_single_pair_dpo():
    """K = 2: -log sigmoid(beta*((pol_w - ref_w) - (pol_l - ref_l))), with the
    second response the preferred one (Sec. 2.1, Sec. 3.1)."""
    rng = np.random.default_rng(1)
    pol = rng.standard_normal((5, 2)) * 20
    ref = rng.standard_normal((5, 2)) * 20
    beta = 0.1
    loss, rows, _ = orc.pair_loss([2] * 5, pol, ref, beta)
    want = -torch.nn.functional.logsigmoid(
        beta * torch.tensor((pol[:, 1] - ref[:, 1]) - (pol[:, 0] - ref[:, 0])))
    assert rows == pytest.approx(want.numpy(), rel=1e-13)
    assert loss == pytest.approx(float(want.mean()), rel=1e-13)


def test_reward_model_without_reference():
    """No reference: rewards are beta * score (the reward-model BT loss)."""
    s = np.array([[1.0, 3.0, 2.0]])
    loss, _, _ = orc.pair_loss([3], s, None, 1.0)
    pairs = [(1, 0), (2, 0), (2, 1)]  # (preferred, other)
    want = np.mean([-float(torch.nn.functional.logsigmoid(torch.tensor(s[0, a] - s[0, c])))
                    for a, c in pairs])
    assert loss == pytest.approx(want, rel=1e-14)


def test_all_pairs_mean_by_enumeration():
    rng = np.random.default_rng(5)
    num = [4, 2, 1, 3, 0]
    pol = rng.standard_normal((5, 4)) * 5
    ref = rng.standard_normal((5, 4)) * 5
    loss, rows, _ = orc.pair_loss(num, pol, ref, 0.5)
    per_row = []
    for b, K in enumerate(num):
        if K < 2:
            assert rows[b] == 0.0
            continue
        z = 0.5 * (pol[b, :K] - ref[b, :K])
        terms = [math.log1p(math.exp(-(z[a] - z[c]))) for c, a in itertools.combinations(range(K), 2)]
        assert rows[b] == pytest.approx(np.mean(terms), rel=1e-13)
        per_row.append(np.mean(terms))
    assert loss == pytest.approx(np.mean(per_row), rel=1e-13)


def test_swapping_order_flips_the_margin():
    """softplus(-x) - softplus(x) = -x: swapping the two responses of a K = 2 row
    changes its loss by exactly the reward margin."""
    pol = np.array([[-3.0, 5.0]])
    ref = np.array([[1.0, 0.5]])
    beta = 0.3
    a, _, _ = orc.pair_loss([2], pol, ref, beta)
    b, _, _ = orc.pair_loss([2], pol[:, ::-1].copy(), ref[:, ::-1].copy(), beta)
    margin = beta * ((5.0 - 0.5) - (-3.0 - 1.0))
    assert a - b == pytest.approx(-margin, rel=1e-13)


def test_loss_gradient_finite_differences():
    rng = np.random.default_rng(6)
    num = [3, 2, 1, 4]
    pol = rng.standard_normal((4, 4)) * 3
    ref = rng.standard_normal((4, 4)) * 3
    beta = 0.7
    _, _, g = orc.pair_loss(num, pol, ref, beta)
    eps = 1e-6
    for b in range(4):
        for k in range(4):
            p1 = pol.copy(); p1[b, k] += eps
            p2 = pol.copy(); p2[b, k] -= eps
            num_g = (orc.pair_loss(num, p1, ref, beta)[0] - orc.pair_loss(num, p2, ref, beta)[0]) / (2 * eps)
            assert g[b, k] == pytest.approx(num_g, abs=1e-8)


def test_loss_needs_a_pair():
    with pytest.raises(ValueError):
        orc.pair_loss([1, 0], np.zeros((2, 1)), None, 0.1)
