"""Pins of the oracle's reward-model head (reading R17): packing gives the score
of each unpacked (prompt, response) sequence (Sec. 3.2), the head is linear
(closed forms), its gradients match central finite differences, and the scores
feed the Bradley-Terry loss of Sec. 2.1 unchanged."""
import math

import numpy as np

from oracle import pp_oracle as orc
from paper_2602_24082_amd import workload as wl


def _case(seed, prompts, resps, H, pad=None):
    pack = wl.make_pack(prompts, resps, pad=pad)
    rng = np.random.default_rng(seed)
    hidden = rng.normal(size=(pack.total_tokens, H))
    w = rng.normal(size=H)
    return pack, hidden, w, rng


def test_packed_scores_equal_unpacked_last_token():
    pack, hidden, w, _ = _case(1, [4, 1, 3], [[2, 0, 3], [1], [0, 5]], 6, pad=[1, 0, 2])
    bias = 0.25
    got = orc.rm_scores(*pack.oracle_args(), hidden, w, bias)
    for b in range(pack.num_rows):
        r0, P = int(pack.row_start[b]), int(pack.prompt_len[b])
        for k in range(int(pack.num_resp[b])):
            o, L = int(pack.resp_off[b, k]), int(pack.resp_len[b, k])
            # the unpacked sequence (prompt, response k), hidden states copied out
            seq = np.concatenate([hidden[r0:r0 + P], hidden[r0 + o:r0 + o + L]])
            want = float(seq[-1] @ w) + bias
            assert abs(got[b, k] - want) < 1e-12


def test_linear_head_closed_forms():
    pack, hidden, w, _ = _case(2, [3], [[2, 4]], 5)
    e2 = np.eye(5)[2]
    s = orc.rm_scores(*pack.oracle_args(), hidden, e2, -1.0)
    assert s[0, 0] == hidden[3 + 2 - 1, 2] - 1.0 and s[0, 1] == hidden[5 + 4 - 1, 2] - 1.0
    # doubling w doubles the bias-free score
    s1 = orc.rm_scores(*pack.oracle_args(), hidden, w)
    s2 = orc.rm_scores(*pack.oracle_args(), hidden, 2 * w)
    assert np.allclose(s2, 2 * s1, rtol=0, atol=1e-12)


def test_empty_sequence_scores_zero_and_has_no_gradient():
    pack, hidden, w, _ = _case(3, [0, 2], [[0, 3], [0]], 4)
    s = orc.rm_scores(*pack.oracle_args(), hidden, w, 5.0)
    assert s[0, 0] == 0.0  # no prompt, empty response: no token at all
    assert s[1, 0] == float(hidden[int(pack.row_start[1]) + 1] @ w) + 5.0  # empty response -> P-1
    dh, dw, db = orc.rm_scores_grad(*pack.oracle_args(), hidden, w, np.array([[7.0, 0.0], [0.0, 0.0]]))
    assert not dh.any() and not dw.any() and db == 0.0


def test_gradients_finite_differences():
    pack, hidden, w, rng = _case(4, [3, 2], [[2, 0], [1, 3]], 4, pad=[1, 0])
    dsc = rng.normal(size=(pack.num_rows, pack.max_resp))
    args = pack.oracle_args()
    dh, dw, db = orc.rm_scores_grad(*args, hidden, w, dsc)
    f = lambda hh, ww, bb: float((dsc * orc.rm_scores(*args, hh, ww, bb)).sum())
    h = 1e-6
    for idx in np.ndindex(*hidden.shape):
        hp, hm = hidden.copy(), hidden.copy()
        hp[idx] += h
        hm[idx] -= h
        assert abs((f(hp, w, 0.0) - f(hm, w, 0.0)) / (2 * h) - dh[idx]) < 1e-8
    for i in range(w.size):
        wp, wm = w.copy(), w.copy()
        wp[i] += h
        wm[i] -= h
        assert abs((f(hidden, wp, 0.0) - f(hidden, wm, 0.0)) / (2 * h) - dw[i]) < 1e-8
    assert abs((f(hidden, w, h) - f(hidden, w, -h)) / (2 * h) - db) < 1e-8


def test_scores_feed_bradley_terry():
    # K = 2: -log sigmoid(r_w - r_l) with the larger index preferred (Sec. 2.1, Sec. 3.1)
    pack, hidden, w, _ = _case(5, [4], [[3, 2]], 8)
    s = orc.rm_scores(*pack.oracle_args(), hidden, w)
    loss, _, _ = orc.pair_loss([2], s, None, 1.0)
    assert abs(loss - (-math.log(1.0 / (1.0 + math.exp(-(s[0, 1] - s[0, 0])))))) < 1e-12
