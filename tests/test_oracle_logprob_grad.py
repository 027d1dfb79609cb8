"""Pins of the oracle's log-prob backward (reading R16) against facts that do
not come from the oracle's own formula: central finite differences of the
(separately pinned) forward, the softmax simplex, the sharing of the last prompt
row by every response (Sec. 3.2), and the rows that predict nothing."""
import numpy as np

from oracle import pp_oracle as orc
from paper_2602_24082_amd import workload as wl


def _case(seed, prompt_lens, resp_lens, V, pad=None):
    pack = wl.make_pack(prompt_lens, resp_lens, pad=pad)
    rng = np.random.default_rng(seed)
    T = pack.total_tokens
    logits = rng.normal(0.0, 1.5, size=(T, V))
    tokens = rng.integers(0, V, size=T)
    dseq = rng.normal(size=(pack.num_rows, pack.max_resp))
    return pack, logits, tokens, dseq


def test_finite_differences_of_the_forward():
    pack, logits, tokens, dseq = _case(1, [3, 1], [[2, 3], [1, 0, 2]], V=5, pad=[1, 2])
    args = pack.oracle_args()
    grad = orc.seq_logprob_grad(*args, logits, tokens, dseq)

    def f(x):
        seq, _ = orc.seq_logprob(*args, x, tokens)
        return float((dseq * seq).sum())

    h = 1e-6
    fd = np.zeros_like(logits)
    for idx in np.ndindex(*logits.shape):
        xp = logits.copy()
        xm = logits.copy()
        xp[idx] += h
        xm[idx] -= h
        fd[idx] = (f(xp) - f(xm)) / (2 * h)
    assert np.abs(grad - fd).max() < 1e-8


def test_rows_sum_to_zero_and_unused_rows_are_zero():
    pack, logits, tokens, dseq = _case(2, [5, 4, 2], [[3, 1], [2], [4, 2, 1]], V=11, pad=[0, 3, 1])
    args = pack.oracle_args()
    grad = orc.seq_logprob_grad(*args, logits, tokens, dseq)
    # gradient rows are (sums of) onehot - softmax: each sums to zero
    assert np.abs(grad.sum(axis=1)).max() < 1e-12
    used = set()
    for b in range(pack.num_rows):
        r0, P = int(pack.row_start[b]), int(pack.prompt_len[b])
        for k in range(int(pack.num_resp[b])):
            o, L = int(pack.resp_off[b, k]), int(pack.resp_len[b, k])
            if L > 0:
                used.add(r0 + P - 1)
            used.update(r0 + o + j - 1 for j in range(1, L))
    unused = [r for r in range(pack.total_tokens) if r not in used]
    assert unused and np.all(grad[unused] == 0.0)


def test_last_prompt_row_gathers_every_response():
    P, lens, V = 4, [2, 3, 1], 6
    pack, logits, tokens, dseq = _case(3, [P], [lens], V=V)
    grad = orc.seq_logprob_grad(*pack.oracle_args(), logits, tokens, dseq)
    row = logits[P - 1]
    p = np.exp(row - row.max())
    p /= p.sum()
    want = np.zeros(V)
    for k, o in enumerate(pack.resp_off[0, :3]):
        want += dseq[0, k] * (np.eye(V)[tokens[o]] - p)
    assert np.abs(grad[P - 1] - want).max() < 1e-12


def test_single_token_response_closed_form():
    # one response of one token: d/dx [x_y - logsumexp(x)] = e_y - softmax(x)
    V = 9
    pack, logits, tokens, dseq = _case(4, [2], [[1]], V=V)
    grad = orc.seq_logprob_grad(*pack.oracle_args(), logits, tokens, dseq)
    x = logits[1]
    sm = np.exp(x) / np.exp(x).sum()
    assert np.abs(grad[1] - dseq[0, 0] * (np.eye(V)[tokens[2]] - sm)).max() < 1e-12
    assert np.all(grad[[0, 2]] == 0.0)


def test_out_of_range_label_poisons_only_its_row():
    pack, logits, tokens, dseq = _case(5, [3], [[3, 2]], V=7)
    t_bad = int(pack.resp_off[0, 0]) + 2  # third token of response 0, predicted by row t_bad - 1
    tokens = tokens.copy()
    tokens[t_bad] = 7
    grad = orc.seq_logprob_grad(*pack.oracle_args(), logits, tokens, dseq)
    assert np.all(np.isnan(grad[t_bad - 1]))
    others = [r for r in range(pack.total_tokens) if r != t_bad - 1]
    assert np.all(np.isfinite(grad[others]))


def test_predicting_rows_by_hand_and_by_the_gradient():
    """The rows the gathered backward writes: a row written out by hand, the
    pinned row count, and -- for random logits and nonzero dseq -- exactly the
    rows where the (finite-difference pinned) gradient is not zero."""
    # P = 3, responses of 2 and 2 tokens at 3..4 and 5..6, one padding token:
    # row 2 predicts tokens 3 and 5, row 3 predicts 4, row 5 predicts 6
    pack = wl.make_pack([3], [[2, 2]], pad=[1])
    assert orc.logprob_predicting_rows(*pack.oracle_args()) == [2, 3, 5]
    for seed, P, L, pad in ((3, [4, 1, 6], [[2, 0, 3], [1, 1], [5]], [0, 2, 1]),
                            (4, [2, 9], [[1], [4, 4, 1, 2]], [3, 0])):
        pack, logits, tokens, dseq = _case(seed, P, L, V=6, pad=pad)
        args = pack.oracle_args()
        rows = orc.logprob_predicting_rows(*args)
        assert len(rows) == orc.logprob_rows_needed(pack.prompt_len, pack.num_resp, pack.resp_len.tolist())
        grad = orc.seq_logprob_grad(*args, logits, tokens, np.where(dseq == 0, 1.0, dseq))
        assert rows == sorted(np.flatnonzero(np.abs(grad).sum(axis=1) > 0).tolist())
