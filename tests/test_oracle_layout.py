"""Pins of the oracle's pack layout: mask, segment and position IDs, tile
classes, pair counts and the cost model (Sec. 3.2, Sec. 3.2.1, Table 1)."""
import itertools
import math
import os

import numpy as np
import pytest

from oracle import pp_oracle as orc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_fixture(name):
    rows = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            rows.setdefault(key, []).append(vals)
    return rows


def test_mask_matches_hand_written_example():
    fx = _read_fixture("mask_p3_r2_r2_pad1.txt")
    T = int(fx["T"][0][0])
    P = int(fx["P"][0][0])
    offs = [int(r[0]) for r in fx["resp"]]
    lens = [int(r[1]) for r in fx["resp"]]
    seg = orc.row_segment_ids(T, P, offs, lens)
    pos = orc.row_position_ids(T, P, offs, lens)
    M = orc.row_mask(T, P, offs, lens)
    assert seg.tolist() == [int(x) for x in fx["seg"][0]]
    assert pos.tolist() == [int(x) for x in fx["pos"][0]]
    want = np.array([[int(x) for x in r] for r in fx["mask"]], dtype=bool)
    assert (M == want).all()
    tiles = orc.tile_classes(M, 2, 2)
    want_t = np.array([[int(x) for x in r] for r in fx["tiles22"]], dtype=np.uint8)
    assert (tiles == want_t).all()


def _brute_visible(T, P, offs, lens, i, j):
    """Visibility of key j from query i stated sentence by sentence (Sec. 3.2)."""
    def segment(t):
        if t < P:
            return "prompt"
        for k, (o, L) in enumerate(zip(offs, lens)):
            if o <= t < o + L:
                return k
        return None
    si, sj = segment(i), segment(j)
    if si is None or sj is None:
        return False          # padding sees nothing and is seen by nothing
    if j > i:
        return False          # causal
    if sj == "prompt":
        return True           # every token sees the whole (earlier) prompt
    return si == sj           # a response sees only its own earlier tokens


@pytest.mark.parametrize("P,lens,pad", [(0, [3, 2], 0), (4, [], 2), (5, [0, 3, 1], 1),
                                        (1, [1, 1, 1, 1], 0), (6, [2, 5], 3)])
def test_mask_brute_force(P, lens, pad):
    offs = []
    o = P
    for L in lens:
        offs.append(o)
        o += L
    T = o + pad
    M = orc.row_mask(T, P, offs, lens)
    for i in range(T):
        for j in range(T):
            assert M[i, j] == _brute_visible(T, P, offs, lens, i, j), (i, j)


def test_tile_classes_brute_force():
    rng = np.random.default_rng(5)
    for _ in range(20):
        P = int(rng.integers(0, 9))
        lens = [int(x) for x in rng.integers(0, 7, size=int(rng.integers(0, 4)))]
        offs = []
        o = P
        for L in lens:
            offs.append(o)
            o += L
        T = o + int(rng.integers(0, 3))
        if T == 0:
            continue
        M = orc.row_mask(T, P, offs, lens)
        for bq, bk in [(1, 1), (2, 3), (4, 4), (3, 2)]:
            got = orc.tile_classes(M, bq, bk)
            for a in range(got.shape[0]):
                for b in range(got.shape[1]):
                    cells = [M[i, j] for i in range(a * bq, min(T, a * bq + bq))
                             for j in range(b * bk, min(T, b * bk + bk))]
                    want = 0 if not any(cells) else (2 if all(cells) else 1)
                    assert got[a, b] == want


def test_useful_pairs_closed_form():
    """Visible pairs of a row: P(P+1)/2 + sum_k [L_k P + L_k(L_k+1)/2]."""
    rng = np.random.default_rng(7)
    for _ in range(30):
        B = int(rng.integers(1, 4))
        P = [int(x) for x in rng.integers(0, 40, size=B)]
        L = [[int(x) for x in rng.integers(0, 20, size=int(rng.integers(0, 4)))] for _ in range(B)]
        K = [len(r) for r in L]
        want = sum(p * (p + 1) // 2 + sum(l * p + l * (l + 1) // 2 for l in ls) for p, ls in zip(P, L))
        assert orc.useful_pairs(P, K, L) == want


def test_position_ids_restart_each_response():
    """Each response's position IDs equal the positions it has when laid out
    alone after the prompt (Sec. 3.2)."""
    P, lens = 7, [3, 5, 2]
    offs = [7, 10, 15]
    pos = orc.row_position_ids(17, P, offs, lens)
    for o, L in zip(offs, lens):
        unpacked = list(range(P + L))
        assert pos[:P].tolist() == unpacked[:P]
        assert pos[o:o + L].tolist() == unpacked[P:]


def test_prompt_only_row_is_plain_causal():
    """No responses (or P=0 with one response): the mask is the lower triangle."""
    M = orc.row_mask(6, 6, [], [])
    assert (M == np.tril(np.ones((6, 6), bool))).all()
    M = orc.row_mask(5, 0, [0], [5])
    assert (M == np.tril(np.ones((5, 5), bool))).all()


def test_zero_prompt_is_document_masking():
    """P = 0: K independent causal documents (sequence packing, Sec. 2.2)."""
    lens = [3, 4, 2]
    M = orc.row_mask(9, 0, [0, 3, 7], lens)
    want = np.zeros((9, 9), bool)
    o = 0
    for L in lens:
        want[o:o + L, o:o + L] = np.tril(np.ones((L, L), bool))
        o += L
    assert (M == want).all()


# ---------------------------------------------------------------- cost model


def _table1():
    out = {}
    for k, v in _read_fixture("table1_lengths.txt").items():
        out[k] = [float(x) for x in v[0]]
    return out


def test_table1_datasets_satisfy_eq1():
    """The paper reports that Eq. (1) holds on its three K=2 datasets (Sec. 5.1),
    so their packed/unpacked cost ratio is below 1."""
    for name, (lin, lmax, lmin) in _table1().items():
        assert orc.packing_is_cheaper(lin, [lmin, lmax]), name
        assert orc.cost_ratio(lin, [lmin, lmax]) < 1.0, name
        # the RLAIF-V case, with its long image prefix, is the most favourable
    r = {n: orc.cost_ratio(a, [c, b]) for n, (a, b, c) in _table1().items()}
    assert min(r, key=r.get) == "rlaif_v"


def test_cost_ratio_below_one_iff_eq1():
    rng = np.random.default_rng(3)
    for _ in range(2000):
        K = int(rng.integers(2, 6))
        lin = float(rng.uniform(0, 1000))
        l = [float(x) for x in rng.uniform(1, 1000, size=K)]
        r = orc.cost_ratio(lin, l)
        if abs(r - 1.0) < 1e-9:
            continue
        assert (r < 1.0) == orc.packing_is_cheaper(lin, l)


def test_memory_ratio_at_most_one():
    """With linear-memory attention the ratio is <= 1, and < 1 once the prompt is
    non-empty or the responses differ in length (Sec. 3.2.1)."""
    rng = np.random.default_rng(4)
    for _ in range(2000):
        K = int(rng.integers(2, 6))
        lin = float(rng.uniform(0, 500))
        l = [float(x) for x in rng.uniform(1, 500, size=K)]
        m = orc.memory_ratio(lin, l)
        assert m <= 1.0 + 1e-12
        if lin > 1e-6 or max(l) - min(l) > 1e-6:
            assert m < 1.0
    assert orc.memory_ratio(0.0, [10.0, 10.0]) == pytest.approx(1.0)


def test_long_responses_make_packing_costlier():
    """Limitations: responses much longer than the prompt raise the cost."""
    assert orc.cost_ratio(10.0, [2000.0, 2000.0]) > 1.0
    assert not orc.packing_is_cheaper(10.0, [2000.0, 2000.0])
    # equal-length responses with an empty prompt: (K l)^2 / (K l^2) = K
    assert orc.cost_ratio(0.0, [50.0] * 3) == pytest.approx(3.0)


def test_logprob_rows_needed_brute_force():
    rng = np.random.default_rng(9)
    for _ in range(30):
        B = int(rng.integers(1, 4))
        P = [int(x) for x in rng.integers(1, 10, size=B)]
        L = [[int(x) for x in rng.integers(0, 6, size=int(rng.integers(0, 4)))] for _ in range(B)]
        K = [len(r) for r in L]
        want = 0
        for p, ls in zip(P, L):
            rows = set()
            o = p
            for l in ls:
                for j in range(l):
                    rows.add(p - 1 if j == 0 else o + j - 1)
                o += l
            want += len(rows)
        assert orc.logprob_rows_needed(P, K, L) == want
