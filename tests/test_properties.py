"""Property-based tests (hypothesis) of the host planner, the descriptor checks
and the oracle, over random packed layouts: rows of a prompt of 0-70 tokens,
0-4 responses of 0-50 tokens and 0-9 padding tokens, 1-4 rows.  Examples are
derived from a fixed seed (derandomize) so a run is reproducible; each property
sees 40-60 layouts.  CPU only."""
import math

import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, assume, given, settings
from hypothesis import strategies as st

from oracle import pp_oracle as orc
from paper_2602_24082_amd import binding
from paper_2602_24082_amd import workload as wl

SETTINGS = settings(max_examples=60, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])

row_st = st.tuples(st.integers(0, 70), st.lists(st.integers(0, 50), max_size=4), st.integers(0, 9))


def _pack(rows):
    return wl.make_pack([r[0] for r in rows], [r[1] for r in rows], pad=[r[2] for r in rows])


pack_st = st.lists(row_st, min_size=1, max_size=4).map(_pack)


@SETTINGS
@given(pack_st, st.sampled_from([(1, 1), (16, 16), (32, 32), (32, 64), (128, 64), (7, 5)]))
def test_export_equals_oracle(pack, blocks):
    """Position IDs, segment IDs and tile classes bit for bit (Sec. 3.2)."""
    bq, bk = blocks
    pos, seg, tiles = binding.pp_pack_export(pack, bq, bk)
    args = pack.oracle_args()
    assert (pos == orc.pack_position_ids(*args)).all()
    assert (seg == orc.pack_segment_ids(*args)).all()
    assert (tiles == orc.pack_tile_classes(*args, bq, bk)).all()


@SETTINGS
@given(pack_st, st.sampled_from([(4, 2), (8, 8), (6, 3)]))
def test_stored_ds_region_counts_visible_blocks(pack, heads):
    """The backward's stored-dS region is one 2 KB tile per head for every 32 x 32
    block of the oracle's mask with a visible pair, for the self-contained calls
    and for plans alike."""
    hq, hkv = heads
    n_blocks = int((orc.pack_tile_classes(*pack.oracle_args(), 32, 32) > 0).sum())
    lean = binding.pp_workspace_size(pack, hq, hkv, 128, fwd=False, bwd=True, loss=False)[1]
    full, plan_full = binding.pp_bwd_stored_ds_workspace_size(pack, hq, hkv, 128)
    assert full - lean == hq * n_blocks * 2048
    assert plan_full - binding.pp_plan_workspace_size(pack, hq, hkv, 128) == hq * n_blocks * 2048


@SETTINGS
@given(pack_st)
def test_pack_stats_tokens_and_pairs(pack):
    """Token and visible-pair counts of pp_pack_stats from their definitions."""
    stt = binding.pp_pack_stats(pack)
    P, K, L = pack.prompt_len, pack.num_resp, pack.resp_len
    packed = sum(int(P[b]) + int(L[b, :K[b]].sum()) for b in range(pack.num_rows))
    unpacked = sum(sum(int(P[b]) + int(x) for x in L[b, :K[b]]) if K[b] else int(P[b])
                   for b in range(pack.num_rows))
    assert stt["tokens_packed"] == packed
    assert stt["tokens_unpacked"] == unpacked
    masks = [orc.row_mask(T, p, o, ln) for _, T, p, o, ln in
             (orc._row_fields(*pack.oracle_args(), b) for b in range(pack.num_rows))]
    assert stt["pairs_packed"] == sum(int(m.sum()) for m in masks)
    assert stt["pairs_packed"] <= stt["pairs_dense_packed"]


def _corrupt(pack, kind, b):
    rs, P, K = pack.row_start.copy(), pack.prompt_len.copy(), pack.num_resp.copy()
    off, ln = pack.resp_off.copy(), pack.resp_len.copy()
    T = np.diff(rs)
    if kind == 0:
        rs[0] = 1
    elif kind == 1:
        rs[b + 1] = rs[b] - 1
    elif kind == 2:
        P[b] = -1
    elif kind == 3:
        K[b] = pack.max_resp + 1
    elif kind == 4:
        off[b, 0] += 1
    elif kind == 5:
        P[b] = T[b] + 1
    elif kind == 6:
        ln[b, 0] = -1
    return wl.Pack(rs, P, K, off, ln)


@SETTINGS
@given(pack_st, st.integers(0, 6), st.integers(0, 3))
def test_corrupted_descriptor_is_an_error(pack, kind, b):
    """Every broken invariant of the descriptor comes back as PP_ERR_BAD_LAYOUT
    from the host checks, before anything else runs (never a crash or a plan)."""
    b = b % pack.num_rows
    if kind in (4, 6):
        assume(pack.num_resp[b] >= 1)
    bad = _corrupt(pack, kind, b)
    for call in (lambda p: binding.pp_pack_export(p, 32, 32),
                 lambda p: binding.pp_workspace_size(p, 4, 2, 128, fwd=True, bwd=True, loss=False),
                 lambda p: binding.pp_pack_stats(p)):
        with pytest.raises(binding.PPError) as e:
            call(bad)
        assert binding.STATUS[e.value.status] == "PP_ERR_BAD_LAYOUT", (kind, e.value)


def _causal_attention(q, k, v, G, scale):
    """Plain causal attention of one sequence, fp64, with its LSE."""
    T, hq, _ = q.shape
    kk = k.repeat_interleave(G, dim=1)
    vv = v.repeat_interleave(G, dim=1)
    s = torch.einsum("ihd,jhd->hij", q, kk) * scale
    s = s.masked_fill(torch.triu(torch.ones(T, T, dtype=torch.bool), 1), float("-inf"))
    lse = torch.logsumexp(s, dim=-1)
    out = torch.einsum("hij,jhd->ihd", torch.exp(s - lse[..., None]), vv)
    return out, lse


small_row_st = st.tuples(st.integers(0, 24), st.lists(st.integers(0, 16), max_size=3), st.integers(0, 4))


@settings(max_examples=40, deadline=None, derandomize=True)
@given(st.lists(small_row_st, min_size=1, max_size=2).map(_pack), st.integers(0, 2**31 - 1))
def test_oracle_packed_attention_equals_unpacked(pack, seed):
    """Fact (a) of Sec. 3.2 on the oracle: each (prompt, response_k) sequence
    taken out of the packed row and attended causally on its own gives the packed
    outputs and LSE of its tokens; padding rows are zero."""
    hq, hkv, d = 4, 2, 8
    T = pack.total_tokens
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(T, hq, d, generator=g, dtype=torch.float64)
    k = torch.randn(T, hkv, d, generator=g, dtype=torch.float64)
    v = torch.randn(T, hkv, d, generator=g, dtype=torch.float64)
    args = pack.oracle_args()
    O, LSE = orc.attn_fwd(*args, q.numpy(), k.numpy(), v.numpy())
    covered = np.zeros(T, bool)
    for b in range(pack.num_rows):
        r0, _, P, offs, lens = orc._row_fields(*args, b)
        seqs = [list(range(P)) + list(range(o, o + n)) for o, n in zip(offs, lens)] or [list(range(P))]
        for idx in seqs:
            if not idx:
                continue
            flat = [r0 + x for x in idx]
            out, lse = _causal_attention(q[flat], k[flat], v[flat], hq // hkv, 1.0 / math.sqrt(d))
            assert np.abs(out.numpy() - O[flat]).max() < 1e-12
            assert np.abs(lse.numpy().T - LSE[:, flat].T).max() < 1e-12
            covered[flat] = True
    assert (O[~covered] == 0).all() and (LSE[:, ~covered] == 0).all()
