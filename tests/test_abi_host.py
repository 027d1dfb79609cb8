"""Host-side tests of the C ABI: the library loads and exports every declared
symbol, the planner's integer outputs equal the oracle's bit for bit, and bad
arguments come back as error codes before anything touches a GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import pp_oracle as orc
from paper_2602_24082_amd import binding
from paper_2602_24082_amd import workload as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = []
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            src = open(os.path.join(ROOT, "include", fn)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names += re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\**\s+(pp_[a-z_]+)\s*\(", src, re.M)
    return sorted(set(names))


def test_library_exports_every_declared_symbol():
    L = binding.lib()
    declared = _declared_functions()
    assert "pp_attn_fwd" in declared and "pp_dpo_loss" in declared
    for name in declared:
        assert hasattr(L, name), name
    assert set(binding.EXPORTED) <= set(declared)


def test_status_strings():
    L = binding.lib()
    for s in range(6):
        assert L.pp_status_string(s)
    assert L.pp_version() >= 100


def _random_pack(rng, B=None, pad=True, zero_prompt_ok=True):
    B = B or int(rng.integers(1, 5))
    P = [int(rng.integers(0 if zero_prompt_ok else 1, 40)) for _ in range(B)]
    L = [[int(x) for x in rng.integers(0, 30, size=int(rng.integers(0, 5)))] for _ in range(B)]
    padv = [int(rng.integers(0, 9)) if pad else 0 for _ in range(B)]
    return wl.make_pack(P, L, pad=padv)


@pytest.mark.parametrize("bq,bk", [(1, 1), (2, 3), (16, 16), (32, 64), (128, 64), (128, 128), (7, 5)])
def test_export_matches_oracle_bit_exact(bq, bk):
    rng = np.random.default_rng(bq * 1000 + bk)
    for _ in range(8):
        pack = _random_pack(rng)
        pos, seg, tiles = binding.pp_pack_export(pack, bq, bk)
        args = pack.oracle_args()
        assert (pos == orc.pack_position_ids(*args)).all()
        assert (seg == orc.pack_segment_ids(*args)).all()
        assert (tiles == orc.pack_tile_classes(*args, bq, bk)).all()


def test_export_golden_fixture_row():
    pack = wl.make_pack([3], [[2, 2]], pad=[1])
    pos, seg, tiles = binding.pp_pack_export(pack, 2, 2)
    assert pos.tolist() == [0, 1, 2, 3, 4, 3, 4, 0]
    assert seg.tolist() == [0, 0, 0, 1, 1, 2, 2, -1]
    assert tiles.reshape(4, 4).tolist() == [[1, 0, 0, 0], [2, 1, 0, 0], [2, 1, 1, 0], [1, 1, 1, 1]]


def test_export_config_sized_rows():
    """Full-size rows of the 8B-shaped workload at the kernels' own tile sizes."""
    pack = wl.config_pack(wl.LLAMA3_8B, rows=2)
    for bq, bk in [(128, 64), (32, 128)]:
        _, _, tiles = binding.pp_pack_export(pack, bq, bk)
        assert (tiles == orc.pack_tile_classes(*pack.oracle_args(), bq, bk)).all()


# ------------------------------------------------------------- error codes


def _raw_desc(row_start, prompt, num, off, ln, kmax):
    arrs = [np.asarray(x, np.int32) for x in (row_start, prompt, num, off, ln)]
    ptr = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    d = binding._Desc(len(prompt), kmax, *[ptr(a) for a in arrs])
    return d, arrs


def _fwd_status(desc, hq=4, hkv=2, d=64, dtype=0):
    L = binding.lib()
    fake = ctypes.c_void_p(16)  # never dereferenced: validation fails first
    return L.pp_attn_fwd(ctypes.byref(desc), dtype, hq, hkv, d, 0.0, fake, fake, fake, fake, fake,
                         fake, 1 << 30, None)


def test_bad_layouts_are_rejected_before_launch():
    good, a = _raw_desc([0, 10], [4], [2], [4, 7], [3, 3], 2)
    cases = [
        (_raw_desc([0, 10], [4], [2], [4, 8], [3, 2], 2), 2),     # gap between responses
        (_raw_desc([0, 10], [4], [2], [5, 8], [3, 2], 2), 2),     # first response not at P
        (_raw_desc([0, 8], [4], [2], [4, 7], [3, 3], 2), 2),      # overflows the row
        (_raw_desc([0, 10], [-1], [0], [0, 0], [0, 0], 2), 2),    # negative prompt
        (_raw_desc([0, 10], [4], [3], [4, 7], [3, 3], 2), 2),     # more responses than max
        (_raw_desc([0, 10], [4], [2], [4, 4], [-1, 3], 2), 2),    # negative length
        (_raw_desc([1, 10], [4], [0], [0, 0], [0, 0], 2), 2),     # row_start[0] != 0
        (_raw_desc([0, 10, 5], [4, 0], [0, 0], [0, 0, 0, 0], [0, 0, 0, 0], 2), 2),  # decreasing
    ]
    for (d, keep), want in cases:
        assert _fwd_status(d) == want, binding.lib().pp_last_error()
        assert binding.lib().pp_last_error()


def test_bad_heads_and_dims():
    d, keep = _raw_desc([0, 10], [4], [2], [4, 7], [3, 3], 2)
    assert _fwd_status(d, hq=4, hkv=3) == 1
    assert _fwd_status(d, hq=0, hkv=1) == 1
    assert _fwd_status(d, d=96) == 3
    assert _fwd_status(d, d=256) == 3
    assert _fwd_status(d, dtype=7) == 1


def test_workspace_too_small_and_nulls():
    L = binding.lib()
    d, keep = _raw_desc([0, 10], [4], [2], [4, 7], [3, 3], 2)
    fake = ctypes.c_void_p(16)
    st = L.pp_attn_fwd(ctypes.byref(d), 0, 4, 2, 64, 0.0, fake, fake, fake, fake, fake, fake, 1, None)
    assert st == 4
    st = L.pp_attn_fwd(ctypes.byref(d), 0, 4, 2, 64, 0.0, None, fake, fake, fake, fake, fake, 1 << 30, None)
    assert st == 1
    assert L.pp_attn_fwd(None, 0, 4, 2, 64, 0.0, fake, fake, fake, fake, fake, fake, 1 << 30, None) == 1


def test_logprob_needs_a_prompt():
    L = binding.lib()
    d, keep = _raw_desc([0, 5], [0], [1], [0], [5], 1)
    fake = ctypes.c_void_p(16)
    st = L.pp_seq_logprob(ctypes.byref(d), 0, 100, fake, fake, fake, None, fake, 1 << 30, None)
    assert st == 2
    # the same row is fine for attention (document-masked packing)
    assert binding.pp_workspace_size(wl.make_pack([0], [[5]]), 2, 1, 64)[0] > 0


def test_logprob_bwd_argument_checks():
    L = binding.lib()
    fake = ctypes.c_void_p(16)
    d, keep = _raw_desc([0, 5], [0], [1], [0], [5], 1)
    assert L.pp_seq_logprob_bwd(ctypes.byref(d), 0, 100, fake, fake, fake, fake, fake, 1 << 30, None) == 2
    d, keep = _raw_desc([0, 12], [4], [2], [4, 7], [3, 3], 2)
    assert L.pp_seq_logprob_bwd(ctypes.byref(d), 0, 0, fake, fake, fake, fake, fake, 1 << 30, None) == 1
    assert L.pp_seq_logprob_bwd(ctypes.byref(d), 0, 100, fake, fake, None, fake, fake, 1 << 30, None) == 1
    assert L.pp_seq_logprob_bwd(ctypes.byref(d), 0, 100, fake, fake, fake, None, fake, 1 << 30, None) == 1
    assert L.pp_seq_logprob_bwd(ctypes.byref(d), 0, 100, fake, fake, fake, fake, fake, 1, None) == 4
    # more responses per row than the backward stages per logit row
    K = 257
    d, keep = _raw_desc([0, 300], [10], [K], [10 + k for k in range(K)], [1] * K, K)
    assert L.pp_seq_logprob_bwd(ctypes.byref(d), 0, 100, fake, fake, fake, fake, fake, 1 << 30, None) == 3


def test_rm_head_argument_checks():
    L = binding.lib()
    fake = ctypes.c_void_p(16)
    d, keep = _raw_desc([0, 12], [4], [2], [4, 7], [3, 3], 2)
    n = ctypes.c_size_t(0)
    assert L.pp_rm_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0 and n.value > 0
    assert L.pp_rm_workspace_size(ctypes.byref(d), None) == 1
    assert L.pp_rm_scores(ctypes.byref(d), 0, 0, fake, fake, 0.0, fake, fake, 1 << 30, None) == 1
    assert L.pp_rm_scores(ctypes.byref(d), 7, 64, fake, fake, 0.0, fake, fake, 1 << 30, None) == 1
    assert L.pp_rm_scores(ctypes.byref(d), 0, 64, fake, None, 0.0, fake, fake, 1 << 30, None) == 1
    assert L.pp_rm_scores(ctypes.byref(d), 0, 64, fake, fake, 0.0, fake, fake, 1, None) == 4
    assert L.pp_rm_scores_bwd(ctypes.byref(d), 0, 64, fake, fake, None, fake, fake, None, fake, 1 << 30, None) == 1
    assert L.pp_rm_scores_bwd(ctypes.byref(d), 0, 64, fake, fake, fake, fake, fake, None, fake, 1, None) == 4
    bad, keep2 = _raw_desc([0, 12], [4], [2], [5, 7], [3, 3], 2)  # gap after the prompt
    assert L.pp_rm_scores(ctypes.byref(bad), 0, 64, fake, fake, 0.0, fake, fake, 1 << 30, None) == 2


def test_pack_stats_against_oracle():
    # single rows: the ratios are the oracle's per-data-point cost model (pinned
    # against Table 1); multi-row batches: counts against explicit masks
    for P, lens in [(228, [251, 130]), (720, [469, 331]), (600, [110, 90]), (64, [1000, 900]), (5, [0, 3, 7])]:
        st = binding.pp_pack_stats(wl.make_pack([P], [lens]))
        nz = [L for L in lens]
        assert st["eq1_cost_ratio"] == pytest.approx(orc.cost_ratio(P, nz), rel=1e-12)
        assert st["eq1_memory_ratio"] == pytest.approx(orc.memory_ratio(P, nz), rel=1e-12)
        assert st["rows_eq1_cheaper"] == int(orc.packing_is_cheaper(P, nz))
    rng = np.random.default_rng(11)
    for _ in range(6):
        pack = _random_pack(rng, zero_prompt_ok=True)
        st = binding.pp_pack_stats(pack)
        args = pack.oracle_args()
        packed = unpacked = dense = tok_p = tok_u = 0
        seqs = []
        for b in range(pack.num_rows):
            r0, T, P, offs, lens = orc._row_fields(*args, b)
            packed += int(orc.row_mask(T, P, offs, lens).sum())
            n = P + sum(lens)
            dense += n * (n + 1) // 2
            tok_p += n
            for L in (lens if lens else [0]):
                m = orc.row_mask(P + L, P, [P], [L]) if lens else orc.row_mask(P, P, [], [])
                unpacked += int(m.sum())
                tok_u += P + L
                seqs.append(P + L)
        assert st["pairs_packed"] == packed == orc.useful_pairs(pack.prompt_len, pack.num_resp, pack.resp_len)
        assert st["pairs_unpacked"] == unpacked and st["pairs_dense_packed"] == dense
        assert st["tokens_packed"] == tok_p and st["tokens_unpacked"] == tok_u
        assert st["tokens_padded"] == len(seqs) * max(seqs)
        assert st["rows_eq1_cheaper"] == sum(
            int(orc.packing_is_cheaper(int(pack.prompt_len[b]), list(pack.resp_len[b, :int(pack.num_resp[b])])))
            for b in range(pack.num_rows) if int(pack.num_resp[b]) > 0)


def test_loss_argument_checks():
    L = binding.lib()
    fake = ctypes.c_void_p(16)
    nr = np.array([1, 0], np.int32)
    st = L.pp_dpo_loss(2, 2, ctypes.c_void_p(nr.ctypes.data), fake, None, 0.1, fake, None, None, fake, 4096, None)
    assert st == 1  # no row with two responses
    nr = np.array([3, 2], np.int32)
    st = L.pp_dpo_loss(2, 2, ctypes.c_void_p(nr.ctypes.data), fake, None, 0.1, fake, None, None, fake, 4096, None)
    assert st == 1  # num_resp above max_resp
    nr = np.array([2, 2], np.int32)
    st = L.pp_dpo_loss(2, 2, ctypes.c_void_p(nr.ctypes.data), fake, None, 0.1, fake, None, None, fake, 4, None)
    assert st == 4  # workspace


def test_workspace_sizes_grow_with_batch():
    small = wl.config_pack(wl.TINY_FP32)
    big = wl.config_pack(wl.LLAMA3_8B)
    a = binding.pp_workspace_size(small, 4, 4, 64, 1000, logprob=True)
    b = binding.pp_workspace_size(big, 32, 8, 128, 128256, logprob=True)
    assert all(x > 0 for x in a) and all(y >= x for x, y in zip(a, b))


def test_rope_argument_checks():
    """Rotary entry points: bad base, head_dim, NULLs and workspace come back as
    error codes before anything is enqueued."""
    L = binding.lib()
    fake = ctypes.c_void_p(16)
    d, keep = _raw_desc([0, 12], [4], [2], [4, 7], [3, 3], 2)
    n = ctypes.c_size_t(0)
    assert L.pp_rope_workspace_size(ctypes.byref(d), 128, ctypes.byref(n)) == 0 and n.value >= 12 * 4 + 64 * 8
    assert L.pp_rope_workspace_size(ctypes.byref(d), 12, ctypes.byref(n)) == 3
    assert L.pp_rope_workspace_size(ctypes.byref(d), 128, None) == 1
    rope = lambda dt=0, H=2, hd=128, base=10000.0, x=fake, y=fake, nb=1 << 30: L.pp_rope(
        ctypes.byref(d), dt, H, hd, base, 0, x, y, fake, nb, None)
    assert rope(hd=100) == 3
    assert rope(base=0.0) == 1 and rope(base=-5.0) == 1 and rope(base=float("inf")) == 1
    assert rope(H=0) == 1 and rope(dt=9) == 1
    assert rope(x=None) == 1 and rope(y=None) == 1
    assert rope(nb=1) == 4
    fwd = lambda base=10000.0, qr=fake, kr=fake, hd=128, nb=1 << 30: L.pp_attn_fwd_rope(
        ctypes.byref(d), 0, 4, 2, hd, 0.0, base, fake, fake, fake, fake, fake, qr, kr, fake, nb, None)
    assert fwd(base=0.0) == 1
    assert fwd(kr=None) == 1
    assert fwd(hd=96) == 3
    assert fwd(nb=1) == 4
    bwd = lambda base=10000.0, nb=1 << 30: L.pp_attn_bwd_rope(
        ctypes.byref(d), 0, 4, 2, 128, 0.0, base, fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, nb,
        None)
    assert bwd(base=float("nan")) == 1
    assert bwd(nb=1) == 4


def test_misaligned_tensors_rejected():
    """Attention and rotary tensors must be 16-byte aligned (lse 4-byte): a
    misaligned pointer comes back as PP_ERR_INVALID_ARGUMENT before anything is
    enqueued."""
    L = binding.lib()
    ok, off8, off2 = ctypes.c_void_p(4096), ctypes.c_void_p(4096 + 8), ctypes.c_void_p(4096 + 2)
    d, keep = _raw_desc([0, 12], [4], [2], [4, 7], [3, 3], 2)
    nb = 1 << 30

    def fwd(q=ok, k=ok, v=ok, o=ok, lse=ok):
        return L.pp_attn_fwd(ctypes.byref(d), 0, 4, 2, 128, 0.0, q, k, v, o, lse, ok, nb, None)

    for kw in ("q", "k", "v", "o"):
        assert fwd(**{kw: off8}) == 1, kw
    assert fwd(lse=off2) == 1
    assert b"aligned" in L.pp_last_error()

    def bwd(**kw):
        a = dict(q=ok, k=ok, v=ok, o=ok, lse=ok, dout=ok, dq=ok, dk=ok, dv=ok)
        a.update(kw)
        return L.pp_attn_bwd(ctypes.byref(d), 0, 4, 2, 128, 0.0, a["q"], a["k"], a["v"], a["o"], a["lse"],
                             a["dout"], a["dq"], a["dk"], a["dv"], ok, nb, None)

    for kw in ("q", "k", "v", "o", "dout", "dq", "dk", "dv"):
        assert bwd(**{kw: off8}) == 1, kw
    assert bwd(lse=off2) == 1
    rope = lambda x=ok, y=ok: L.pp_rope(ctypes.byref(d), 0, 2, 128, 10000.0, 0, x, y, ok, nb, None)
    assert rope(x=off8) == 1 and rope(y=off8) == 1
    fwd_r = lambda qr=ok, kr=ok: L.pp_attn_fwd_rope(ctypes.byref(d), 0, 4, 2, 128, 0.0, 10000.0, ok, ok, ok, ok, ok,
                                                    qr, kr, ok, nb, None)
    assert fwd_r(qr=off8) == 1 and fwd_r(kr=off8) == 1


def test_plan_argument_checks():
    """Reusable plans: size query, creation and the planned calls validate their
    arguments on the host; a plan of an empty pack needs no copy, so its whole
    lifecycle runs here."""
    L = binding.lib()
    ok = ctypes.c_void_p(4096)
    d, keep = _raw_desc([0, 12], [4], [2], [4, 7], [3, 3], 2)
    n = ctypes.c_size_t(0)
    assert L.pp_plan_workspace_size(ctypes.byref(d), 0, 4, 2, 128, ctypes.byref(n)) == 0
    f, b = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert L.pp_workspace_size(ctypes.byref(d), 0, 4, 2, 128, 0, ctypes.byref(f), ctypes.byref(b), None, None) == 0
    assert n.value >= f.value + b.value
    assert L.pp_plan_workspace_size(ctypes.byref(d), 0, 4, 2, 96, ctypes.byref(n)) == 3
    assert L.pp_plan_workspace_size(ctypes.byref(d), 0, 4, 3, 128, ctypes.byref(n)) == 1
    assert L.pp_plan_workspace_size(ctypes.byref(d), 0, 4, 2, 128, None) == 1
    h = ctypes.c_void_p(1234)
    assert L.pp_plan_create(ctypes.byref(d), 0, 4, 2, 128, None, ok, 1 << 30, None, None) == 1
    assert L.pp_plan_create(ctypes.byref(d), 0, 4, 2, 128, None, ok, 16, None, ctypes.byref(h)) == 4
    assert h.value is None  # no handle on error
    bad = ctypes.c_float(-1.0)
    assert L.pp_plan_create(ctypes.byref(d), 0, 4, 2, 128, ctypes.byref(bad), ok, 1 << 30, None,
                            ctypes.byref(h)) == 1
    assert L.pp_attn_fwd_planned(None, 0.0, ok, ok, ok, ok, ok, None, None, None) == 1
    assert L.pp_attn_bwd_planned(None, 0.0, ok, ok, ok, ok, ok, ok, ok, ok, ok, None) == 1
    assert L.pp_plan_destroy(None) == 0
    # an empty pack (one row of no tokens): create, use and destroy without a device
    e, keep_e = _raw_desc([0, 0], [0], [0], [0], [0], 1)
    assert L.pp_plan_workspace_size(ctypes.byref(e), 0, 4, 2, 128, ctypes.byref(n)) == 0
    ws = ctypes.c_void_p(4096) if n.value else None
    assert L.pp_plan_create(ctypes.byref(e), 0, 4, 2, 128, None, ws, n.value, None, ctypes.byref(h)) == 0
    assert h.value is not None
    assert L.pp_attn_fwd_planned(h, 0.0, ok, ok, ok, ok, ok, None, None, None) == 0
    assert L.pp_attn_fwd_planned(h, 0.0, ok, ok, ctypes.c_void_p(4096 + 8), ok, ok, None, None, None) == 1
    assert L.pp_attn_bwd_planned(h, 0.0, ok, ok, ok, ok, ok, ok, ok, ok, ok, None) == 0
    assert L.pp_plan_destroy(h) == 0


def test_timing_select_accepts_lists():
    L = binding.lib()
    for arg in (None, b"", b"pp_attn_fwd", b"pp_attn_fwd,pp_logprob_rows", b",pp_attn_bwd_dq,,", b","):
        assert L.pp_timing_select(arg) == 0, arg
    assert L.pp_timing_select(None) == 0
    # nothing was launched, so nothing was timed
    assert L.pp_timing_reset() == 0 and L.pp_timing_count() == 0


def test_misaligned_workspace_rejected():
    """A workspace off a 256-byte boundary is refused before anything is enqueued."""
    L = binding.lib()
    ok = ctypes.c_void_p(4096)
    off = ctypes.c_void_p(4096 + 16)
    big = 1 << 30
    d, keep = _raw_desc([0, 12], [4], [2], [4, 7], [3, 3], 2)
    assert L.pp_attn_fwd(ctypes.byref(d), 0, 4, 2, 64, 0.0, ok, ok, ok, ok, ok, off, big, None) == 1
    assert L.pp_attn_bwd(ctypes.byref(d), 0, 4, 2, 64, 0.0, ok, ok, ok, ok, ok, ok, ok, ok, ok, off, big, None) == 1
    assert L.pp_seq_logprob(ctypes.byref(d), 0, 1000, ok, ok, ok, None, off, big, None) == 1
    num = (ctypes.c_int32 * 2)(2, 2)
    assert L.pp_dpo_loss(2, 2, num, ok, ok, ctypes.c_float(0.1), ok, None, None, off, big, None) == 1
    h = ctypes.c_void_p(0)
    assert L.pp_plan_create(ctypes.byref(d), 0, 4, 2, 128, None, off, big, None, ctypes.byref(h)) == 1
    assert h.value is None
    assert b"256-byte" in L.pp_last_error()


def test_noalloc_forward_rejects_packs_beyond_its_static_scratch():
    """pp_attn_fwd_noalloc checks, before anything touches a GPU, that the pack's
    plan fits the library's static scratch, and names the limit when it does
    not (2000 rows of 300 tokens: 600K tokens of per-token metadata, > 4 MiB)."""
    import torch
    pack = wl.make_pack([200] * 2000, [[50, 50]] * 2000)
    f, = binding.pp_workspace_size(pack, 8, 2, 128, fwd=True, bwd=False, loss=False)[:1]
    assert f > binding.NOALLOC_SCRATCH_BYTES
    h = binding._DescHolder(pack)
    L = binding.lib()
    dummy = ctypes.c_void_p(1 << 12)  # never dereferenced: the size check comes first
    st = L.pp_attn_fwd_noalloc(h.ref, 8, 2, 128, 0.0, dummy, dummy, dummy, dummy, dummy, None)
    assert st == 4  # PP_ERR_WORKSPACE_TOO_SMALL
    msg = L.pp_last_error().decode()
    assert str(binding.NOALLOC_SCRATCH_BYTES) in msg and str(f) in msg
    # and bad arguments are still reported as such, not as a size problem
    small = wl.make_pack([20], [[5, 5]])
    hs = binding._DescHolder(small)
    assert L.pp_attn_fwd_noalloc(hs.ref, 8, 3, 128, 0.0, dummy, dummy, dummy, dummy, dummy, None) == 1
    assert L.pp_attn_fwd_noalloc(hs.ref, 8, 2, 96, 0.0, dummy, dummy, dummy, dummy, dummy, None) == 3


def test_stored_ds_region_is_one_tile_per_visible_block_and_head():
    """The backward's stored-dS region -- the difference between the stored-dS
    mode's workspace and the default one -- holds one 32 x 32 bf16 tile (2 KB) per query head
    for every 32 x 32 block of a row's mask that has a visible pair (the
    oracle's dense mask), and nothing more: the visible queries of 32
    consecutive keys form one run from the block's diagonal, which is what the
    key-major pass computes and stores.  Also for plans."""
    rng = np.random.default_rng(7)
    packs = [_random_pack(rng) for _ in range(16)]
    packs += [wl.make_pack([300], [[200, 5, 130]], pad=[17]), wl.make_pack([0], [[64, 64]]),
              wl.make_pack([40], [[]]), wl.make_pack([127, 1], [[1, 129, 2], [0, 33]])]
    for pack in packs:
        n_blocks = int((orc.pack_tile_classes(*pack.oracle_args(), 32, 32) > 0).sum())
        for hq, hkv in ((4, 2), (3, 1)):
            lean = binding.pp_workspace_size(pack, hq, hkv, 64, fwd=False, bwd=True, loss=False)[1]
            full, plan_full = binding.pp_bwd_stored_ds_workspace_size(pack, hq, hkv, 64)
            assert full - lean == hq * n_blocks * 2048
            assert plan_full - binding.pp_plan_workspace_size(pack, hq, hkv, 64) == hq * n_blocks * 2048


def test_backward_below_the_recompute_workspace_is_refused():
    pack = wl.make_pack([50], [[20, 30]])
    lean = binding.pp_workspace_size(pack, 2, 1, 64, fwd=False, bwd=True, loss=False)[1]
    full, _ = binding.pp_bwd_stored_ds_workspace_size(pack, 2, 1, 64)
    assert 0 < lean < full
    L = binding.lib()
    h = binding._DescHolder(pack)
    fake = ctypes.c_void_p(256)  # never dereferenced: the size check comes first
    st = L.pp_attn_bwd(h.ref, binding.PP_BF16, 2, 1, 64, 0.0, fake, fake, fake, fake, fake, fake, fake, fake,
                       fake, fake, lean - 1, None)
    assert binding.STATUS[st] == "PP_ERR_WORKSPACE_TOO_SMALL"
    assert b"with the stored dS" in L.pp_last_error()
