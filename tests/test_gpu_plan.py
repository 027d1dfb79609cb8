"""GPU tests of the reusable plan (pp_plan_create + pp_attn_{fwd,bwd}_planned).

The planned calls run the same kernels on the same metadata as the
self-contained entry points, so their outputs must be bit-identical to
pp_attn_fwd / pp_attn_bwd (and the rotary variants) for the same inputs; one
case is also checked against the oracle directly, at the attention tolerances
(O max-abs <= 1e-2 beyond its bf16 rounding, LSE within 2e-4 + 2^-16 |LSE|; dQ, dK, dV
relative Frobenius <= 2e-2 on the whole tensor and on every prompt and response).  A plan is
reused for several "layers" (different q, k, v) and does not depend on the
caller's descriptor arrays after creation.
"""
import numpy as np
import pytest
import torch

from oracle import pp_oracle as orc
from paper_2602_24082_amd import binding as pp
from paper_2602_24082_amd import workload as wl
from gradcheck import check_grad
from tolerances import lse_excess, o_excess

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _ragged():
    return wl.make_pack([300, 0, 129, 5, 64], [[70, 45], [33, 64], [1, 0, 200], [130], [64, 64]],
                        pad=[3, 0, 0, 17, 0])


@pytest.mark.parametrize("dtype,d,hq,hkv,store_ds", [(torch.bfloat16, 128, 8, 2, False),
                                                      (torch.bfloat16, 64, 4, 4, False),
                                                      (torch.float32, 64, 4, 2, False),
                                                      (torch.bfloat16, 128, 8, 2, True)])
def test_planned_equals_self_contained(dtype, d, hq, hkv, store_ds):
    """A plan made with the larger workspace runs the stored-dS backward, as the
    self-contained call does with its larger workspace."""
    pack = _ragged()
    print(f"case plan T={pack.total_tokens} d={d} hq={hq} hkv={hkv} {dtype} store_ds={store_ds}", flush=True)
    code = pp.PP_FP32 if dtype == torch.float32 else pp.PP_BF16
    plan = pp.pp_plan_create(pack, hq, hkv, d, dtype=code, device=DEV, store_ds=store_ds)
    for layer in range(3):
        q, k, v, do = wl.qkv(pack, hq, hkv, d, 300 + layer, dtype, device=DEV)
        o1, l1 = pp.pp_attn_fwd(pack, q, k, v)
        o2, l2 = pp.pp_attn_fwd_planned(plan, q, k, v)
        g1 = pp.pp_attn_bwd(pack, q, k, v, o1, l1, do, store_ds=store_ds)
        g2 = pp.pp_attn_bwd_planned(plan, q, k, v, o2, l2, do)
        torch.cuda.synchronize()
        assert torch.equal(o1, o2) and torch.equal(l1, l2), layer
        for a, b in zip(g1, g2):
            assert torch.equal(a, b), layer
    pp.pp_plan_destroy(plan)


def test_planned_matches_oracle():
    pack = _ragged()
    hq, hkv, d = 8, 2, 128
    print(f"case plan-oracle T={pack.total_tokens}", flush=True)
    # the binding's descriptor arrays are released as soon as pp_plan_create
    # returns: the plan keeps its own copy of everything it needs
    plan = pp.pp_plan_create(pack, hq, hkv, d, device=DEV)
    q, k, v, do = wl.qkv(pack, hq, hkv, d, 41, torch.bfloat16, device="cpu")
    o, lse = pp.pp_attn_fwd_planned(plan, *(x.to(DEV) for x in (q, k, v)))
    dq, dk, dv = pp.pp_attn_bwd_planned(plan, q.to(DEV), k.to(DEV), v.to(DEV), o, lse, do.to(DEV))
    args = pack.oracle_args()
    qn, kn, vn, don = (x.double().numpy() for x in (q, k, v, do))
    O, L = orc.attn_fwd(*args, qn, kn, vn)
    assert o_excess(o.double().cpu().numpy(), O, True) <= 0
    assert lse_excess(lse.double().cpu().numpy(), L) <= 0
    for name, got, ref in zip(("dq", "dk", "dv"), (dq, dk, dv), orc.attn_bwd(*args, qn, kn, vn, don)):
        g = got.double().cpu().numpy()
        assert np.isfinite(g).all()
        check_grad(pack, name, g, ref)


def test_rotary_plan_equals_rotary_entry_points():
    pack = wl.make_pack([500, 77], [[100, 28, 300], [64, 64]], pad=[0, 5])
    hq, hkv, d, base = 8, 2, 128, 500000.0
    print(f"case plan-rope T={pack.total_tokens}", flush=True)
    q, k, v, do = wl.qkv(pack, hq, hkv, d, 77, torch.bfloat16, device=DEV)
    plan = pp.pp_plan_create(pack, hq, hkv, d, rope_base=base, device=DEV)
    o1, l1, qr1, kr1 = pp.pp_attn_fwd_rope(pack, q, k, v, base)
    qr2 = torch.empty_like(q)
    o2, l2, qr2, kr2 = pp.pp_attn_fwd_planned(plan, q, k, v, q_rot=qr2)
    g1 = pp.pp_attn_bwd_rope(pack, qr1, kr1, v, o1, l1, do, base)
    g2 = pp.pp_attn_bwd_planned(plan, qr2, kr2, v, o2, l2, do)
    torch.cuda.synchronize()
    for a, b in [(o1, o2), (l1, l2), (qr1, qr2), (kr1, kr2), *zip(g1, g2)]:
        assert torch.equal(a, b)
    pp.pp_plan_destroy(plan)


def test_planned_full_size_workload_matches_self_contained():
    """The 8B-shaped benchmark batch: planned == self-contained, bit for bit."""
    cfg = wl.LLAMA3_8B
    pack = wl.config_pack(cfg)
    print(f"case plan-fullsize {cfg.name} T={pack.total_tokens}", flush=True)
    q, k, v, do = wl.qkv(pack, cfg.hq, cfg.hkv, cfg.head_dim, 9, torch.bfloat16, DEV)
    plan = pp.pp_plan_create(pack, cfg.hq, cfg.hkv, cfg.head_dim, device=DEV)
    o1, l1 = pp.pp_attn_fwd(pack, q, k, v)
    o2, l2 = pp.pp_attn_fwd_planned(plan, q, k, v)
    g1 = pp.pp_attn_bwd(pack, q, k, v, o1, l1, do)
    g2 = pp.pp_attn_bwd_planned(plan, q, k, v, o2, l2, do)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)


def test_timing_select_times_only_the_named_launches():
    pack = _ragged()
    q, k, v, do = wl.qkv(pack, 8, 2, 128, 501, torch.bfloat16, device=DEV)
    print(f"case timing-select T={pack.total_tokens}", flush=True)
    try:
        pp.pp_timing_select(["pp_attn_fwd", "pp_attn_bwd_dq"])
        pp.pp_timing_reset()
        pp.pp_timing_enable(True)
        for _ in range(3):
            o, lse = pp.pp_attn_fwd(pack, q, k, v)
            pp.pp_attn_bwd(pack, q, k, v, o, lse, do)
        torch.cuda.synchronize()
        pp.pp_timing_enable(False)
        got = pp.pp_timing_get()
        assert set(got) == {"pp_attn_fwd", "pp_attn_bwd_dq"}
        assert all(n == 3 and ms > 0 for ms, n in got.values())
        # back to every launch
        pp.pp_timing_select(None)
        pp.pp_timing_reset()
        pp.pp_timing_enable(True)
        o, lse = pp.pp_attn_fwd(pack, q, k, v)
        pp.pp_attn_bwd(pack, q, k, v, o, lse, do)
        torch.cuda.synchronize()
        pp.pp_timing_enable(False)
        assert {"pp_attn_fwd", "pp_attn_bwd_dkdv", "pp_attn_bwd_dq", "pp_stage"} <= set(pp.pp_timing_get())
    finally:
        pp.pp_timing_enable(False)
        pp.pp_timing_select(None)
        pp.pp_timing_reset()


def test_self_contained_calls_from_two_threads():
    """Two host threads, each on its own stream, call the self-contained entry
    points (which stage their metadata through the shared pinned ring) over and
    over; every result equals the single-threaded one bit for bit."""
    import threading
    packs = [_ragged(), wl.make_pack([500, 77], [[100, 28, 300], [64, 64]], pad=[0, 5])]
    hq, hkv, d = 8, 2, 128
    inputs = [wl.qkv(pk, hq, hkv, d, 600 + i, torch.bfloat16, device=DEV) for i, pk in enumerate(packs)]
    print(f"case two-threads T={[pk.total_tokens for pk in packs]}", flush=True)

    def run(i):
        q, k, v, do = inputs[i]
        o, lse = pp.pp_attn_fwd(packs[i], q, k, v)
        return (o, lse, *pp.pp_attn_bwd(packs[i], q, k, v, o, lse, do))

    want = [run(i) for i in range(2)]
    torch.cuda.synchronize()
    errors = []

    def worker(i):
        try:
            s = torch.cuda.Stream(device=DEV)
            with torch.cuda.stream(s):
                for _ in range(12):
                    got = run(i)
                    s.synchronize()
                    if not all(torch.equal(a, b) for a, b in zip(got, want[i])):
                        errors.append(f"thread {i}: result differs")
                        return
        except Exception as e:  # surfaced below
            errors.append(f"thread {i}: {e!r}")

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker did not finish"
    assert not errors, errors
