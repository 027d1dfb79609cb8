"""Benchmark of the preference-packing hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config WORKLOAD]

One step = one pass of the whole hot path over one packed batch of the
Llama-3-8B-shaped workload (8 rows, 32 query / 8 kv heads, head_dim 128, prompt
U[256,1536], K=2 responses U[64,512], bf16):

    plan -> attention forward -> attention backward (dQ, dK, dV)
         -> per-response log-probs of policy and reference logits
            (Llama-3 vocabulary 128256, bf16) -> DPO loss (beta 0.1)

The headline value is the attention's useful throughput: only visible
(query, key) pairs count, 4*d*Hq per pair forward and 10*d*Hq backward
(the FlashAttention convention), divided by the attention's own time inside
the timed steps (HIP events on the stream).  Printed as ONE JSON line, with the
roofline of the dominant kernel (its algorithmic FLOPs or bytes per launch over
its average launch time, from the library's per-launch HIP events), the oracle
timed on the host cores on a bounded sample, and the speedup over the same
kernels on the unpacked, prompt-duplicated, padded layout.

    python bench.py --calib-copy      # plain device copy of known size, for
                                      # scaling rocprofv3 FETCH_SIZE/WRITE_SIZE
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2602_24082_amd import binding as pp  # noqa: E402
from paper_2602_24082_amd import workload as wl  # noqa: E402

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA (vendor, 2.4 GHz)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E (vendor)
LOGPROB_VOCAB = 128256      # Llama-3 vocabulary for the 8B-shaped workload
HIDDEN_DIM = {32: 4096, 64: 8192}  # model width by query-head count (Llama-3-8B, Qwen2-72B)
LOGPROB_SIGMA = 3.0
ROPE_BASE = {32: 500000.0, 64: 1000000.0}  # rotary base by query-head count (Llama-3, Qwen2)
DPO_BETA = 0.1


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "traffic_dpo_step_llama3_8b_gqa32x8_d128.txt")


def source_hash() -> str:
    """sha256 over the library's sources (the build id embedded in the library)."""
    from paper_2602_24082_amd.build import source_digest
    return source_digest()


def traffic_from_profile(kernel: str):
    """HBM bytes per launch of `kernel` from the committed counter summary, or
    None when there is none or the sources changed since it was taken."""
    if not os.path.exists(TRAFFIC_PROFILE):
        return None
    rec, digest = {}, None
    for line in open(TRAFFIC_PROFILE):
        if line.startswith("source_sha256:"):
            digest = line.split(":", 1)[1].strip()
        elif line.startswith("kernel "):
            parts = line.split()
            kv = dict(x.split("=") for x in parts[2:])
            rec[parts[1]] = int(float(kv["hbm_bytes"]))
    if digest != source_hash():
        return None
    return rec.get(kernel)


def useful_pairs(pack: wl.Pack) -> int:
    """Visible (query, key) pairs: P(P+1)/2 + sum_k [L_k P + L_k(L_k+1)/2] per row."""
    n = 0
    for b in range(pack.num_rows):
        P = int(pack.prompt_len[b])
        n += P * (P + 1) // 2
        for k in range(int(pack.num_resp[b])):
            L = int(pack.resp_len[b, k])
            n += L * P + L * (L + 1) // 2
    return n


def logit_rows_needed(pack: wl.Pack) -> int:
    n = 0
    for b in range(pack.num_rows):
        lens = [int(pack.resp_len[b, k]) for k in range(int(pack.num_resp[b]))]
        if any(L > 0 for L in lens):
            n += 1 + sum(max(L - 1, 0) for L in lens)
    return n


class Attn:
    """Inputs, outputs and workspaces of one attention fwd+bwd on a pack; with
    store_ds the backward's workspace holds the stored dS (its other mode)."""

    def __init__(self, pack, hq, hkv, d, seed, dev, store_ds=False):
        self.pack = pack
        self.q, self.k, self.v, self.do = wl.qkv(pack, hq, hkv, d, seed, torch.bfloat16, dev)
        T = pack.total_tokens
        self.o = torch.empty_like(self.q)
        self.lse = torch.empty(hq, T, dtype=torch.float32, device=dev)
        self.dq = torch.empty_like(self.q)
        self.dk = torch.empty_like(self.k)
        self.dv = torch.empty_like(self.v)
        f, b, _, _ = pp.pp_workspace_size(pack, hq, hkv, d, fwd=True, bwd=True, loss=False)
        if store_ds:
            b = pp.pp_bwd_stored_ds_workspace_size(pack, hq, hkv, d)[0]
        self.ws_f = torch.empty(max(f, 1), dtype=torch.uint8, device=dev)
        self.ws_b = torch.empty(max(b, 1), dtype=torch.uint8, device=dev)

    def fwd(self):
        pp.pp_attn_fwd(self.pack, self.q, self.k, self.v, out=self.o, lse=self.lse, ws=self.ws_f)

    def bwd(self):
        pp.pp_attn_bwd(self.pack, self.q, self.k, self.v, self.o, self.lse, self.do, dq=self.dq,
                       dk=self.dk, dv=self.dv, ws=self.ws_b)

    def run(self):
        self.fwd()
        self.bwd()


def median_time(fn, iters=10, warmup=3, reps=5):
    """Median over `reps` repetitions of the mean time of `iters` back-to-back
    calls (HIP events on the stream): one repetition disturbed by a host stall
    that lets the GPU run dry does not move the result."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(iters):
            fn()
        e.record()
        torch.cuda.synchronize()
        times.append(s.elapsed_time(e) / iters)
    return float(np.median(times))


def time_attention(pack, hq, hkv, d, dev, iters=10, warmup=3, store_ds=False):
    a = Attn(pack, hq, hkv, d, 977, dev, store_ds=store_ds)
    ms = median_time(a.run, iters, warmup)
    del a
    torch.cuda.empty_cache()
    return ms


def comparator(pack, hq, hkv, d, dev):
    """Attention fwd+bwd of the packed batch against the same samples unpacked
    (prompt repeated per response: padded, and unpadded), and against a dense
    causal kernel over the packed rows; plus the predicted ratios of the cost
    model of Sec. 3.2.1 and the batch's KV bytes per layer."""
    padded = wl.unpacked_padded(pack)
    varlen = wl.unpacked_varlen(pack)
    dense = wl.packed_dense_causal(pack)
    t_packed = time_attention(pack, hq, hkv, d, dev)
    t_pad = time_attention(padded, hq, hkv, d, dev)
    t_var = time_attention(varlen, hq, hkv, d, dev)
    t_dense = time_attention(dense, hq, hkv, d, dev)
    comp = {"packed_ms": round(t_packed, 4), "unpacked_padded_ms": round(t_pad, 4),
            "unpacked_varlen_ms": round(t_var, 4), "packed_dense_causal_ms": round(t_dense, 4),
            "speedup_vs_padded": round(t_pad / t_packed, 3),
            "speedup_vs_varlen": round(t_var / t_packed, 3),
            "padded_layout": f"{padded.num_rows} sequences x {int(padded.row_lengths()[0])} tokens"}
    st = pp.pp_pack_stats(pack)
    kv = lambda tokens: int(tokens) * hkv * d * 2 * 2
    cost = {
        "eq1_cost_ratio": round(st["eq1_cost_ratio"], 4),
        "eq1_predicted_speedup": round(1.0 / st["eq1_cost_ratio"], 3),
        "rows_eq1_cheaper": f'{st["rows_eq1_cheaper"]}/{st["rows_with_responses"]}',
        "measured_dense_packed_over_varlen": round(t_dense / t_var, 3),
        "pairs_packed_over_unpacked": round(st["pairs_packed"] / st["pairs_unpacked"], 4),
        "pairs_dense_packed_over_unpacked": round(st["pairs_dense_packed"] / st["pairs_unpacked"], 4),
        "measured_packed_over_varlen": round(t_packed / t_var, 3),
        "eq1_memory_ratio": round(st["eq1_memory_ratio"], 4),
        "kv_bytes_per_layer": {"packed": kv(st["tokens_packed"]), "unpacked": kv(st["tokens_unpacked"]),
                               "padded": kv(st["tokens_padded"])},
        "kv_ratio_packed_over_unpacked": round(st["tokens_packed"] / st["tokens_unpacked"], 4),
    }
    return comp, cost


def cpu_baseline(pack, cfg, rows, seed):
    """The oracle (fp64 numpy) on a bounded sample of the same workload: the
    attention forward and backward of the given rows, all heads."""
    from oracle import pp_oracle as orc
    from threadpoolctl import threadpool_info
    flops = 0
    secs = 0.0
    for b in rows:
        one = wl.make_pack([int(pack.prompt_len[b])], [pack.resp_len[b, :int(pack.num_resp[b])].tolist()])
        q, k, v, do = wl.qkv(one, cfg.hq, cfg.hkv, cfg.head_dim, seed + b, torch.bfloat16, "cpu")
        qn, kn, vn, don = (x.double().numpy() for x in (q, k, v, do))
        args = one.oracle_args()
        t0 = time.perf_counter()
        orc.attn_fwd(*args, qn, kn, vn)
        orc.attn_bwd(*args, qn, kn, vn, don)
        secs += time.perf_counter() - t0
        flops += 14 * cfg.head_dim * cfg.hq * useful_pairs(one)
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = max([i.get("num_threads", 1) for i in blas] + [1])
    return {"value": flops / secs / 1e12, "unit": "useful TFLOP/s (attention fwd+bwd)",
            "cores": int(threads), "kind": "oracle",
            "cpu_model": cpu_model(), "usable_cores": len(os.sched_getaffinity(0)),
            "blas_threads": int(threads),
            "blas": ",".join(sorted({f'{i.get("internal_api", "?")} {i.get("version", "")}'.strip() for i in blas})),
            "sample": (f"rows {list(rows)} of the benchmarked batch (T={[int(pack.row_lengths()[b]) for b in rows]}), "
                       f"all {cfg.hq} heads, attention fwd+bwd in fp64 numpy, {secs:.1f} s; 'cores' = the BLAS "
                       f"threads the oracle's matrix products ran on (its elementwise work is single-threaded)")}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def attention_memory(pack, hq, hkv, d, dev, store_ds=False):
    """Device memory of one attention fwd+bwd on a layout: the allocator's
    high-water mark above what was allocated before, with q, k, v, dO, the
    outputs O and LSE, the gradients and both workspaces live (the library
    allocates nothing itself: every byte is a caller tensor).  Returns
    (peak bytes, of which activations q, k, v, O, LSE)."""
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    base = torch.cuda.memory_allocated(dev)
    torch.cuda.reset_peak_memory_stats(dev)
    a = Attn(pack, hq, hkv, d, 977, dev, store_ds=store_ds)
    a.run()
    torch.cuda.synchronize()
    peak = torch.cuda.max_memory_allocated(dev) - base
    act = sum(t.numel() * t.element_size() for t in (a.q, a.k, a.v, a.o, a.lse))
    del a
    torch.cuda.empty_cache()
    return int(peak), int(act)


def memory_leg(pack, hq, hkv, d, dev):
    """Measured attention memory of the packed layout against the unpacked
    layouts (Sec. 3.2.1: with linear-memory attention, memory follows tokens),
    next to the ratios the cost model predicts."""
    st = pp.pp_pack_stats(pack)
    out = {}
    for name, lay in (("packed", pack), ("unpacked_varlen", wl.unpacked_varlen(pack)),
                      ("unpacked_padded", wl.unpacked_padded(pack))):
        peak, act = attention_memory(lay, hq, hkv, d, dev)
        out[name] = {"tokens": lay.total_tokens, "peak_bytes": peak, "activation_bytes": act}
    for name in ("unpacked_varlen", "unpacked_padded"):
        out[f"packed_over_{name}_peak"] = round(out["packed"]["peak_bytes"] / out[name]["peak_bytes"], 4)
        out[f"packed_over_{name}_activations"] = round(
            out["packed"]["activation_bytes"] / out[name]["activation_bytes"], 4)
    out["tokens_packed_over_unpacked"] = round(st["tokens_packed"] / st["tokens_unpacked"], 4)
    out["eq1_memory_ratio"] = round(st["eq1_memory_ratio"], 4)
    # the backward's other mode keeps dS (one bf16 per pair of each visible
    # 32 x 32 block, per head): memory then follows pairs, not tokens
    peak, _ = attention_memory(pack, hq, hkv, d, dev, store_ds=True)
    out["packed_stored_ds_peak_bytes"] = peak
    out["measured_by"] = ("torch.cuda.max_memory_allocated over one attention fwd+bwd (inputs, dO, O, LSE, "
                          "gradients, workspaces; the default backward, which recomputes S and dP in its dQ pass)")
    return out


def attention_kernels(pack, hq, hkv, d, dev, iters=5, store_ds=False):
    """Per-kernel average launch times of attention fwd+bwd on a pack (library
    events around every launch) and each kernel's fraction of the bf16 peak on
    its useful work."""
    a = Attn(pack, hq, hkv, d, 977, dev, store_ds=store_ds)
    for _ in range(2):
        a.run()
    torch.cuda.synchronize()
    pp.pp_timing_select(None)
    pp.pp_timing_reset()
    pp.pp_timing_enable(True)
    for _ in range(iters):
        a.run()
    torch.cuda.synchronize()
    pp.pp_timing_enable(False)
    kt = pp.pp_timing_get()
    del a
    torch.cuda.empty_cache()
    U = useful_pairs(pack)
    per = {"pp_attn_fwd": 4, "pp_attn_bwd_dkdv": 8, "pp_attn_bwd_dq": 2}
    out = {}
    for k, units in per.items():
        if k in kt:
            ms = kt[k][0] / kt[k][1]
            ach = units * d * hq * U / (ms * 1e-3) / 1e12
            out[k] = {"avg_ms": round(ms, 4), "useful_TFLOP_s": round(ach, 1), "frac": round(ach / PEAK_BF16_TFLOPS, 4)}
    if "pp_attn_bwd_prep" in kt:
        out["pp_attn_bwd_prep"] = {"avg_ms": round(kt["pp_attn_bwd_prep"][0] / kt["pp_attn_bwd_prep"][1], 4)}
    bwd_k = ("pp_attn_bwd_prep", "pp_attn_bwd_dkdv", "pp_attn_bwd_dq")
    bwd_ms = sum(kt[k][0] / kt[k][1] for k in bwd_k if k in kt)
    if bwd_ms > 0:
        ach = 10 * d * hq * U / (bwd_ms * 1e-3) / 1e12
        out["backward_10_units"] = {"ms": round(bwd_ms, 4), "useful_TFLOP_s": round(ach, 1),
                                    "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                                    "rule": "over the backward's kernels (delta pre-pass when present, dK/dV, dQ)"}
    return out


def stored_ds_leg(pack, hq, hkv, d, dev, with_kernels=True):
    """The backward's other mode: dK/dV stores dS and the dQ pass reads it back
    instead of recomputing S and dP.  Attention fwd+bwd time against the
    default mode (timed alternately), the dS bytes and the kernels."""
    U = useful_pairs(pack)
    lean = pp.pp_workspace_size(pack, hq, hkv, d, fwd=False, bwd=True, loss=False)[1]
    full = pp.pp_bwd_stored_ds_workspace_size(pack, hq, hkv, d)[0]
    t_s, t_r = [], []
    for _ in range(2):
        t_r.append(time_attention(pack, hq, hkv, d, dev, iters=5, warmup=2))
        t_s.append(time_attention(pack, hq, hkv, d, dev, iters=5, warmup=2, store_ds=True))
    ts, tr = min(t_s), min(t_r)
    out = {"attn_fwd_bwd_ms": round(ts, 4), "useful_TFLOP_s": round(14 * d * hq * U / (ts * 1e-3) / 1e12, 1),
           "recompute_mode_ms": round(tr, 4), "speedup_over_recompute_mode": round(tr / ts, 4),
           "ds_bytes": int(full - lean), "bwd_workspace_bytes": int(full),
           "rule": "best of two alternating runs of each mode"}
    if with_kernels:
        out["kernels"] = attention_kernels(pack, hq, hkv, d, dev, store_ds=True)
    return out


def workload_leg(cfg, dev):
    """Attention fwd+bwd of another workload: useful TFLOP/s of the whole pass
    (HIP events around it, no per-launch events inside) and per kernel, and the
    speedup over the same kernels on the unpacked padded layout."""
    pack = wl.config_pack(cfg)
    hq, hkv, d = cfg.hq, cfg.hkv, cfg.head_dim
    U = useful_pairs(pack)
    t = time_attention(pack, hq, hkv, d, dev, iters=5, warmup=2)
    t_pad = time_attention(wl.unpacked_padded(pack), hq, hkv, d, dev, iters=3, warmup=1)
    tf = 14 * d * hq * U / (t * 1e-3) / 1e12
    return {"workload": cfg.name, "rows": pack.num_rows, "tokens": pack.total_tokens, "useful_pairs": U,
            "attn_fwd_bwd_ms": round(t, 4), "useful_TFLOP_s": round(tf, 1),
            "pct_bf16_peak": round(100 * tf / PEAK_BF16_TFLOPS, 2),
            "unpacked_padded_ms": round(t_pad, 4), "speedup_vs_padded": round(t_pad / t, 3),
            "kernels": attention_kernels(pack, hq, hkv, d, dev),
            "stored_ds": stored_ds_leg(pack, hq, hkv, d, dev, with_kernels=False)}


def chain_sorting(dev, reps=1):
    """The full DPO kernel chain (attention fwd+bwd, policy and reference
    log-probs, loss) of the 72B-shaped workload: a pool of 128 samples cut into 8
    batches of 16 rows, in draw order ("unsorted") or by packed length
    ("sorted"), on the packed layout and on the unpacked layout (every
    (prompt, response) pair its own sequence: attention padded to the batch's
    longest pair, log-probs over the unpadded pairs).  Reports the single-GPU
    total over the 8 batches and a simulated 8-rank data-parallel step (each
    virtual rank runs 2 rows; a step costs its slowest rank)."""
    cfg = wl.DPO_CHAIN
    P, L, unsorted, sorted_b = wl.dpo_chain_pool(cfg)
    V = cfg.vocab
    max_tokens = 0
    layouts = {}
    for name, batches in (("unsorted", unsorted), ("sorted", sorted_b)):
        for bi, rows in enumerate(batches):
            pk = wl.make_pack([P[i] for i in rows], [L[i] for i in rows])
            lp_pack = wl.make_pack([P[i] for i in rows for _ in L[i]], [[l] for i in rows for l in L[i]])
            layouts[(name, bi)] = (pk, wl.unpacked_padded(pk), lp_pack, rows)
            max_tokens = max(max_tokens, pk.total_tokens, lp_pack.total_tokens)
    logits = [wl.randn_rows(max_tokens, V, 7 + m, torch.bfloat16, dev, cfg.logit_sigma) for m in range(2)]
    tokens = wl.randint((max_tokens,), V, 9, dev)

    def chain_ms(att_pack, lp_pack):
        a = Attn(att_pack, cfg.hq, cfg.hkv, cfg.head_dim, 977, dev)
        T = lp_pack.total_tokens
        seqs = [torch.empty(lp_pack.num_rows, lp_pack.max_resp, dtype=torch.float32, device=dev) for _ in range(2)]
        ws = torch.empty(pp.pp_workspace_size(lp_pack, vocab=V, fwd=False, bwd=False, logprob=True, loss=False)[2],
                         dtype=torch.uint8, device=dev)
        if lp_pack.max_resp >= 2:
            num, pol, ref = lp_pack.num_resp.tolist(), seqs[0], seqs[1]
        else:  # one response per row: regroup the K responses of each sample for the loss
            num = None

        def run():
            a.run()
            for m in range(2):
                pp.pp_seq_logprob(lp_pack, logits[m][:T], tokens[:T], seq=seqs[m], ws=ws)
            if num is not None:
                pp.pp_dpo_loss(num, pol, ref, cfg.beta)
            else:
                k = 2
                pp.pp_dpo_loss([k] * (lp_pack.num_rows // k), seqs[0].view(-1, k), seqs[1].view(-1, k), cfg.beta)
        run()
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(reps):
            run()
        e.record()
        torch.cuda.synchronize()
        del a
        return s.elapsed_time(e) / reps

    cells = {}
    for name in ("unsorted", "sorted"):
        for lay in ("packed", "unpacked_padded"):
            total = 0.0
            dp = 0.0
            for bi in range(8):
                pk, padded, lp_pack, rows = layouts[(name, bi)]
                if lay == "packed":
                    total += chain_ms(pk, pk)
                else:
                    total += chain_ms(padded, lp_pack)
                ranks = []
                for r in range(8):
                    sub = rows[2 * r:2 * r + 2]
                    spk = wl.make_pack([P[i] for i in sub], [L[i] for i in sub])
                    if lay == "packed":
                        ranks.append(chain_ms(spk, spk))
                    else:
                        slp = wl.make_pack([P[i] for i in sub for _ in L[i]], [[l] for i in sub for l in L[i]])
                        ranks.append(chain_ms(wl.unpacked_padded(spk), slp))
                dp += max(ranks)
            cells[f"{lay}_{name}"] = {"one_gpu_ms": round(total, 3), "simulated_dp8_ms": round(dp, 3),
                                      "one_gpu_samples_per_s": round(128 / (total * 1e-3), 1),
                                      "simulated_dp8_samples_per_s": round(128 / (dp * 1e-3), 1)}
    base = cells["unpacked_padded_unsorted"]
    for c in cells.values():
        c["one_gpu_speedup"] = round(base["one_gpu_ms"] / c["one_gpu_ms"], 3)
        c["simulated_dp8_speedup"] = round(base["simulated_dp8_ms"] / c["simulated_dp8_ms"], 3)
    del logits, tokens
    torch.cuda.empty_cache()
    return {"metric": "DPO kernel chain with batch sorting (72B-shaped, 128 samples, 8 batches of 16)",
            "unit": "ms", "workload": cfg.name, "vocab": V, "beta": cfg.beta, "cells": cells}


def plan_leg(pack, cfg, seed, dev, layers=8):
    """The reusable plan: the pack planned and staged once (pp_plan_create), then
    attention fwd+bwd on it for several layers in a row (different q, k, v
    would not change the work), against the same layers through the
    self-contained pp_attn_fwd / pp_attn_bwd, which plan and copy metadata in
    every call.  Reports per-layer times and the plan's own cost (host
    planning time, GPU time of its one metadata copy)."""
    hq, hkv, d = cfg.hq, cfg.hkv, cfg.head_dim
    a = Attn(pack, hq, hkv, d, seed, dev)
    ws_p = torch.empty(pp.pp_plan_workspace_size(pack, hq, hkv, d), dtype=torch.uint8, device=dev)
    plan = pp.pp_plan_create(pack, hq, hkv, d, ws=ws_p, device=dev)

    def planned():
        for _ in range(layers):
            pp.pp_attn_fwd_planned(plan, a.q, a.k, a.v, out=a.o, lse=a.lse)
            pp.pp_attn_bwd_planned(plan, a.q, a.k, a.v, a.o, a.lse, a.do, dq=a.dq, dk=a.dk, dv=a.dv)

    def self_contained():
        for _ in range(layers):
            a.run()

    t_plan = median_time(planned, iters=3, warmup=2) / layers
    t_self = median_time(self_contained, iters=3, warmup=2) / layers
    host = []
    for _ in range(10):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        p2 = pp.pp_plan_create(pack, hq, hkv, d, ws=ws_p, device=dev)
        host.append((time.perf_counter() - t0) * 1e3)
        pp.pp_plan_destroy(p2)
    gpu_copy = median_time(lambda: pp.pp_plan_destroy(pp.pp_plan_create(pack, hq, hkv, d, ws=ws_p, device=dev)),
                           iters=5, warmup=2)
    pp.pp_plan_destroy(plan)
    useful = 14 * d * hq * useful_pairs(pack)
    return {"layers": layers, "planned_ms_per_layer": round(t_plan, 4),
            "self_contained_ms_per_layer": round(t_self, 4),
            "planned_useful_TFLOP_s": round(useful / (t_plan * 1e-3) / 1e12, 1),
            "plan_create_host_ms": round(float(np.median(host)), 4),
            "plan_create_stream_ms": round(gpu_copy, 4),
            "note": "value stays on pp_attn_fwd/pp_attn_bwd (plan + copy inside every call); this leg reuses "
                    "one staged plan across layers, as a model would"}


def rope_leg(pack, cfg, seed, dev, base, iters=10):
    """Attention fwd+bwd with rotary embeddings on the packed position IDs: the
    fused entry points (queries rotated in the forward's prologue, dq and dk
    rotated back in the backward's epilogues, keys rotated once) against the
    same work done as separate passes (pp_rope on q and k, plain attention,
    pp_rope inverse on dq and dk), and plain attention without rotation."""
    hq, hkv, d = cfg.hq, cfg.hkv, cfg.head_dim
    a = Attn(pack, hq, hkv, d, seed, dev)
    q_rot, k_rot = torch.empty_like(a.q), torch.empty_like(a.k)
    ws_r = torch.empty(pp.pp_rope_workspace_size(pack, d), dtype=torch.uint8, device=dev)

    def fused():
        pp.pp_attn_fwd_rope(pack, a.q, a.k, a.v, base, out=a.o, lse=a.lse, q_rot=q_rot, k_rot=k_rot, ws=a.ws_f)
        pp.pp_attn_bwd_rope(pack, q_rot, k_rot, a.v, a.o, a.lse, a.do, base, dq=a.dq, dk=a.dk, dv=a.dv, ws=a.ws_b)

    def separate():
        pp.pp_rope(pack, a.q, base, out=q_rot, ws=ws_r)
        pp.pp_rope(pack, a.k, base, out=k_rot, ws=ws_r)
        pp.pp_attn_fwd(pack, q_rot, k_rot, a.v, out=a.o, lse=a.lse, ws=a.ws_f)
        pp.pp_attn_bwd(pack, q_rot, k_rot, a.v, a.o, a.lse, a.do, dq=a.dq, dk=a.dk, dv=a.dv, ws=a.ws_b)
        pp.pp_rope(pack, a.dq, base, inverse=True, out=a.dq, ws=ws_r)
        pp.pp_rope(pack, a.dk, base, inverse=True, out=a.dk, ws=ws_r)

    def timed(fn):
        return median_time(fn, iters)

    t_plain = timed(a.run)
    t_fused = timed(fused)
    t_sep = timed(separate)
    # the standalone rotation of q alone: bytes = read + write of q (bf16)
    pp.pp_timing_reset()
    pp.pp_timing_enable(True)
    for _ in range(iters):
        pp.pp_rope(pack, a.q, base, out=q_rot, ws=ws_r)
    torch.cuda.synchronize()
    pp.pp_timing_enable(False)
    kr = pp.pp_timing_get()["pp_rope"]
    q_bytes = pack.total_tokens * hq * d * 2 * 2
    gbs = q_bytes / (kr[0] / kr[1] * 1e-3) / 1e9
    out = {"rope_base": base, "fused_fwd_bwd_ms": round(t_fused, 4), "separate_passes_ms": round(t_sep, 4),
           "plain_attention_ms": round(t_plain, 4), "fused_over_plain": round(t_fused / t_plain, 3),
           "separate_over_fused": round(t_sep / t_fused, 3),
           "pp_rope_q": {"avg_ms": round(kr[0] / kr[1], 4), "GB_per_s": round(gbs, 1),
                         "frac_hbm": round(gbs / PEAK_HBM_GBS, 4), "algorithmic_bytes": q_bytes}}
    del a
    torch.cuda.empty_cache()
    return out


def calib_copy(dev):
    """A plain device copy of 1 GiB, five times: read 1 GiB + write 1 GiB each."""
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calib_copy_bytes": n, "launches": 5}))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--prewarm-s", type=float, default=2.0,
                    help="untimed steps for this many seconds before the warm-up steps: the first GPU "
                         "process on a fresh machine otherwise times some steps before the clocks settle")
    ap.add_argument("--config", default=wl.LLAMA3_8B.name, choices=sorted(wl.BY_NAME),
                    help="the workload of the timed steps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-comparator", action="store_true")
    ap.add_argument("--calib-copy", action="store_true")
    ap.add_argument("--chain-sorting", action="store_true", help="print only the DPO chain leg")
    ap.add_argument("--attn-loop", type=int, default=0,
                    help="profiling mode: run only N attention fwd+bwd passes on --config's batch "
                         "(default backward mode; --store-ds for the other) and print their mean time")
    ap.add_argument("--store-ds", action="store_true", help="with --attn-loop: the stored-dS backward")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the other workloads, the measured memory and the DPO chain")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the packed rows shard by "
              "data parallelism with no exchange, so multi-GPU throughput is N x this line)", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    if args.calib_copy:
        calib_copy(dev)
        return
    if args.chain_sorting:
        print(json.dumps(chain_sorting(dev)))
        return
    cfg = wl.BY_NAME[args.config]
    if args.attn_loop:
        pack = wl.config_pack(cfg)
        ms = time_attention(pack, cfg.hq, cfg.hkv, cfg.head_dim, dev, iters=args.attn_loop, warmup=2,
                            store_ds=args.store_ds)
        print(json.dumps({"workload": cfg.name, "store_ds": args.store_ds, "attn_fwd_bwd_ms": round(ms, 4)}))
        return

    pack = wl.config_pack(cfg)
    T = pack.total_tokens
    seed = wl.tensor_seed(cfg.index, 0)
    attn = Attn(pack, cfg.hq, cfg.hkv, cfg.head_dim, seed, dev)
    V = cfg.vocab or LOGPROB_VOCAB
    sigma = cfg.logit_sigma if cfg.vocab else LOGPROB_SIGMA
    logits_pol = wl.randn_rows(T, V, seed + wl.STREAM_LOGITS_POL, torch.bfloat16, dev, sigma)
    logits_ref = wl.randn_rows(T, V, seed + wl.STREAM_LOGITS_REF, torch.bfloat16, dev, sigma)
    tokens = wl.randint((T,), V, seed + wl.STREAM_TOKENS, dev)
    Kmax = pack.max_resp
    seq_pol = torch.empty(pack.num_rows, Kmax, dtype=torch.float32, device=dev)
    seq_ref = torch.empty_like(seq_pol)
    lp_ws_n = pp.pp_workspace_size(pack, vocab=V, fwd=False, bwd=False, logprob=True, loss=True)
    ws_lp = torch.empty(lp_ws_n[2], dtype=torch.uint8, device=dev)
    ws_loss = torch.empty(max(lp_ws_n[3], 256), dtype=torch.uint8, device=dev)
    num_resp = pack.num_resp.tolist()
    beta = cfg.beta if cfg.vocab else DPO_BETA
    with_ref = cfg.with_ref if cfg.vocab else True

    attn_ev = []

    def step(record):
        if record:
            a0, am, a1 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            a0.record()
        attn.fwd()
        if record:
            am.record()
        attn.bwd()
        if record:
            a1.record()
            attn_ev.append((a0, am, a1))
        pp.pp_seq_logprob(pack, logits_pol, tokens, seq=seq_pol, ws=ws_lp)
        if with_ref:
            pp.pp_seq_logprob(pack, logits_ref, tokens, seq=seq_ref, ws=ws_lp)
        return pp.pp_dpo_loss(num_resp, seq_pol, seq_ref if with_ref else None, beta, ws=ws_loss)

    U = useful_pairs(pack)
    d, hq = cfg.head_dim, cfg.hq
    fwd_flops = 4 * d * hq * U
    bwd_flops = 10 * d * hq * U
    useful = fwd_flops + bwd_flops
    # algorithmic work per launch of each kernel (FLOPs of the GEMMs its algorithm
    # performs, or bytes it must move)
    n_rows = logit_rows_needed(pack)
    # dQ's useful work is its own product, dQ = scale dS K (2 d Hq per pair);
    # the S and dP it recomputes (4 d Hq per pair) are counted by dK/dV
    per_launch = {
        "pp_attn_fwd": ("mfma", 4 * d * hq * U),
        "pp_attn_bwd_dkdv": ("mfma", 8 * d * hq * U),
        "pp_attn_bwd_dq": ("mfma", 2 * d * hq * U),
        "pp_logprob_rows": ("hbm", n_rows * V * 2 + n_rows * 16),
    }

    t_pre = time.perf_counter()
    n_pre = 0
    while time.perf_counter() - t_pre < args.prewarm_s:
        step(False)
        n_pre += 1
        if n_pre % 50 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        step(False)
    # per-kernel breakdown: a short pass with every launch between hipEvents picks
    # the kernel with the largest time per step; the timed steps then carry events
    # on that kernel alone, so the rest of each step runs as it does untimed
    torch.cuda.synchronize()
    n_breakdown = max(3, min(args.steps, 10))
    pp.pp_timing_select(None)
    pp.pp_timing_reset()
    pp.pp_timing_enable(True)
    for _ in range(n_breakdown):
        step(False)
    torch.cuda.synchronize()
    pp.pp_timing_enable(False)
    kern_all = pp.pp_timing_get()
    dom = max((k for k in kern_all if k in per_launch), key=lambda k: kern_all[k][0])
    pp.pp_timing_select([dom])
    pp.pp_timing_reset()
    pp.pp_timing_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        loss, _, _ = step(True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    pp.pp_timing_enable(False)
    pp.pp_timing_select(None)
    kern = pp.pp_timing_get()  # the dominant kernel, over the timed steps
    ms_step = (t1 - t0) * 1e3 / args.steps
    attn_each = [a.elapsed_time(b) for a, _, b in attn_ev]
    bwd_each = [m.elapsed_time(b) for _, m, b in attn_ev]
    attn_ms = sum(attn_each) / args.steps
    loss_val = float(loss.item())
    tflops = useful / (attn_ms * 1e-3) / 1e12

    bound, work = per_launch[dom]
    avg_ms = kern[dom][0] / kern[dom][1]
    traffic = traffic_from_profile(dom) if cfg is wl.LLAMA3_8B else None
    if bound == "mfma":
        ach = work / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "kernel": dom, "achieved": round(ach, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4), "traffic": traffic,
                "algorithmic_flops_per_launch": work, "avg_launch_ms": round(avg_ms, 4)}
    else:
        ach = work / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "kernel": dom, "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": traffic,
                "algorithmic_bytes_per_launch": work, "avg_launch_ms": round(avg_ms, 4)}
    kernels = {k: {"avg_ms": round(v[0] / v[1], 4), "launches": v[1]} for k, v in kern_all.items()}
    # every attention kernel against the bf16 MFMA peak (algorithmic FLOPs per launch)
    attn_roofs = {}
    for k in ("pp_attn_fwd", "pp_attn_bwd_dkdv", "pp_attn_bwd_dq"):
        if k in kern_all:
            k_ms = kern_all[k][0] / kern_all[k][1]
            ach = per_launch[k][1] / (k_ms * 1e-3) / 1e12
            attn_roofs[k] = {"achieved_TFLOP_s": round(ach, 1), "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                             "avg_ms": round(k_ms, 4), "algorithmic_flops_per_launch": per_launch[k][1]}
    if "pp_attn_bwd_dq" in attn_roofs:
        # the recomputed S and dP, executed but not useful
        k_ms = attn_roofs["pp_attn_bwd_dq"]["avg_ms"]
        attn_roofs["pp_attn_bwd_dq"]["recompute_flops_per_launch"] = 4 * d * hq * U
        attn_roofs["pp_attn_bwd_dq"]["executed_TFLOP_s"] = round(6 * d * hq * U / (k_ms * 1e-3) / 1e12, 1)
    # the whole backward call (metadata copy, dQ with delta, dK/dV) from the
    # HIP events around it in the timed steps
    bwd_ms = float(np.median(bwd_each))
    ach = 10 * d * hq * U / (bwd_ms * 1e-3) / 1e12
    attn_roofs["backward_10_units"] = {"ms": round(bwd_ms, 4), "useful_TFLOP_s": round(ach, 1),
                                       "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                                       "rule": "10 d Hq FLOPs per visible pair over the whole pp_attn_bwd call "
                                               "(median over the timed steps)"}
    lp = kern.get("pp_logprob_rows") or kern_all.get("pp_logprob_rows")
    logprob = None
    if lp:
        lp_ms = lp[0] / lp[1]
        gbs = (n_rows * V * 2 + n_rows * 16) / (lp_ms * 1e-3) / 1e9
        logprob = {"kernel": "pp_logprob_rows", "GB_per_s": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
                   "rows": n_rows, "vocab": V, "avg_ms": round(lp_ms, 4),
                   "traffic": traffic_from_profile("pp_logprob_rows") if cfg is wl.LLAMA3_8B else None}

    # log-prob backward (the next link of the DPO chain): timed on its own, the
    # step above keeps to the forward hot path
    dlogits = torch.empty_like(logits_pol)
    _, _, dseq = pp.pp_dpo_loss(num_resp, seq_pol, seq_ref if with_ref else None, beta, ws=ws_loss)
    for _ in range(2):
        pp.pp_seq_logprob_bwd(pack, logits_pol, tokens, dseq, dlogits=dlogits, ws=ws_lp)
    torch.cuda.synchronize()
    pp.pp_timing_reset()
    pp.pp_timing_enable(True)
    for _ in range(max(3, args.steps // 2)):
        pp.pp_seq_logprob_bwd(pack, logits_pol, tokens, dseq, dlogits=dlogits, ws=ws_lp)
    torch.cuda.synchronize()
    pp.pp_timing_enable(False)
    kb = pp.pp_timing_get().get("pp_logprob_bwd")
    logprob_bwd = None
    if kb:
        kb_ms = kb[0] / kb[1]
        nbytes = n_rows * V * 2 + T * V * 2
        gbs = nbytes / (kb_ms * 1e-3) / 1e9
        logprob_bwd = {"kernel": "pp_logprob_bwd", "GB_per_s": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
                       "algorithmic_bytes": nbytes, "avg_ms": round(kb_ms, 4),
                       "bytes_rule": "needed logit rows read once + every dlogits row written once (bf16)",
                       "traffic": traffic_from_profile("pp_logprob_bwd") if cfg is wl.LLAMA3_8B else None}
    del dlogits
    # the gathered form: only the predicting rows are written
    n_g = pp.pp_logprob_row_count(pack)
    d_rows = torch.empty(n_g, V, dtype=logits_pol.dtype, device=dev)
    r_idx = torch.empty(n_g, dtype=torch.int32, device=dev)
    for _ in range(2):
        pp.pp_seq_logprob_bwd_rows(pack, logits_pol, tokens, dseq, dlogits_rows=d_rows, row_index=r_idx, ws=ws_lp)
    torch.cuda.synchronize()
    pp.pp_timing_reset()
    pp.pp_timing_enable(True)
    for _ in range(max(3, args.steps // 2)):
        pp.pp_seq_logprob_bwd_rows(pack, logits_pol, tokens, dseq, dlogits_rows=d_rows, row_index=r_idx, ws=ws_lp)
    torch.cuda.synchronize()
    pp.pp_timing_enable(False)
    kg = pp.pp_timing_get().get("pp_logprob_bwd_rows")
    if kg and logprob_bwd is not None:
        kg_ms = kg[0] / kg[1]
        nbytes = 2 * n_g * V * 2 + n_g * 4
        gbs = nbytes / (kg_ms * 1e-3) / 1e9
        logprob_bwd["gathered_rows"] = {"kernel": "pp_logprob_bwd_rows", "rows": n_g, "GB_per_s": round(gbs, 1),
                                        "frac_hbm": round(gbs / PEAK_HBM_GBS, 4), "algorithmic_bytes": nbytes,
                                        "avg_ms": round(kg_ms, 4),
                                        "bytes_rule": "each predicting row read once and written once (bf16)"}
    del d_rows, r_idx

    # reward-model head (scores on each response's last hidden state, then its
    # backward) on the same pack, hidden size of the named model
    hid = HIDDEN_DIM.get(cfg.hq, 4096)
    hidden = wl.randn((T, hid), seed + 11, torch.bfloat16, dev)
    w_head = wl.randn((hid,), seed + 12, torch.bfloat16, dev, sigma=0.02)
    ws_rm = torch.empty(max(pp.pp_rm_workspace_size(pack), 1), dtype=torch.uint8, device=dev)
    dsc = torch.ones(pack.num_rows, Kmax, device=dev)
    for _ in range(2):
        pp.pp_rm_scores(pack, hidden, w_head, 0.0, ws=ws_rm)
        pp.pp_rm_scores_bwd(pack, hidden, w_head, dsc, ws=ws_rm)
    torch.cuda.synchronize()
    pp.pp_timing_reset()
    pp.pp_timing_enable(True)
    for _ in range(5):
        pp.pp_rm_scores(pack, hidden, w_head, 0.0, ws=ws_rm)
        pp.pp_rm_scores_bwd(pack, hidden, w_head, dsc, ws=ws_rm)
    torch.cuda.synchronize()
    pp.pp_timing_enable(False)
    kr = pp.pp_timing_get()
    rm_head = {"hidden_dim": hid, **{k: round(v[0] / v[1], 4) for k, v in kr.items() if k.startswith("pp_rm")},
               "unit": "ms per launch",
               "dhidden_GB_per_s": round(T * hid * 2 / (kr["pp_rm_dhidden"][0] / kr["pp_rm_dhidden"][1] * 1e-3) / 1e9, 1)}
    del hidden

    rope = rope_leg(pack, cfg, seed, dev, ROPE_BASE.get(cfg.hq, 500000.0))
    plan = plan_leg(pack, cfg, seed, dev)

    comp = cost = losing = None
    if not args.no_comparator:
        comp, cost = comparator(pack, hq, cfg.hkv, d, dev)
        losing = comparator(wl.losing_regime_pack(), hq, cfg.hkv, d, dev)
        losing = {"workload": "8 rows, prompt 32-96, K=2 responses 768-1024 (responses >> prompt)",
                  **losing[0], **losing[1]}

    memory = workloads = chain = stored = None
    if not args.no_extra:
        # free the step's large buffers first: the other legs allocate their own
        del logits_pol, logits_ref, attn
        torch.cuda.empty_cache()
        memory = memory_leg(pack, hq, cfg.hkv, d, dev)
        stored = stored_ds_leg(pack, hq, cfg.hkv, d, dev)
        workloads = {c.name: workload_leg(c, dev) for c in (wl.RM_K4, wl.LONG_PREFIX, wl.DPO_CHAIN) if c is not cfg}
        chain = chain_sorting(dev)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(pack, cfg, list(range(pack.num_rows)), seed)

    out = {
        "metric": "packed attn fwd+bwd useful TFLOP/s (% bf16 peak); speedup vs unpacked padded",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "attn_ms_per_step": round(attn_ms, 4),
        "attn_ms_median_step": round(float(np.median(attn_each)), 4),
        "attn_ms_steps": [round(x, 4) for x in attn_each],
        "prewarm": {"seconds": args.prewarm_s, "steps": n_pre},
        "pct_bf16_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": cfg.name, "rows": pack.num_rows, "tokens": T, "hq": hq, "hkv": cfg.hkv,
                   "head_dim": d, "useful_pairs": U, "logprob_vocab": V, "beta": beta,
                   "parallelism": "none (1 GPU)"},
        "speedup_vs_padded": comp["speedup_vs_padded"] if comp else None,
        "comparator": comp,
        "cost_model": cost,
        "losing_regime": losing,
        "logprob": logprob,
        "logprob_bwd": logprob_bwd,
        "rm_head": rm_head,
        "rope": rope,
        "plan": plan,
        "memory": memory,
        "workloads": workloads,
        "dpo_chain_sorting": chain,
        "kernels": kernels,
        "kernel_breakdown_steps": n_breakdown,
        "attention_rooflines": attn_roofs,
        "stored_ds_backward": stored,
        "roofline": roof,
        "cpu_baseline": cpu,
        "loss": loss_val,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
