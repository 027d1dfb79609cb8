"""Seeded synthetic inputs for packed preference batches.

This module only draws lengths and random tensors and lays rows out on the flat
token axis; it holds none of the method's arithmetic (no mask, no softmax, no
log-prob, no loss), so that the library and the independent checker can both be
fed from it.

Layout of a batch of B packed rows (Sec. 3.2: the prompt once, then the K
responses one after another):

* rows are concatenated on one flat token axis; row b spans
  [row_start[b], row_start[b+1]) and has capacity T_b = row_start[b+1]-row_start[b];
* the prompt occupies the first P_b tokens of the row;
* response k occupies [resp_off[b,k], resp_off[b,k] + resp_len[b,k]) relative to
  the row start, with resp_off[b,0] = P_b and each response following the
  previous one directly;
* tokens after P_b + sum_k resp_len[b,k] are padding.

Responses are stored in the paper's ranking order: a larger index is preferred
(Sec. 3.1).

Workload shapes follow the synthetic configurations: a tiny fp32 check case, a
Llama-3-8B-shaped GQA layer (32/8 heads, d 128), a K=4 reward-model case with a
128256-entry vocabulary, a long-prefix Qwen2-72B-shaped case (64/8 heads) and a
72B-shaped DPO chain with log-normal lengths and vocabulary 152064.  The paper's
datasets (Orca DPO pairs, Capybara, RLAIF-V, Tulu3) are not available; these
draws stand in for them.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np
import torch

SEED_ROOT = (2602, 24082)


@dataclasses.dataclass
class Pack:
    """Host description of a packed batch (all int32 numpy arrays)."""

    row_start: np.ndarray   # [B+1]
    prompt_len: np.ndarray  # [B]
    num_resp: np.ndarray    # [B]
    resp_off: np.ndarray    # [B, Kmax]
    resp_len: np.ndarray    # [B, Kmax]

    @property
    def num_rows(self) -> int:
        return int(self.prompt_len.shape[0])

    @property
    def max_resp(self) -> int:
        return int(self.resp_off.shape[1])

    @property
    def total_tokens(self) -> int:
        return int(self.row_start[-1])

    def row_lengths(self) -> np.ndarray:
        return np.diff(self.row_start)

    def oracle_args(self):
        """(row_start, prompt_len, num_resp, resp_off, resp_len) as plain lists,
        the argument order the checker takes."""
        return (self.row_start.tolist(), self.prompt_len.tolist(), self.num_resp.tolist(),
                self.resp_off.tolist(), self.resp_len.tolist())


def make_pack(prompt_lens: Sequence[int], resp_lens: Sequence[Sequence[int]],
              pad: Optional[Sequence[int]] = None, max_resp: Optional[int] = None) -> Pack:
    """Lay out rows: prompt, then responses back to back, then `pad[b]` padding
    tokens."""
    B = len(prompt_lens)
    Kmax = max([len(r) for r in resp_lens] + [0]) if max_resp is None else max_resp
    row_start = np.zeros(B + 1, np.int32)
    prompt = np.asarray(prompt_lens, np.int32).reshape(B)
    num = np.zeros(B, np.int32)
    off = np.zeros((B, Kmax), np.int32)
    ln = np.zeros((B, Kmax), np.int32)
    for b in range(B):
        o = int(prompt[b])
        num[b] = len(resp_lens[b])
        for k, L in enumerate(resp_lens[b]):
            off[b, k] = o
            ln[b, k] = int(L)
            o += int(L)
        extra = 0 if pad is None else int(pad[b])
        row_start[b + 1] = row_start[b] + o + extra
    return Pack(row_start, prompt, num, off, ln)


# ----------------------------------------------------------------------------
# The five synthetic configurations
# ----------------------------------------------------------------------------


@dataclasses.dataclass
class Config:
    name: str
    index: int
    hq: int
    hkv: int
    head_dim: int
    rows: int
    dtype: str             # "fp32" or "bf16" (inputs)
    vocab: int = 0         # 0: no log-prob leg
    logit_sigma: float = 1.0
    beta: float = 0.1
    with_ref: bool = True
    capacity: int = 0      # largest allowed packed row


CONFIGS: List[Config] = [
    Config("tiny_fp32_mha4_d64", 0, 4, 4, 64, 4, "fp32", vocab=1000, logit_sigma=2.0, beta=0.1,
           with_ref=True, capacity=256),
    Config("llama3_8b_gqa32x8_d128_k2", 1, 32, 8, 128, 8, "bf16", vocab=0, capacity=4096),
    Config("rm_k4_gqa32x8_d128_v128256", 2, 32, 8, 128, 8, "bf16", vocab=128256, logit_sigma=3.0,
           beta=1.0, with_ref=False, capacity=4096),
    Config("long_prefix_qwen72b_gqa64x8_d128", 3, 64, 8, 128, 8, "bf16", vocab=0, capacity=8192),
    Config("dpo_chain_qwen72b_gqa64x8_d128_v152064", 4, 64, 8, 128, 16, "bf16", vocab=152064,
           logit_sigma=1.0, beta=0.1, with_ref=True, capacity=8192),
]
# the configurations by name (index is only their seed stream)
TINY_FP32, LLAMA3_8B, RM_K4, LONG_PREFIX, DPO_CHAIN = CONFIGS
BY_NAME = {c.name: c for c in CONFIGS}


def _rng(cfg_index: int, stream: int, extra: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([*SEED_ROOT, cfg_index, stream, extra]))


def _lognormal_int(rng, median, sigma, lo, hi, n):
    x = np.exp(np.log(median) + sigma * rng.standard_normal(n))
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


def draw_lengths(cfg: Config, rows: Optional[int] = None, batch: int = 0):
    """Prompt and response lengths of one batch of a configuration."""
    B = cfg.rows if rows is None else rows
    rng = _rng(cfg.index, 0, batch)
    if cfg.name == TINY_FP32.name:
        P = rng.integers(64, 128, size=B, endpoint=True)
        L = rng.integers(16, 64, size=(B, 2), endpoint=True)
    elif cfg.name == LLAMA3_8B.name:
        P = rng.integers(256, 1536, size=B, endpoint=True)
        L = rng.integers(64, 512, size=(B, 2), endpoint=True)
    elif cfg.name == RM_K4.name:
        P = rng.integers(512, 2048, size=B, endpoint=True)
        L = rng.integers(32, 384, size=(B, 4), endpoint=True)
    elif cfg.name == LONG_PREFIX.name:
        P = rng.integers(2048, 6144, size=B, endpoint=True)
        L = rng.integers(64, 256, size=(B, 2), endpoint=True)
    elif cfg.name == DPO_CHAIN.name:
        P = _lognormal_int(rng, 1024, 0.6, 1, 6144, B)
        L = _lognormal_int(rng, 192, 0.6, 1, 1024, B * 2).reshape(B, 2)
    else:
        raise ValueError(cfg.name)
    return P.tolist(), L.tolist()


def config_pack(cfg: Config, rows: Optional[int] = None, batch: int = 0) -> Pack:
    P, L = draw_lengths(cfg, rows, batch)
    return make_pack(P, L)


def dpo_chain_pool(cfg: Config, pool: int = 128, batch_rows: int = 16):
    """Pool of samples for the sorted-versus-unsorted comparison: returns the
    lengths of `pool` samples and the row order of the unsorted (draw order) and
    sorted (by packed length) batchings, each a list of index lists."""
    P, L = draw_lengths(cfg, rows=pool, batch=1000)
    total = [P[i] + sum(L[i]) for i in range(pool)]
    unsorted = [list(range(s, s + batch_rows)) for s in range(0, pool, batch_rows)]
    order = sorted(range(pool), key=lambda i: (-total[i], i))
    sorted_b = [order[s:s + batch_rows] for s in range(0, pool, batch_rows)]
    return P, L, unsorted, sorted_b


# ----------------------------------------------------------------------------
# Comparator layouts: the same samples without packing
# ----------------------------------------------------------------------------


def unpacked_padded(pack: Pack) -> Pack:
    """Every (prompt, response_k) pair as its own sequence, all padded to the
    longest one: B*K rows of S_pad = max(P_b + L_bk) tokens, each described as a
    prompt-only row (K = 0) of S_pad tokens, so the whole padded length is
    attended causally as a padded batch is."""
    seqs = []
    for b in range(pack.num_rows):
        for k in range(int(pack.num_resp[b])):
            seqs.append(int(pack.prompt_len[b]) + int(pack.resp_len[b, k]))
    S = max(seqs) if seqs else 0
    return make_pack([S] * len(seqs), [[] for _ in seqs], max_resp=0)


def unpacked_varlen(pack: Pack) -> Pack:
    """Every (prompt, response_k) pair as its own unpadded sequence."""
    seqs = []
    for b in range(pack.num_rows):
        for k in range(int(pack.num_resp[b])):
            seqs.append(int(pack.prompt_len[b]) + int(pack.resp_len[b, k]))
    return make_pack(seqs, [[] for _ in seqs], max_resp=0)


def packed_dense_causal(pack: Pack) -> Pack:
    """Cost comparator for a kernel that cannot skip the blocks hiding one
    response from another: each packed row's real tokens attended causally as one
    sequence (a prompt-only row of P_b + sum_k L_bk tokens).  Its outputs are not
    the packed semantics; only its work matters (the dense cost of Sec. 3.2.1)."""
    lens = [int(pack.prompt_len[b]) + int(pack.resp_len[b, :int(pack.num_resp[b])].sum())
            for b in range(pack.num_rows)]
    return make_pack(lens, [[] for _ in lens], max_resp=0)


def losing_regime_pack(rows: int = 8, seed: int = 231) -> Pack:
    """Responses much longer than the prompt (prompt uniform 32-96, K = 2
    responses uniform 768-1024): the regime where Eq. (1) predicts that packing
    costs more than the unpacked layout for dense attention."""
    rng = np.random.default_rng(np.random.SeedSequence([2602, 24082, seed]))
    P = [int(x) for x in rng.integers(32, 97, size=rows)]
    L = [[int(x) for x in rng.integers(768, 1025, size=2)] for _ in range(rows)]
    return make_pack(P, L)


# ----------------------------------------------------------------------------
# Random tensors
# ----------------------------------------------------------------------------


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def tensor_seed(cfg_index: int, stream: int, batch: int = 0) -> int:
    return int(_rng(cfg_index, 100 + stream, batch).integers(0, 2**62))


STREAM_Q, STREAM_K, STREAM_V, STREAM_DO, STREAM_LOGITS_POL, STREAM_LOGITS_REF, STREAM_TOKENS = range(7)


def randn(shape, seed: int, dtype=torch.bfloat16, device="cpu", sigma: float = 1.0) -> torch.Tensor:
    """N(0, sigma) drawn in fp32 from a seeded torch generator, then cast
    (round to nearest even for bf16)."""
    g = _gen(device, seed)
    x = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    if sigma != 1.0:
        x.mul_(sigma)
    return x.to(dtype)


def randn_rows(rows: int, cols: int, seed: int, dtype, device, sigma: float,
               chunk_rows: int = 2048) -> torch.Tensor:
    """Large [rows, cols] N(0, sigma) matrix drawn in chunks so the fp32
    staging never exceeds chunk_rows*cols floats."""
    out = torch.empty(rows, cols, dtype=dtype, device=device)
    g = _gen(device, seed)
    for r in range(0, rows, chunk_rows):
        n = min(chunk_rows, rows - r)
        x = torch.randn(n, cols, generator=g, device=device, dtype=torch.float32)
        if sigma != 1.0:
            x.mul_(sigma)
        out[r:r + n].copy_(x)
    return out


def randint(shape, high: int, seed: int, device="cpu") -> torch.Tensor:
    g = _gen(device, seed)
    return torch.randint(0, high, shape, generator=g, device=device, dtype=torch.int32)


def qkv(pack: Pack, hq: int, hkv: int, d: int, seed_base: int, dtype, device="cpu", with_do=True):
    """Q, K, V (and dO) ~ N(0, 1) on the flat token axis."""
    T = pack.total_tokens
    q = randn((T, hq, d), seed_base + STREAM_Q, dtype, device)
    k = randn((T, hkv, d), seed_base + STREAM_K, dtype, device)
    v = randn((T, hkv, d), seed_base + STREAM_V, dtype, device)
    do = randn((T, hq, d), seed_base + STREAM_DO, dtype, device) if with_do else None
    return q, k, v, do
