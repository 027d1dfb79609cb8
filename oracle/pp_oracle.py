"""Plain fp64 CPU oracle for preference-packed attention and the DPO / Bradley-Terry
reductions.

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously-correct definition
that the HIP path is checked against.  Only the test suite, the smoke check and
the benchmark's CPU-baseline leg may import it; the library never does, and it
shares no code with the library (no kernels, headers, helpers or tables).

Everything here is written from the paper's statement of the method:

* Preference data point: one prompt x and K ranked responses y^1..y^K, with
  y^a preferred over y^b whenever a > b (Sec. 3.1, "Symbols").
* Preference packing: the prompt is written once, followed by the K responses
  one after another, d = (x, y^1, ..., y^K) (Sec. 3.2).
* The packing attention mask is causal; every response attends to the whole
  prompt and to its own earlier tokens and never to another response; position
  IDs keep each token's original (unpacked) position (Sec. 3.2 and the caption
  of Figure 1).  Packing must give exactly the results of the unpacked layout
  (Sec. 3.2).
* Reward-model Bradley-Terry loss over (preferred, dispreferred) pairs and the
  DPO implicit reward (Sec. 2.1), extended to K > 2 ranked responses (Sec. 2.1,
  last paragraph).
* Attention cost model and efficiency condition, Eq. (1) (Sec. 3.2.1).

Readings taken where the paper is silent or garbled (each is also listed in the
design notes):

R1  Mask: the figure is missing; the mask follows the prose.  Query i may see
    key j iff j <= i, neither is padding, and key j is a prompt token or lies in
    the same response as query i.
R2  Position IDs: prompt token t keeps t; token j of a response gets P + j
    (the position it has in its own unpacked sequence); padding gets 0.
R3  The DPO reward printed in Sec. 2.1 lacks the logarithm; we use
    r = beta * (log pi_theta(y|x) - log pi_ref(y|x)), the cited DPO form.
R4  The loss in Sec. 2.1 is printed without its minus sign; we minimise
    -log sigmoid(r_w - r_l) = softplus(-(r_w - r_l)).
R5  Preference order follows Sec. 3.1: the response with the larger index is
    preferred.
R6  K > 2: all K(K-1)/2 ranked pairs, mean over the pairs of a row, then mean
    over the rows that have at least two responses.
R7  A response's score log pi(y|x) is the SUM of its token log-probabilities.
R8  The first token of every response is predicted from the last prompt
    position P-1 (the position that predicts it in the unpacked layout), so a
    row with a non-empty response needs P >= 1.
R9  Softmax scale 1/sqrt(d) unless given; q-head h uses kv-head floor(h/G).
R10 Padding tokens: attention output, LSE and all gradients are 0; an empty
    response scores 0; rows with fewer than two responses are left out of the
    loss mean.
R16 Log-prob backward: the gradient reaching the logits is that of
    sum_{b,k} g_bk * seq_bk for given g = dL/dseq (the loss gradient); logit rows
    that predict no response token get 0, and a label outside the vocabulary
    makes its whole predicting row NaN (the forward makes the sum NaN).
R17 Reward model: Sec. 2.1 only says the model maps a token sequence to a
    scalar; we read it as a linear head on the hidden state of the sequence's
    last token.  In the packed row the unpacked sequence (prompt, response k)
    ends at o_k + L_k - 1, or at P - 1 when the response is empty (the prompt's
    hidden states are those of the unpacked prompt, since a prompt token sees
    only the prompt); a sequence with no token scores 0.
R19 Rotary position embedding: the paper states only that packed tokens keep
    their original position IDs (Sec. 3.2); the models it trains (Llama, Qwen)
    encode those IDs with rotary embeddings.  We use the half-split form of
    those models: for j < d/2, frequency w_j = base^(-2j/d), and the pair
    (x_j, x_{j+d/2}) of a token at position p is rotated by the angle p * w_j
    (counter-clockwise: x_j cos - x_{j+d/2} sin, x_{j+d/2} cos + x_j sin),
    applied to queries and keys before the attention scores.

All floating-point work is numpy float64.  Parity of every function here is
pinned by tests against closed forms, brute force on tiny inputs, finite
differences, library routines for special cases and values the paper prints.
"""
from __future__ import annotations

import math

import numpy as np

# ----------------------------------------------------------------------------
# Pack layout: segment IDs, position IDs, mask, tile classes (Sec. 3.2)
# ----------------------------------------------------------------------------


def row_segment_ids(T: int, P: int, offs, lens) -> np.ndarray:
    """Segment of every token of one packed row (Sec. 3.2, reading R1).

    0 = prompt, k = response k (1-based, in the stored order), -1 = padding.
    """
    seg = np.full(T, -1, dtype=np.int64)
    seg[:P] = 0
    for k, (o, L) in enumerate(zip(offs, lens)):
        seg[o:o + L] = k + 1
    return seg


def row_position_ids(T: int, P: int, offs, lens) -> np.ndarray:
    """Position IDs that keep each token's unpacked position (Sec. 3.2, R2)."""
    pos = np.zeros(T, dtype=np.int64)
    pos[:P] = np.arange(P)
    for o, L in zip(offs, lens):
        pos[o:o + L] = P + np.arange(L)
    return pos


def row_mask(T: int, P: int, offs, lens) -> np.ndarray:
    """Dense boolean [T, T] preference-packing mask of one row (Sec. 3.2, R1).

    M[i, j] is True iff query i may attend to key j: causal (j <= i), neither
    token is padding, and key j is a prompt token or shares query i's response.
    """
    seg = row_segment_ids(T, P, offs, lens)
    i = np.arange(T)[:, None]          # query index
    j = np.arange(T)[None, :]          # key index
    si = seg[:, None]
    sj = seg[None, :]
    M = (j <= i) & (si >= 0) & (sj >= 0) & ((sj == 0) | (sj == si))
    return M


def tile_classes(M: np.ndarray, bq: int, bk: int) -> np.ndarray:
    """Classify the (bq x bk) tiles of a row's mask: 0 EMPTY, 1 PARTIAL, 2 FULL.

    Tiles on the ragged edge are clipped to the row.  EMPTY = no visible pair,
    FULL = every pair of the (clipped) tile visible, PARTIAL otherwise.
    """
    T = M.shape[0]
    nq = -(-T // bq)
    nk = -(-T // bk)
    out = np.zeros((nq, nk), dtype=np.uint8)
    for a in range(nq):
        for b in range(nk):
            blk = M[a * bq:min(T, (a + 1) * bq), b * bk:min(T, (b + 1) * bk)]
            if not blk.any():
                out[a, b] = 0
            elif blk.all():
                out[a, b] = 2
            else:
                out[a, b] = 1
    return out


def _row_fields(row_start, prompt_len, num_resp, resp_off, resp_len, b):
    r0, r1 = int(row_start[b]), int(row_start[b + 1])
    K = int(num_resp[b])
    offs = [int(x) for x in resp_off[b][:K]]
    lens = [int(x) for x in resp_len[b][:K]]
    return r0, r1 - r0, int(prompt_len[b]), offs, lens


def pack_segment_ids(row_start, prompt_len, num_resp, resp_off, resp_len):
    """Segment IDs over the flat token axis, row by row."""
    out = []
    for b in range(len(prompt_len)):
        _, T, P, offs, lens = _row_fields(row_start, prompt_len, num_resp, resp_off, resp_len, b)
        out.append(row_segment_ids(T, P, offs, lens))
    return np.concatenate(out) if out else np.zeros(0, np.int64)


def pack_position_ids(row_start, prompt_len, num_resp, resp_off, resp_len):
    """Position IDs over the flat token axis, row by row."""
    out = []
    for b in range(len(prompt_len)):
        _, T, P, offs, lens = _row_fields(row_start, prompt_len, num_resp, resp_off, resp_len, b)
        out.append(row_position_ids(T, P, offs, lens))
    return np.concatenate(out) if out else np.zeros(0, np.int64)


def pack_tile_classes(row_start, prompt_len, num_resp, resp_off, resp_len, bq, bk):
    """Tile classes of every row, each row's [nq, nk] grid flattened row-major,
    rows concatenated."""
    out = []
    for b in range(len(prompt_len)):
        _, T, P, offs, lens = _row_fields(row_start, prompt_len, num_resp, resp_off, resp_len, b)
        if T == 0:
            continue
        out.append(tile_classes(row_mask(T, P, offs, lens), bq, bk).ravel())
    return np.concatenate(out) if out else np.zeros(0, np.uint8)


# ----------------------------------------------------------------------------
# Attention forward and backward with an explicit dense mask (Sec. 3.2)
# ----------------------------------------------------------------------------


def attn_fwd(row_start, prompt_len, num_resp, resp_off, resp_len, q, k, v, scale=None):
    """Masked softmax attention over every packed row.

    q: [sumT, Hq, d], k and v: [sumT, Hkv, d] (any float type; computed in fp64).
    Returns O [sumT, Hq, d] and LSE [Hq, sumT] (natural log), both float64.
    Query h reads kv-head h // (Hq / Hkv) (R9).  Rows with no visible key
    (padding) give O = 0 and LSE = 0 (R10).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    sumT, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    O = np.zeros((sumT, Hq, d))
    LSE = np.zeros((Hq, sumT))
    for b in range(len(prompt_len)):
        r0, T, P, offs, lens = _row_fields(row_start, prompt_len, num_resp, resp_off, resp_len, b)
        if T == 0:
            continue
        M = row_mask(T, P, offs, lens)
        has = M.any(axis=1)
        for h in range(Hq):
            g = h // G
            Qh = q[r0:r0 + T, h, :]
            Kg = k[r0:r0 + T, g, :]
            Vg = v[r0:r0 + T, g, :]
            S = scale * (Qh @ Kg.T)
            S = np.where(M, S, -np.inf)
            m = np.where(has, S.max(axis=1, initial=-np.inf), 0.0)
            E = np.where(M, np.exp(S - m[:, None]), 0.0)
            l = E.sum(axis=1)
            Pm = np.where(has[:, None], E / np.where(has, l, 1.0)[:, None], 0.0)
            O[r0:r0 + T, h, :] = Pm @ Vg
            LSE[h, r0:r0 + T] = np.where(has, m + np.log(np.where(has, l, 1.0)), 0.0)
    return O, LSE


def attn_probs(row_start, prompt_len, num_resp, resp_off, resp_len, q, k, b, h, scale=None):
    """The softmax matrix P of row b, query head h (for the row-sum fact)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    d = q.shape[2]
    G = q.shape[1] // k.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    r0, T, P, offs, lens = _row_fields(row_start, prompt_len, num_resp, resp_off, resp_len, b)
    M = row_mask(T, P, offs, lens)
    S = scale * (q[r0:r0 + T, h, :] @ k[r0:r0 + T, h // G, :].T)
    S = np.where(M, S, -np.inf)
    has = M.any(axis=1)
    m = np.where(has, S.max(axis=1, initial=-np.inf), 0.0)
    E = np.where(M, np.exp(S - m[:, None]), 0.0)
    l = E.sum(axis=1)
    return np.where(has[:, None], E / np.where(has, l, 1.0)[:, None], 0.0), M


def attn_bwd(row_start, prompt_len, num_resp, resp_off, resp_len, q, k, v, dout, scale=None):
    """Gradients of sum(dout * O) with respect to q, k and v (dense formulas).

    dV_g = sum_{h in g} P_h^T dO_h;  dP = dO_h V_g^T;  delta = rowsum(dO_h * O_h);
    dS = P * (dP - delta);  dQ_h = scale dS K_g;  dK_g = scale sum_{h in g} dS^T Q_h.
    Returns dq [sumT,Hq,d], dk, dv [sumT,Hkv,d] in float64.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    dout = np.asarray(dout, dtype=np.float64)
    sumT, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(len(prompt_len)):
        r0, T, P, offs, lens = _row_fields(row_start, prompt_len, num_resp, resp_off, resp_len, b)
        if T == 0:
            continue
        M = row_mask(T, P, offs, lens)
        has = M.any(axis=1)
        for h in range(Hq):
            g = h // G
            Qh = q[r0:r0 + T, h, :]
            Kg = k[r0:r0 + T, g, :]
            Vg = v[r0:r0 + T, g, :]
            dOh = dout[r0:r0 + T, h, :]
            S = np.where(M, scale * (Qh @ Kg.T), -np.inf)
            m = np.where(has, S.max(axis=1, initial=-np.inf), 0.0)
            E = np.where(M, np.exp(S - m[:, None]), 0.0)
            l = E.sum(axis=1)
            Pm = np.where(has[:, None], E / np.where(has, l, 1.0)[:, None], 0.0)
            Oh = Pm @ Vg
            dv[r0:r0 + T, g, :] += Pm.T @ dOh
            dP = dOh @ Vg.T
            delta = (dOh * Oh).sum(axis=1)
            dS = Pm * (dP - delta[:, None])
            dq[r0:r0 + T, h, :] = scale * (dS @ Kg)
            dk[r0:r0 + T, g, :] += scale * (dS.T @ Qh)
    return dq, dk, dv


# ----------------------------------------------------------------------------
# Rotary position embedding with the packed position IDs (Sec. 3.2, R2, R19)
# ----------------------------------------------------------------------------


def rope_angles(pos, d: int, base: float) -> np.ndarray:
    """Rotation angle of every (token, pair) [n, d/2]: pos * base^(-2j/d) (R19)."""
    pos = np.asarray(pos, dtype=np.float64)
    j = np.arange(d // 2, dtype=np.float64)
    w = base ** (-2.0 * j / d)
    return pos[:, None] * w[None, :]


def rope(x, pos, base: float, inverse: bool = False) -> np.ndarray:
    """Rotate every head of every token by its position (R19).

    x: [n, H, d]; pos: [n].  Pair j is (x[..., j], x[..., j + d/2]).  With
    inverse=True the rotation is undone (the transpose of the rotation, which is
    also the map that carries a gradient back through it).
    """
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[2]
    a = rope_angles(pos, d, base)[:, None, :]          # [n, 1, d/2]
    c, s = np.cos(a), np.sin(a)
    if inverse:
        s = -s
    x1, x2 = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def pack_rope(row_start, prompt_len, num_resp, resp_off, resp_len, x, base, inverse=False):
    """RoPE over the flat token axis with the packed position IDs (R2)."""
    pos = pack_position_ids(row_start, prompt_len, num_resp, resp_off, resp_len)
    return rope(x, pos, base, inverse)


def attn_fwd_rope(row_start, prompt_len, num_resp, resp_off, resp_len, q, k, v, base, scale=None):
    """Attention of rotated queries and keys: returns O, LSE and the rotated q, k."""
    args = (row_start, prompt_len, num_resp, resp_off, resp_len)
    qr = pack_rope(*args, q, base)
    kr = pack_rope(*args, k, base)
    O, LSE = attn_fwd(*args, qr, kr, v, scale)
    return O, LSE, qr, kr


def attn_bwd_rope(row_start, prompt_len, num_resp, resp_off, resp_len, q, k, v, dout, base, scale=None):
    """Gradients of sum(dout * O) with respect to the UN-rotated q and k, and v.

    The attention gradients with respect to the rotated q and k are carried back
    through the rotation by its transpose (the inverse rotation).
    """
    args = (row_start, prompt_len, num_resp, resp_off, resp_len)
    qr = pack_rope(*args, q, base)
    kr = pack_rope(*args, k, base)
    dqr, dkr, dv = attn_bwd(*args, qr, kr, v, dout, scale)
    return pack_rope(*args, dqr, base, inverse=True), pack_rope(*args, dkr, base, inverse=True), dv


# ----------------------------------------------------------------------------
# Sequence log-probabilities (Sec. 2.1 reward inputs; Sec. 3.2 equivalence)
# ----------------------------------------------------------------------------


def logsumexp_row(x: np.ndarray) -> float:
    """ln sum_v exp(x_v) of one row, computed stably in fp64."""
    m = x.max()
    return float(m + np.log(np.exp(x - m).sum()))


def seq_logprob(row_start, prompt_len, num_resp, resp_off, resp_len, logits, tokens):
    """Per-response summed token log-probabilities of a packed batch (R7, R8).

    logits: [sumT, V]; row t of the flat axis holds the next-token logits
    produced at packed position t.  tokens: [sumT] packed input IDs.
    For token j of response k of row b (row-relative position t = o_bk + j) the
    predicting position is P_b - 1 when j = 0 and t - 1 otherwise; its label is
    tokens[t].  Returns seq [B, Kmax] (empty slots 0) and tok [sumT] holding the
    log-probability of every response token at that token's own position
    (0 elsewhere).  A label outside [0, V) makes that response's sum NaN.
    """
    logits = np.asarray(logits, dtype=np.float64)
    tokens = np.asarray(tokens)
    B = len(prompt_len)
    Kmax = max([len(r) for r in resp_off] + [0])
    V = logits.shape[1]
    seq = np.zeros((B, Kmax))
    tok = np.zeros(logits.shape[0])
    for b in range(B):
        r0, T, P, offs, lens = _row_fields(row_start, prompt_len, num_resp, resp_off, resp_len, b)
        for kk, (o, L) in enumerate(zip(offs, lens)):
            s = 0.0
            for j in range(L):
                t = o + j
                src = (P - 1) if j == 0 else (t - 1)
                y = int(tokens[r0 + t])
                if not (0 <= y < V):
                    lp = float("nan")
                else:
                    row = logits[r0 + src]
                    lp = float(row[y]) - logsumexp_row(row)
                tok[r0 + t] = lp
                s += lp
            seq[b, kk] = s
    return seq, tok


def seq_logprob_grad(row_start, prompt_len, num_resp, resp_off, resp_len, logits, tokens, dseq):
    """Gradient of sum_{b,k} dseq[b,k] * seq[b,k] with respect to the logits (R16).

    seq is seq_logprob's per-response sum, so every response token contributes
    dseq[b,k] * (onehot(label) - softmax(predicting row)) to the row that
    predicts it: the last prompt row once per response (its first token), the
    row before the token otherwise.  Rows that predict no response token get 0.
    A label outside [0, V) makes the whole predicting row NaN.
    """
    logits = np.asarray(logits, dtype=np.float64)
    tokens = np.asarray(tokens)
    dseq = np.asarray(dseq, dtype=np.float64)
    V = logits.shape[1]
    grad = np.zeros_like(logits)
    bad = np.zeros(logits.shape[0], dtype=bool)
    for b in range(len(prompt_len)):
        r0, T, P, offs, lens = _row_fields(row_start, prompt_len, num_resp, resp_off, resp_len, b)
        for kk, (o, L) in enumerate(zip(offs, lens)):
            g = float(dseq[b, kk])
            for j in range(L):
                t = o + j
                src = r0 + ((P - 1) if j == 0 else (t - 1))
                y = int(tokens[r0 + t])
                if not (0 <= y < V):
                    bad[src] = True
                    continue
                row = logits[src]
                p = np.exp(row - logsumexp_row(row))
                grad[src] -= g * p
                grad[src, y] += g
    grad[bad] = np.nan
    return grad


def rm_score_rows(row_start, prompt_len, num_resp, resp_off, resp_len):
    """Flat row whose hidden state scores each (row, response) slot (R17): the
    last token of the unpacked sequence (prompt, response k), i.e. o_k + L_k - 1,
    or the last prompt token P - 1 when the response is empty; -1 when the
    sequence has no token at all or the slot is unused.  Returns [B, Kmax]."""
    B = len(prompt_len)
    Kmax = max([len(r) for r in resp_off] + [0])
    out = np.full((B, Kmax), -1, dtype=np.int64)
    for b in range(B):
        r0, T, P, offs, lens = _row_fields(row_start, prompt_len, num_resp, resp_off, resp_len, b)
        for kk, (o, L) in enumerate(zip(offs, lens)):
            last = o + L - 1 if L > 0 else P - 1
            out[b, kk] = r0 + last if last >= 0 else -1
    return out


def rm_scores(row_start, prompt_len, num_resp, resp_off, resp_len, hidden, w, bias=0.0):
    """Reward-model scores (Sec. 2.1, R17): a linear head w . h + bias on the
    hidden state that ends each (prompt, response) sequence.  hidden [sumT, H];
    returns [B, Kmax] with 0 for unused slots and token-less sequences."""
    hidden = np.asarray(hidden, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    rows = rm_score_rows(row_start, prompt_len, num_resp, resp_off, resp_len)
    out = np.zeros(rows.shape)
    for idx in np.ndindex(*rows.shape):
        if rows[idx] >= 0:
            out[idx] = float(hidden[rows[idx]] @ w) + bias
    return out


def rm_scores_grad(row_start, prompt_len, num_resp, resp_off, resp_len, hidden, w, dscores):
    """Gradients of sum(dscores * rm_scores) with respect to hidden, w and bias:
    dhidden[row] = sum of dscores over the slots read at that row, times w (0 on
    every other row); dw = sum over slots of dscores * h_row; dbias = sum of the
    dscores of the slots that have a row."""
    hidden = np.asarray(hidden, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    dscores = np.asarray(dscores, dtype=np.float64)
    rows = rm_score_rows(row_start, prompt_len, num_resp, resp_off, resp_len)
    dh = np.zeros_like(hidden)
    dw = np.zeros_like(w)
    db = 0.0
    for idx in np.ndindex(*rows.shape):
        r = rows[idx]
        if r >= 0:
            g = float(dscores[idx])
            dh[r] += g * w
            dw += g * hidden[r]
            db += g
    return dh, dw, db


def logprob_rows_needed(prompt_len, num_resp, resp_len):
    """Number of logit rows read: each row with a non-empty response reads P-1
    once plus L-1 rows per response (Sec. 3.2 packed layout, R8)."""
    n = 0
    for b in range(len(prompt_len)):
        lens = [int(x) for x in resp_len[b][:int(num_resp[b])]]
        if any(L > 0 for L in lens):
            n += 1 + sum(max(L - 1, 0) for L in lens)
    return n


def logprob_predicting_rows(row_start, prompt_len, num_resp, resp_off, resp_len):
    """Flat logit rows that predict at least one response token, ascending
    (Sec. 3.2 packed layout, R8): token j of response k of row b is predicted by
    the row's last prompt position when j = 0 and by the position before it
    otherwise."""
    rows = set()
    for b in range(len(prompt_len)):
        r0, P = int(row_start[b]), int(prompt_len[b])
        for k in range(int(num_resp[b])):
            o, L = int(resp_off[b][k]), int(resp_len[b][k])
            for j in range(L):
                rows.add(r0 + (P - 1 if j == 0 else o + j - 1))
    return sorted(rows)


# ----------------------------------------------------------------------------
# Bradley-Terry / DPO loss over ranked pairs (Sec. 2.1, R3-R6, R10)
# ----------------------------------------------------------------------------


def softplus(x: float) -> float:
    """ln(1 + e^x), stable for large |x|."""
    if x > 0:
        return x + math.log1p(math.exp(-x))
    return math.log1p(math.exp(x))


def sigmoid(x: float) -> float:
    if x >= 0:
        return 1.0 / (1.0 + math.exp(-x))
    e = math.exp(x)
    return e / (1.0 + e)


def pair_loss(num_resp, logp_pol, logp_ref, beta):
    """Ranked-pair Bradley-Terry loss with DPO rewards.

    z_k = beta * (s_pol,k - s_ref,k), or beta * s_pol,k without a reference.
    For each row and every pair a > c (a preferred, R5) the loss term is
    softplus(-(z_a - z_c)).  row_loss = mean over the row's pairs; loss = mean
    of row_loss over rows with >= 2 responses.  Returns (loss, row_loss [B],
    dlogp_pol [B, Kmax]) where dlogp_pol = d loss / d logp_pol.
    Raises ValueError when no row has two responses.
    """
    s_pol = np.asarray(logp_pol, dtype=np.float64)
    s_ref = None if logp_ref is None else np.asarray(logp_ref, dtype=np.float64)
    B, Kmax = s_pol.shape
    rows = [b for b in range(B) if int(num_resp[b]) >= 2]
    if not rows:
        raise ValueError("no row has two responses")
    R = len(rows)
    row_loss = np.zeros(B)
    grad = np.zeros((B, Kmax))
    for b in rows:
        K = int(num_resp[b])
        z = [beta * (s_pol[b, i] - (0.0 if s_ref is None else s_ref[b, i])) for i in range(K)]
        npairs = K * (K - 1) // 2
        acc = 0.0
        for a in range(K):
            for c in range(a):
                delta = z[a] - z[c]
                acc += softplus(-delta)
                w = sigmoid(-delta)
                grad[b, a] += -w * beta / (npairs * R)
                grad[b, c] += +w * beta / (npairs * R)
        row_loss[b] = acc / npairs
    loss = sum(row_loss[b] for b in rows) / R
    return float(loss), row_loss, grad


# ----------------------------------------------------------------------------
# Cost model (Sec. 3.2.1)
# ----------------------------------------------------------------------------


def cost_ratio(l_in: float, l_resp) -> float:
    """C_pp / C_original: packed cost (l_in + sum l)^2 over K (l_in + max l)^2."""
    K = len(l_resp)
    return (l_in + sum(l_resp)) ** 2 / (K * (l_in + max(l_resp)) ** 2)


def packing_is_cheaper(l_in: float, l_resp) -> bool:
    """Efficiency condition, Eq. (1): l_in + sum l < sqrt(K) (l_in + max l)."""
    K = len(l_resp)
    return (l_in + sum(l_resp)) < math.sqrt(K) * (l_in + max(l_resp))


def memory_ratio(l_in: float, l_resp) -> float:
    """Attention-memory ratio with a linear-memory attention (Sec. 3.2.1)."""
    K = len(l_resp)
    return (l_in + sum(l_resp)) / (K * (l_in + max(l_resp)))


def useful_pairs(prompt_len, num_resp, resp_len) -> int:
    """Number of visible (query, key) pairs of a packed batch, by counting the
    dense masks' True entries row by row."""
    total = 0
    for b in range(len(prompt_len)):
        P = int(prompt_len[b])
        lens = [int(x) for x in resp_len[b][:int(num_resp[b])]]
        offs = []
        o = P
        for L in lens:
            offs.append(o)
            o += L
        total += int(row_mask(o, P, offs, lens).sum())
    return total
