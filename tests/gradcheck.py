"""Gradient checks shared by the GPU parity tests.

The gradient bar is a relative Frobenius error of 2e-2 against the fp64 oracle.
Checked only on whole tensors, an error confined to a few rows -- one short
response, the keys of the last response, a tile that straddles a segment
boundary -- would hide under it.  So every segment of every packed row (its
prompt, and each response) is also held to the bar on its own: the query rows
of the segment for dQ, its key rows for dK and dV, all heads together.

A segment whose reference gradient is tiny next to the tensor's is measured
against a floor instead of its own norm: 5% of the tensor's RMS over the
segment's element count.  (The first token of a row sees one key, so its
softmax row is exactly one-hot and its dS exactly 0 in exact arithmetic; the
kernels' bf16 rounding of P and O leaves a residue there that no relative bar
on a zero can hold.)
"""
import numpy as np

G_TOL = 2e-2
SEG_FLOOR = 0.05


def rel_fro(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


def segments(pack):
    """(label, first flat token, one past the last) of every non-empty prompt
    and response of the pack."""
    out = []
    for b in range(pack.num_rows):
        r0 = int(pack.row_start[b])
        P = int(pack.prompt_len[b])
        if P > 0:
            out.append((f"row {b} prompt", r0, r0 + P))
        for k in range(int(pack.num_resp[b])):
            o, L = int(pack.resp_off[b, k]), int(pack.resp_len[b, k])
            if L > 0:
                out.append((f"row {b} response {k}", r0 + o, r0 + o + L))
    return out


def segment_errors(pack, got, ref, floor=SEG_FLOOR):
    """Relative Frobenius error of every segment's rows (tokens on axis 0)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    errs = []
    for label, a, b in segments(pack):
        g, r = got[a:b], ref[a:b]
        denom = max(float(np.linalg.norm(r)), floor * rms * np.sqrt(r.size), 1e-300)
        errs.append((label, float(np.linalg.norm(g - r)) / denom))
    return errs


def check_grad(pack, name, got, ref, tol=G_TOL):
    """Whole-tensor and per-segment relative Frobenius errors within `tol`;
    returns the largest of them (for the test's log line)."""
    whole = rel_fro(got, ref)
    assert whole <= tol, (name, "whole tensor", whole)
    worst = whole
    for label, err in segment_errors(pack, got, ref):
        assert err <= tol, (name, label, err)
        worst = max(worst, err)
    return worst
