"""The forward-output bar shared by the GPU parity tests.

O must lie within 1e-2 (max-abs) of the fp64 oracle.  A bf16 output cannot do
better than its own rounding, half a bf16 ulp of the exact value (2^-8 at
|O| in [2, 4), 2^-7 in [4, 8)), so for bf16 outputs the bar sits on top of that
rounding.  The rest of the budget covers the bf16 probabilities of the PV
product (2^-9 relative per weight).
"""
import numpy as np

O_BAR = 1e-2


def bf16_half_ulp(x):
    """Half the spacing of bfloat16 numbers (8 significant bits) at |x|: the most a
    correctly rounded bf16 value can differ from x."""
    a = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.exp2(e - 8), 0.0)


def o_excess(got, ref, bf16_out):
    """Largest amount by which |got - ref| exceeds the bar (<= 0 passes)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.size == 0:
        return 0.0
    allow = O_BAR + (bf16_half_ulp(ref) if bf16_out else 0.0)
    return float((np.abs(got - ref) - allow).max())
