"""Pure-Python brute force for tiny shapes (TEST INFRASTRUCTURE ONLY).

A second route to the masked linear, independent of ``tasq_oracle.c``: it
works on the paper's unsigned codes and drops bits one at a time.

* Weights are stored as unsigned n-bit codes with a zero point (App. A.1.1);
  the signed int8 buffer w corresponds to the code Q = w + 128 with integer
  zero point 128.
* Sec. 3.1 Eq. (truncquant): the (n-1)-bit code is floor(Q_n / 2).
* Sec. 3.2.1 Eq. (lsb_extraction): LSB = Q_n - 2 Q_{n-1}; Eq. (lsb_masking):
  with the mask off the LSB is subtracted, the scale is kept.  Applied again
  to the remaining least significant bits, dropping k bits removes
  sum_{j<k} 2^j * LSB_j, where LSB_j is the low bit of the code truncated j
  times.
* Sec. 3.1 Eq. (qalora): the layer output is the plain product of the
  integer activation with the masked integer weight; App. A dequantisation
  multiplies by the two scales.
No numpy, no C: loops over Python integers.
"""
from __future__ import annotations

ZERO_POINT = 128
N_BITS = 8


def truncate_once(q: int) -> int:
    """Eq. (truncquant): one bit less precision, floor(q / 2) on a code >= 0."""
    assert q >= 0
    return q // 2


def masked_code(q: int, b: int) -> int:
    """Unsigned code with its 8 - b least significant bits removed."""
    assert 0 <= q < 1 << N_BITS and 1 <= b <= N_BITS
    out = q
    cur = q                      # the code truncated j times
    for j in range(N_BITS - b):
        nxt = truncate_once(cur)
        lsb = cur - 2 * nxt      # Eq. (lsb_extraction) at precision 8 - j
        out -= (1 << j) * lsb    # Eq. (lsb_masking) with M = 0, weight 2^j
        cur = nxt
    return out


def masked_weight(w: int, b: int) -> int:
    """Signed weight after the mask, via the unsigned code and zero point."""
    return masked_code(w + ZERO_POINT, b) - ZERO_POINT


def masked_linear(X, W, sx, sw, b, bias=None):
    """acc and y as nested lists for X [M][K], W [N][K] (lists of ints)."""
    M, N = len(X), len(W)
    acc = [[0] * N for _ in range(M)]
    y = [[0.0] * N for _ in range(M)]
    Wm = [[masked_weight(int(v), b) for v in row] for row in W]
    for m in range(M):
        for n in range(N):
            s = 0
            for xv, wv in zip(X[m], Wm[n]):
                s += int(xv) * wv
            acc[m][n] = s
            y[m][n] = s * float(sx) * float(sw[n]) + (float(bias[n]) if bias is not None else 0.0)
    return acc, y
