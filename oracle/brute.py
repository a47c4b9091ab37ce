"""Brute-force decode attention in mpmath (50 significant digits).

TEST INFRASTRUCTURE ONLY.  This evaluates the defining formula directly with
no max subtraction and no vectorisation, one (b, h) row and one key at a time:

    O[b,h,:] = sum_j exp(sigma * q.k_j) v_j / sum_j exp(sigma * q.k_j)

with KV head floor(h / g).  Tiny inputs only (it is very slow); it pins the
float64 oracle, which reaches the same numbers by a different route.
"""

from __future__ import annotations

from typing import Optional

import mpmath
import numpy as np


def _f(bits: int) -> mpmath.mpf:
    """Exact value of one bf16 bit pattern."""
    bits = int(bits)
    sign = -1 if bits & 0x8000 else 1
    e = (bits >> 7) & 0xFF
    frac = bits & 0x7F
    if e == 0:
        return sign * mpmath.mpf(frac) * mpmath.mpf(2) ** (-133)
    if e == 0xFF:
        raise ValueError("non-finite bf16 input")
    return sign * (1 + mpmath.mpf(frac) / 128) * mpmath.mpf(2) ** (e - 127)


def brute_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                    cu_seqlens: Optional[np.ndarray] = None,
                    scale: Optional[float] = None, dps: int = 50):
    """Returns (O as nested lists of mpf [B][H_Q][D], lse [B][H_Q])."""
    with mpmath.workdps(dps):
        B, H_Q, D = q.shape
        if cu_seqlens is None:
            L_K, H_KV = k.shape[1], k.shape[2]
        else:
            H_KV = k.shape[1]
        g = H_Q // H_KV
        sigma = 1 / mpmath.sqrt(D) if scale is None else mpmath.mpf(scale)
        O = []
        LSE = []
        for b in range(B):
            if cu_seqlens is None:
                rows = [(b, j) for j in range(L_K)]
                K = lambda r, hk, c: k[r[0], r[1], hk, c]
                V = lambda r, hk, c: v[r[0], r[1], hk, c]
            else:
                rows = list(range(int(cu_seqlens[b]), int(cu_seqlens[b + 1])))
                K = lambda r, hk, c: k[r, hk, c]
                V = lambda r, hk, c: v[r, hk, c]
            ob, lb = [], []
            for h in range(H_Q):
                hk = h // g
                if not rows:
                    ob.append([mpmath.mpf(0)] * D)
                    lb.append(mpmath.mpf("-inf"))
                    continue
                weights = []
                for r in rows:
                    dot = mpmath.fsum(_f(q[b, h, c]) * _f(K(r, hk, c)) for c in range(D))
                    weights.append(mpmath.exp(sigma * dot))
                den = mpmath.fsum(weights)
                ob.append([mpmath.fsum(w * _f(V(r, hk, c)) for w, r in zip(weights, rows)) / den
                           for c in range(D)])
                lb.append(mpmath.log(den))
            O.append(ob)
            LSE.append(lb)
        return O, LSE
