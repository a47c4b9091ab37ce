"""Plain fp64 single-query decode attention, its split mirror and the combine.

TEST INFRASTRUCTURE ONLY (see the package docstring): never used by the
product path.

What is computed (paper, Section 2.1: decode attention with L_Q = 1 is a
softmax-weighted reduction over the sequence dimension; Section 2.2 and 3.1:
num_splits distributes that reduction along the sequence; Section 3.1 and
5.3: the split results are merged by a final reduction).  For query head h of
sequence b, with KV head h' = floor(h / g), g = H_Q / H_KV, scale sigma
(default 1/sqrt(D)) and keys j < L_b:

    s_j   = sigma * sum_c q[b,h,c] * k[j,h',c]
    m     = max_j s_j,   p_j = exp(s_j - m),   l = sum_j p_j
    O     = (sum_j p_j v[j,h',:]) / l,          lse = m + ln l

The split mirror gives, for any partition of the keys into chunks i,
    m_i = max_{j in i} s_j,  l_i = sum_{j in i} exp(s_j - m_i),
    Otilde_i = sum_{j in i} exp(s_j - m_i) v_j
(an empty chunk gives m_i = -inf, l_i = 0, Otilde_i = 0), and the combine is
    M = max_i m_i,  w_i = exp(m_i - M) (0 for empty chunks),
    L = sum_i w_i l_i,  O = (sum_i w_i Otilde_i) / L,  lse = M + ln L.

Readings where the paper is silent: scale 1/sqrt(D); query head h uses KV
head floor(h / g); non-causal (for one query at the end of the sequence the
causal mask removes nothing); an empty sequence gives O = 0, lse = -inf.

Inputs are bf16 bit patterns (uint16), upcast exactly to float64.
"""

from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact bf16 -> float64: the 16 bits are the top half of a float32."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def _seq_rows(lengths: np.ndarray, cu_seqlens: Optional[np.ndarray], L_K: int, b: int) -> Tuple[int, int]:
    """(first row, length) of sequence b in the K/V row space.

    Fixed layout [B, L_K, H_KV, D] is read as B*L_K rows; the varlen layout
    [sum L_b, H_KV, D] starts sequence b at cu_seqlens[b]."""
    if cu_seqlens is None:
        return b * L_K, int(lengths[b])
    return int(cu_seqlens[b]), int(cu_seqlens[b + 1] - cu_seqlens[b])


def _as_rows(x: np.ndarray, cu_seqlens: Optional[np.ndarray]) -> np.ndarray:
    """K or V as float64 rows [n_rows, H_KV, D]."""
    if cu_seqlens is None:
        B, L, H, D = x.shape
        return bf16_bits_to_f64(x.reshape(B * L, H, D))
    return bf16_bits_to_f64(x)


def _check(q: np.ndarray, k: np.ndarray, cu_seqlens) -> Tuple[int, int, int, int, int]:
    B, H_Q, D = q.shape
    if cu_seqlens is None:
        _, L_K, H_KV, _ = k.shape
    else:
        _, H_KV, _ = k.shape
        L_K = 0
    if H_Q % H_KV:
        raise ValueError("H_Q must be a multiple of H_KV")
    return B, H_Q, H_KV, D, L_K


def decode_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                     lengths: Optional[np.ndarray] = None,
                     cu_seqlens: Optional[np.ndarray] = None,
                     scale: Optional[float] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Unsplit attention.  Returns (O [B,H_Q,D] float64, lse [B,H_Q] float64).

    q: uint16 [B,H_Q,D]; k, v: uint16 [B,L_K,H_KV,D] or, with cu_seqlens,
    [sum L_b, H_KV, D]; lengths: int [B] (fixed layout: may be omitted)."""
    B, H_Q, H_KV, D, L_K = _check(q, k, cu_seqlens)
    g = H_Q // H_KV
    sigma = 1.0 / np.sqrt(D) if scale is None else float(scale)
    if lengths is None:
        lengths = np.full(B, L_K, dtype=np.int64)
    qf = bf16_bits_to_f64(q)
    out = np.zeros((B, H_Q, D), dtype=np.float64)
    lse = np.full((B, H_Q), -np.inf, dtype=np.float64)
    for b in range(B):
        # Upcast one sequence at a time so the largest workload never holds
        # more than one sequence of float64 K/V.
        row0, L = _seq_rows(lengths, cu_seqlens, L_K, b)
        if L == 0:
            continue
        if cu_seqlens is None:
            kb = bf16_bits_to_f64(k[b])          # [L, H_KV, D]
            vb = bf16_bits_to_f64(v[b])
        else:
            kb = bf16_bits_to_f64(k[row0:row0 + L])
            vb = bf16_bits_to_f64(v[row0:row0 + L])
        for hk in range(H_KV):
            Qg = qf[b, hk * g:(hk + 1) * g, :]            # [g, D]
            S = sigma * (Qg @ kb[:, hk, :].T)              # [g, L]
            m = S.max(axis=1, keepdims=True)
            P = np.exp(S - m)
            l = P.sum(axis=1, keepdims=True)
            out[b, hk * g:(hk + 1) * g, :] = (P @ vb[:, hk, :]) / l
            lse[b, hk * g:(hk + 1) * g] = (m + np.log(l))[:, 0]
    return out, lse


def even_bounds(L: int, s: int) -> List[int]:
    """Cut points of a balanced partition of L keys into s chunks:
    chunk i is [floor(i*L/s), floor((i+1)*L/s)).  With s > L some chunks are
    empty.  Used by the split mirror in tests; the result of the method does
    not depend on which partition is taken."""
    return [(i * L) // s for i in range(s + 1)]


def split_partials(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                   bounds: Sequence[Sequence[int]],
                   lengths: Optional[np.ndarray] = None,
                   cu_seqlens: Optional[np.ndarray] = None,
                   scale: Optional[float] = None) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Per-chunk partial softmax state for a given partition.

    bounds[b] is the list of s+1 cut points of sequence b (0 = first key,
    last = L_b, non-decreasing).  Returns (o_part [s,B,H_Q,D], m [s,B,H_Q],
    l [s,B,H_Q]) in float64, m in natural-log units of the scaled score."""
    B, H_Q, H_KV, D, L_K = _check(q, k, cu_seqlens)
    g = H_Q // H_KV
    sigma = 1.0 / np.sqrt(D) if scale is None else float(scale)
    if lengths is None:
        lengths = np.full(B, L_K, dtype=np.int64)
    s = len(bounds[0]) - 1
    qf = bf16_bits_to_f64(q)
    o_part = np.zeros((s, B, H_Q, D), dtype=np.float64)
    m_part = np.full((s, B, H_Q), -np.inf, dtype=np.float64)
    l_part = np.zeros((s, B, H_Q), dtype=np.float64)
    for b in range(B):
        row0, L = _seq_rows(lengths, cu_seqlens, L_K, b)
        cuts = list(bounds[b])
        if len(cuts) != s + 1 or cuts[0] != 0 or cuts[-1] != L or any(
                cuts[i] > cuts[i + 1] for i in range(s)):
            raise ValueError(f"bad cut points for sequence {b}: {cuts}")
        if cu_seqlens is None:
            kb = bf16_bits_to_f64(k[b])
            vb = bf16_bits_to_f64(v[b])
        else:
            kb = bf16_bits_to_f64(k[row0:row0 + L])
            vb = bf16_bits_to_f64(v[row0:row0 + L])
        for i in range(s):
            lo, hi = cuts[i], cuts[i + 1]
            if hi == lo:
                continue
            for hk in range(H_KV):
                Qg = qf[b, hk * g:(hk + 1) * g, :]
                S = sigma * (Qg @ kb[lo:hi, hk, :].T)
                m = S.max(axis=1, keepdims=True)
                P = np.exp(S - m)
                o_part[i, b, hk * g:(hk + 1) * g, :] = P @ vb[lo:hi, hk, :]
                m_part[i, b, hk * g:(hk + 1) * g] = m[:, 0]
                l_part[i, b, hk * g:(hk + 1) * g] = P.sum(axis=1)
    return o_part, m_part, l_part


def combine_partials(o_part: np.ndarray, m_part: np.ndarray,
                     l_part: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Log-sum-exp merge of s partial states along axis 0.

    Empty chunks (l_i = 0) get weight 0.  When every chunk is empty the
    result is O = 0, lse = -inf."""
    o_part = np.asarray(o_part, dtype=np.float64)
    m_part = np.asarray(m_part, dtype=np.float64)
    l_part = np.asarray(l_part, dtype=np.float64)
    nonempty = l_part > 0
    M = np.where(nonempty, m_part, -np.inf).max(axis=0)            # [...]
    any_ = nonempty.any(axis=0)
    Msafe = np.where(any_, M, 0.0)
    w = np.where(nonempty, np.exp(np.where(nonempty, m_part, 0.0) - Msafe), 0.0)
    L = (w * l_part).sum(axis=0)
    num = (w[..., None] * o_part).sum(axis=0)
    Lsafe = np.where(any_, L, 1.0)
    O = np.where(any_[..., None], num / Lsafe[..., None], 0.0)
    lse = np.where(any_, Msafe + np.log(Lsafe), -np.inf)
    return O, lse
