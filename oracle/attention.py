"""FlowKV decode attention oracle (NumPy, CPU).  Test infrastructure only.

What the decode attention of one layer computes (the causal-attention
equation of the decoding section, with the 1/sqrt(d) score scaling of Eq. 6
passed in as `scale`), for the query of the current position t and the KV
cache of positions 0..t:

  for each query head h (GQA: head h reads KV group g = h // (H/G)):
      s_j = scale * q_h . k_{g,j}                 j in the attended range
      o_h = sum_j exp(s_j) v_{g,j} / sum_j exp(s_j)

Attended range: 0..t for full (global) attention; for sliding-window
attention of window Lw, max(0, t - Lw + 1)..t.

`decode_attention` evaluates that definition in float64 (scores from the
exact bf16 values, a max shift for range only).  `decode_attention_chunked`
follows FlowKV's chunk sweep instead -- Eq. 6-12 with a query chunk of 1, the
chunks taken left to right with the running max m, denominator l and weighted
sum Y -- and exists to show that the recurrence reproduces the definition.
"""
from __future__ import annotations

import numpy as np

from .q4nx import bf16_to_f32


def attended_range(t: int, window: int):
    """[j0, j1) of the positions the query at position t attends to."""
    j1 = t + 1
    j0 = 0 if window <= 0 else max(0, j1 - window)
    return j0, j1


def _f64(bits):
    return bf16_to_f32(bits).astype(np.float64)


def decode_attention(q_bits, K_bits, V_bits, t: int, window: int, scale: float):
    """q [H][d], K and V [G][L][d] (bf16 bits) -> o [H][d] float64, plus the
    per-head weight bound sum_j p_j |v_j| used by the tolerance."""
    q, K, V = _f64(q_bits), _f64(K_bits), _f64(V_bits)
    H, d = q.shape
    G = K.shape[0]
    hg = H // G
    j0, j1 = attended_range(t, window)
    o = np.zeros((H, d))
    bound = np.zeros((H, d))
    for h in range(H):
        g = h // hg
        s = scale * (K[g, j0:j1] @ q[h])
        w = np.exp(s - s.max())
        p = w / w.sum()
        o[h] = p @ V[g, j0:j1]
        bound[h] = p @ np.abs(V[g, j0:j1])
    return o, bound


def decode_attention_chunked(q_bits, K_bits, V_bits, t: int, window: int, scale: float, chunk: int):
    """The same output through FlowKV's left-to-right chunk recurrence."""
    q, K, V = _f64(q_bits), _f64(K_bits), _f64(V_bits)
    H, d = q.shape
    G = K.shape[0]
    hg = H // G
    j0, j1 = attended_range(t, window)
    o = np.zeros((H, d))
    for h in range(H):
        g = h // hg
        m_left, l_left, Y_left = -np.inf, 0.0, np.zeros(d)
        for c0 in range(j0, j1, chunk):
            c1 = min(j1, c0 + chunk)
            S = scale * (K[g, c0:c1] @ q[h])             # Eq. 6 (one query row)
            m = max(S.max(), m_left)                      # Eq. 7
            F = np.exp(S - m)                             # Eq. 8
            C = np.exp(m_left - m)                        # Eq. 9 (0 for the first chunk)
            l_left = C * l_left + F.sum()                 # Eq. 10
            Y_left = C * Y_left + F @ V[g, c0:c1]         # Eq. 11
            m_left = m
        o[h] = Y_left / l_left                            # Eq. 12
    return o
