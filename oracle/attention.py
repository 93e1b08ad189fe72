"""Exact softmax decode attention over the kept rows (oracle side).

TEST INFRASTRUCTURE ONLY (see the package header).

Section 2 ("Notation") defines a head's output for the current query q as
    o = sum_i alpha_i v_i,   alpha = softmax_i(q . k_i / sqrt(d))
over the pairs the head holds.  Grouped-query heads share their KV head's
cache and keep-set (Appendix F): query head h reads KV head floor(h / G),
G = (query heads) / (KV heads), contiguous groups (reading of the GQA map).
Keys are post-rotary already (Appendix F), so no rotation is applied here.

Everything is evaluated in float64 with the maximum subtracted before the
exponential.  Parity: pinned by the tests (one row returns its value, equal
keys or a zero query return the mean value, a dominant logit returns its
value, permutation invariance, and agreement with torch's
scaled_dot_product_attention in float64).
"""

import numpy as np


def softmax_attention(q, K, V):
    """One query head over N cached rows.

    q: [d], K: [N, d], V: [N, d] (any real dtype; promoted to float64).
    Returns o: [d] float64.
    """
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    d = q.shape[-1]
    logits = (K @ q) / np.sqrt(d)
    w = np.exp(logits - logits.max())
    return (w / w.sum()) @ V


def gqa_decode(q, K_by_head, V_by_head):
    """All query heads of one (sequence, layer) for one decode step.

    q: [Hq, d]; K_by_head / V_by_head: lists of Hkv arrays [N_g, d] holding
    each KV head's kept rows.  Returns [Hq, d] float64.
    """
    q = np.asarray(q, dtype=np.float64)
    hq = q.shape[0]
    hkv = len(K_by_head)
    group = hq // hkv
    out = np.empty_like(q)
    for h in range(hq):
        g = h // group
        out[h] = softmax_attention(q[h], K_by_head[g], V_by_head[g])
    return out
