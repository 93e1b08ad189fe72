"""Reference decode loop: append, attend, evict (oracle side).

TEST INFRASTRUCTURE ONLY (see the package header).

Order within one decode step t (1-based), a reading the paper leaves open:
  1. every (layer, KV head) caches the new pair at position lp + t - 1
     (Section 2: each decode step appends one pair);
  2. every query head attends over its KV head's cached pairs, its own new
     key included (Section 2, "Notation");
  3. at the end of the step the periodic trigger may evict every (layer, KV
     head) of the sequence (Eq. 1, Section 3, Appendix F).
Rows are supplied by the caller as functions of (layer, head, position), so
the oracle never sees memory layout; this is the plain definition with no
blocking or reordering.  Parity: pinned through its parts (see ``evict``
and ``attention``) and by the tests' brute-force step checks.
"""

import numpy as np

from .attention import gqa_decode
from .evict import SequenceReplay


def run_decode(num_layers, num_q_heads, num_kv_heads, prompt_len, steps,
               k_keep, recent_r, every, seed, request_id,
               q_rows, k_rows, v_rows, record_steps=None):
    """Decode one sequence for ``steps`` steps.

    q_rows(layer, step0) -> [Hq, d] query of 0-based step ``step0``.
    k_rows(layer, kv_head, positions) / v_rows(...) -> [n, d] rows.
    record_steps: iterable of 0-based steps whose outputs are returned
    (default: all).

    Returns (outputs, replay): outputs maps step0 -> [L, Hq, d] float64;
    replay holds the final positions per (layer, KV head) and the event log.
    """
    heads = [(l, g) for l in range(num_layers) for g in range(num_kv_heads)]
    rep = SequenceReplay(prompt_len, k_keep, recent_r, every, seed,
                         request_id, heads)
    wanted = None if record_steps is None else set(int(s) for s in record_steps)
    outputs = {}
    for s in range(steps):
        rep.append()
        if wanted is None or s in wanted:
            per_layer = []
            for layer in range(num_layers):
                Ks = [k_rows(layer, g, rep.P[(layer, g)])
                      for g in range(num_kv_heads)]
                Vs = [v_rows(layer, g, rep.P[(layer, g)])
                      for g in range(num_kv_heads)]
                per_layer.append(gqa_decode(q_rows(layer, s), Ks, Vs))
            outputs[s] = np.stack(per_layer)
        rep.end_step()
    return outputs, rep
