"""Seeded synthetic workload rows: queries, keys and values.

This module is input preparation shared by the tests, the benchmark and the
smoke check.  It holds none of the method's arithmetic (no eviction, no
attention): it only produces deterministic rows, identically on the CPU and
on the GPU, so that the CPU oracle and the HIP path see the same inputs.

Distributions (the shapes of the measured workloads):
* queries ~ N(0, 1);
* keys and values ~ N(0, 1) times a per-(layer, KV head, channel) scale drawn
  once from U(0.5, 2), separately for keys and values (``scaled=True``);
  unscaled N(0, 1) for the tiny fp32 case.

Construction.  ``numpy.random.default_rng(seed)`` draws a pool of P rows of
N(0,1) float32 for keys and values, the scale tables, then a second pool of
P rows for queries (so a query is never a copy of a cached key, which would
make its attention collapse onto that one row).  The row for (kind, seq,
layer, head, j) is pool[h mod P] of its kind's pool, where h is an integer
hash of its arguments computed with int64 tensor operations that never
overflow; the float32 product with the scale and the round-to-nearest-even
cast to bfloat16 are IEEE-exact, so CPU and GPU produce bit-identical rows.

``j`` is the row id: a prompt position p < prompt_len uses j = p; a
generated position p uses j = prompt_len + ((p - prompt_len) mod ring) when
``ring`` is set (the benchmark keeps a ring of ``ring`` steps of inputs
resident in HBM), else j = p.  Queries of 0-based decode step s use
j = s mod ring (or s).
"""

import numpy as np
import torch

KIND_Q, KIND_K, KIND_V = 0, 1, 2

_MOD = 2147483647            # 2^31 - 1 (prime); every product stays < 2^63
_MULTS = (48271, 69621, 16807, 39373, 40692)


def _hash(kind, seq, layer, head, j):
    """Integer hash of broadcastable int64 tensors, values in [0, 2^31-1)."""
    h = torch.full((), kind + 1, dtype=torch.int64, device=j.device)
    for x, a in zip((seq, layer, head, j), _MULTS):
        h = (h * a + x + 1) % _MOD
        h = (h ^ (h >> 13)) % _MOD
        h = (h * 1103515245) % _MOD
    h = (h * _MULTS[4] + 12345) % _MOD
    return h ^ (h >> 11)


class Workload:
    """Deterministic rows for one workload shape.

    dtype: torch.float32 or torch.bfloat16.  All row methods accept
    broadcastable int64 tensors (or ints) for their index arguments and
    return float tensors of shape broadcast(...) + [head_dim] on ``device``.
    """

    def __init__(self, seed, num_layers, num_q_heads, num_kv_heads, head_dim,
                 dtype, scaled, ring=None, pool_rows=1 << 16, device="cpu"):
        self.seed = int(seed)
        self.L, self.Hq, self.Hkv, self.d = (int(num_layers), int(num_q_heads),
                                             int(num_kv_heads), int(head_dim))
        self.dtype = dtype
        self.scaled = bool(scaled)
        self.ring = None if ring is None else int(ring)
        self.P = int(pool_rows)
        self.device = torch.device(device)
        rng = np.random.default_rng(self.seed)
        pool = rng.standard_normal((self.P, self.d)).astype(np.float32)
        sk = rng.uniform(0.5, 2.0, (self.L, self.Hkv, self.d)).astype(np.float32)
        sv = rng.uniform(0.5, 2.0, (self.L, self.Hkv, self.d)).astype(np.float32)
        qpool = rng.standard_normal((self.P, self.d)).astype(np.float32)
        self.pool = torch.from_numpy(pool).to(self.device)
        self.qpool = torch.from_numpy(qpool).to(self.device)
        self.scale_k = torch.from_numpy(sk).to(self.device)
        self.scale_v = torch.from_numpy(sv).to(self.device)

    def to(self, device):
        """Same workload with its tables on another device."""
        w = object.__new__(Workload)
        w.__dict__.update(self.__dict__)
        w.device = torch.device(device)
        w.pool = self.pool.to(w.device)
        w.qpool = self.qpool.to(w.device)
        w.scale_k = self.scale_k.to(w.device)
        w.scale_v = self.scale_v.to(w.device)
        return w

    def _t(self, x):
        return torch.as_tensor(x, dtype=torch.int64, device=self.device)

    def row_id(self, positions, prompt_len):
        """Row id j of cached positions (see the module header)."""
        p = self._t(positions)
        if self.ring is None:
            return p
        lp = self._t(prompt_len)
        gen = lp + torch.remainder(p - lp, self.ring)
        return torch.where(p < lp, p, gen)

    def _rows(self, kind, seq, layer, head, j):
        seq, layer, head, j = (self._t(x) for x in (seq, layer, head, j))
        idx = _hash(kind, seq, layer, head, j) % self.P
        x = (self.qpool if kind == KIND_Q else self.pool)[idx]
        if self.scaled and kind != KIND_Q:
            table = self.scale_k if kind == KIND_K else self.scale_v
            lh = torch.broadcast_tensors(layer, head, idx)
            x = x * table[lh[0], lh[1]]
        return x.to(self.dtype)

    def k_rows(self, seq, layer, kv_head, positions, prompt_len):
        """Key rows of the given cached positions."""
        return self._rows(KIND_K, seq, layer, kv_head,
                          self.row_id(positions, prompt_len))

    def v_rows(self, seq, layer, kv_head, positions, prompt_len):
        """Value rows of the given cached positions."""
        return self._rows(KIND_V, seq, layer, kv_head,
                          self.row_id(positions, prompt_len))

    def q_rows(self, seq, layer, q_head, step0):
        """Query rows of 0-based decode step ``step0``."""
        s = self._t(step0)
        j = s if self.ring is None else torch.remainder(s, self.ring)
        return self._rows(KIND_Q, seq, layer, q_head, j)

    # Batched helpers laid out the way the decode entry points take them.

    def q_step(self, seqs, layer, step0s):
        """[n, Hq, d] queries of sequences ``seqs`` at their 0-based steps."""
        seqs = self._t(seqs).view(-1, 1)
        steps = self._t(step0s).view(-1, 1)
        heads = torch.arange(self.Hq, device=self.device).view(1, -1)
        return self.q_rows(seqs, layer, heads, steps)

    def kv_step(self, seqs, layer, positions, prompt_lens):
        """([n, Hkv, d], [n, Hkv, d]) new key/value rows at the given positions."""
        seqs = self._t(seqs).view(-1, 1)
        pos = self._t(positions).view(-1, 1)
        lp = self._t(prompt_lens).view(-1, 1)
        heads = torch.arange(self.Hkv, device=self.device).view(1, -1)
        return (self.k_rows(seqs, layer, heads, pos, lp),
                self.v_rows(seqs, layer, heads, pos, lp))
