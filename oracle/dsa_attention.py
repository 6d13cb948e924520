"""CPU oracle of the paper's DSA Sparse Attention (Section 3.1.2).

TEST INFRASTRUCTURE ONLY: tests/, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` are the only users; the product path never
imports it and it never imports the product path.

For each query token t and head h (paper Section 3.1.2): gather the token's
TopK cached entries from its sparse index list, form the scaled logits
q_nope . Kc_j + q_pe . Kp_j, take a base-2 softmax over them, and accumulate
the weights times Kc_j into a 512-wide output; also return the log-sum-exp.
Plain fp64 numpy on the exactly decoded bf16 inputs (no integer decision
follows from these floats, so the oracle keeps full precision).

Layouts: q_nope [T, H, 512], q_pe [T, H, 64] bf16 bit patterns (uint16);
ckv [num_pages, PS, 512], kpe [num_pages, PS, 64] bf16 bit patterns;
indices [T, TopK] int32 physical cache indices page * PS + slot, -1 = none.
Readings where the paper is silent:
  s_j   = (q_nope . Kc_j + q_pe . Kp_j) * sm_scale * log2(e)    (base-2 logits)
  lse   = log2(sum_j 2^s_j)                                      (base 2)
  out   = sum_j 2^(s_j - lse) * Kc_j                             (values = Kc)
  a token with no valid index: out = 0, lse = -inf.
"""
from __future__ import annotations

import numpy as np

LOG2E = 1.4426950408889634


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact decode of bf16 bit patterns: the high half of an fp32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def sparse_attention(q_nope, q_pe, ckv, kpe, indices, sm_scale: float, tokens=None):
    """Returns (out float64 [n, H, 512], lse float64 [n, H]) for the listed tokens
    (all by default)."""
    T, H, DC = q_nope.shape
    DP = q_pe.shape[2]
    PS = ckv.shape[1]
    kc_all = ckv.reshape(-1, DC)
    kp_all = kpe.reshape(-1, DP)
    toks = range(T) if tokens is None else tokens
    outs, lses = [], []
    for t in toks:
        idx = np.asarray(indices[t])
        idx = idx[idx >= 0]
        if idx.size == 0:
            outs.append(np.zeros((H, DC)))
            lses.append(np.full(H, -np.inf))
            continue
        kc = bf16_to_f64(kc_all[idx])                 # [n, 512]
        kp = bf16_to_f64(kp_all[idx])                 # [n, 64]
        qn = bf16_to_f64(q_nope[t])                   # [H, 512]
        qp = bf16_to_f64(q_pe[t])                     # [H, 64]
        s = (qn @ kc.T + qp @ kp.T) * (float(sm_scale) * LOG2E)   # [H, n]
        m = s.max(axis=1, keepdims=True)
        w = np.exp2(s - m)
        l = w.sum(axis=1, keepdims=True)
        outs.append((w / l) @ kc)
        lses.append((m + np.log2(l))[:, 0])
    return np.stack(outs), np.stack(lses)
