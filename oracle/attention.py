"""Oracle, part 2: naive masked softmax attention (test infrastructure only).

What is computed (the plain definition that the paper's kernel reaches up to rounding,
Algorithm 2 in the appendix "Pseudocode for PSA-Kernel": S = Q K^T, padded positions set to
-inf, safe softmax, P V, accumulated over the kept KV blocks): for query i of one
(batch, head), with the kept key set J_i = { j < N : block(i), block(j) kept },

    s_j  = scale * <q_i, k_j>
    m    = max_{j in J_i} s_j,   p_j = exp(s_j - m),   l = sum_j p_j
    o_i  = (sum_j p_j v_j) / l,  lse_i = m + ln l

Keys at or beyond N do not exist, which is what the -inf padding achieves.  A row whose
J_i is empty (possible with non-zero offsets) gets o_i = 0 and lse_i = -inf: the paper does
not discuss it, this is the reading taken.  The softmax scale is an argument (the paper
does not state it; the workloads use 1/sqrt(d)).  Arithmetic is float64 on the given inputs.
"""
import numpy as np


def masked_attention(q, k, v, keep, block, scale, rows=None, groups=None):
    """Masked attention for one (batch, head).

    q, k, v : arrays [N, d] (any float dtype; upcast to float64)
    keep    : bool/uint8 array [nb, nb], row = query block, column = key block
    block   : tokens per block (block b = tokens [b*block, (b+1)*block))
    rows    : query token indices to evaluate (default: all N)
    groups  : optional int array [N], the block of every token when blocks are not runs of
              consecutive tokens (PSABlocks of the original token order); `block` is then unused
    returns : (o [R, d] float64, lse [R] float64)
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    keep = np.asarray(keep).astype(bool)
    n = k.shape[0]
    rows = np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)
    key_block = np.arange(n) // block if groups is None else np.asarray(groups, dtype=np.int64)
    mask = keep[key_block[rows]][:, key_block]               # [R, N]: q_i may attend to k_j
    s = scale * (q[rows] @ k.T)
    s = np.where(mask, s, -np.inf)
    m = s.max(axis=1)
    o = np.zeros((rows.shape[0], v.shape[1]), dtype=np.float64)
    lse = np.full(rows.shape[0], -np.inf, dtype=np.float64)
    live = np.isfinite(m)
    p = np.exp(s[live] - m[live, None])
    l = p.sum(axis=1)
    o[live] = (p @ v) / l[:, None]
    lse[live] = m[live] + np.log(l)
    return o, lse
