"""Oracle, part 4: PSA-Search (Algorithm 3 in the appendix "Process of PSA-Search", and the
dual interface of Sec. 3.3, "Automatic and Efficient Sparsity Discovery") -- test
infrastructure only.

What is computed:

* The loss of a candidate mask M for one head is the L2 loss between the head's sparse
  attention output under M and its full attention output.  The paper does not spell out the
  normalisation; its thresholds (alpha = 0.007 to 0.03) are only meaningful for a relative
  measure, so the loss here is ||O_M - O_full||_F / ||O_full||_F over all tokens and channels of
  the head (and of every batch element).
* Sparsity(M) = 1 - (kept blocks / all blocks) of the head's block map.
* Selection (Algorithm 3): sort the (loss, M) results of a head by ascending loss; start from the
  lowest-loss mask; walk the sorted list and, for every mask whose loss is at most alpha, take it
  if its sparsity is strictly higher than the current choice's.  Re-running only this step
  re-tunes alpha (the paper keeps HeadResults for that).
* Dual interface: for a target sparsity, the mask of minimal loss among those at least that
  sparse; the paper gives no rule for a target no candidate reaches, the reading taken is the
  sparsest candidate (lowest loss among equally sparse ones).

Ties in the sort keep the candidates' original order (a stable sort).
"""
import numpy as np

from .attention import masked_attention


def l2_loss(o_sparse, o_full):
    """Relative L2 loss of one head: ||o_sparse - o_full|| / ||o_full|| (float64)."""
    a = np.asarray(o_sparse, dtype=np.float64)
    b = np.asarray(o_full, dtype=np.float64)
    den = np.sqrt((b * b).sum())
    num = np.sqrt(((a - b) ** 2).sum())
    return float(num / den) if den > 0 else (0.0 if num == 0 else float("inf"))


def head_results(q, k, v, keeps, block, scale):
    """(loss, sparsity) of every candidate block map in `keeps` for one head (q, k, v [N, d])."""
    nb = -(-q.shape[0] // block)
    o_full, _ = masked_attention(q, k, v, np.ones((nb, nb), dtype=np.uint8), block, scale)
    out = []
    for keep in keeps:
        o, _ = masked_attention(q, k, v, keep, block, scale)
        out.append((l2_loss(o, o_full), 1.0 - float(np.asarray(keep, dtype=bool).mean())))
    return out


def select_alpha(results, alpha):
    """Index of the candidate Algorithm 3 picks for one head; results = [(loss, sparsity), ...]."""
    order = sorted(range(len(results)), key=lambda i: results[i][0])
    best = order[0]
    for i in order:
        loss, sparsity = results[i]
        if loss <= alpha and sparsity > results[best][1]:
            best = i
    return best


def select_target(results, target):
    """Index of the candidate the dual interface picks for a target sparsity."""
    ok = [i for i, (_, s) in enumerate(results) if s >= target]
    if ok:
        return min(ok, key=lambda i: (results[i][0], i))
    top = max(s for _, s in results)
    return min((i for i, (_, s) in enumerate(results) if s == top), key=lambda i: (results[i][0], i))
