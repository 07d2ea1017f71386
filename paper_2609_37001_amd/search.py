"""PSA-Search (Algorithm 3 in the appendix "Process of PSA-Search"; the dual interface of
Sec. 3.3, "Automatic and Efficient Sparsity Discovery").

Scoring runs on the GPU through the library: for candidate c, one psa_attention_fwd call gives
every head its own candidate mask; psa_l2_distance reduces its output against the full
attention output (psa_dense_fwd, computed once).  The loss of a head is the relative L2 distance
sqrt(sum (O_M - O_full)^2 / sum O_full^2) over its tokens, channels and batch elements; the
sparsity of a mask is 1 - kept blocks / all blocks of its block map.  The per-head (loss, mask)
results are kept (HeadResults), so re-tuning alpha or a target sparsity only reruns the
selection on the host:

* select(results, alpha): per head, sort the candidates by loss, start from the lowest-loss one
  and move to any candidate with loss <= alpha and strictly higher sparsity;
* select_target(results, target): per head, the lowest-loss candidate among those with sparsity
  >= target (the sparsest, lowest-loss candidate when none reaches the target).
"""
from dataclasses import dataclass

import numpy as np

from . import _lib, attention_fwd, dense_fwd, l2_distance, Workspace


@dataclass
class HeadResults:
    """Scores of every candidate of every head: loss and sparsity are float64 [heads, C]."""
    candidates: list          # [heads][C] stripe tuples
    loss: np.ndarray
    sparsity: np.ndarray


def score(q, k, v, grid, block, candidates, scale=None, stream=None):
    """HeadResults of candidates[h][c] for q, k, v bf16 [batch, heads, N, d] on the GPU.

    With a stream given, every step runs on it (allocations, library calls and the reductions
    whose results are read on the host); the caller orders q, k, v onto it."""
    import contextlib
    import torch
    b, h, n, d = q.shape
    n_cand = len(candidates[0])
    if len(candidates) != h or any(len(c) != n_cand for c in candidates):
        raise ValueError("candidates must list the same number of masks for every head")
    with (contextlib.nullcontext() if stream is None else torch.cuda.stream(stream)):
        full = dense_fwd(q, k, v, block, scale)
        o = torch.empty_like(q)
        ws = Workspace(b, h, grid, block, q.device)
        sq_err = torch.empty((n_cand, b, h), dtype=torch.float64, device=q.device)
        sq_ref = torch.empty((b, h), dtype=torch.float64, device=q.device)
        l2_ws = torch.empty(int(_lib.lib().psa_l2_workspace_size(b * h)), dtype=torch.uint8, device=q.device)
        kept = torch.empty((n_cand, h), dtype=torch.int64, device=q.device)
        for c in range(n_cand):
            params = [candidates[hh][c] for hh in range(h)]
            # the plan's per-row kept counts give the sparsity without another pass over the map
            _, per_row = attention_fwd(q, k, v, grid, block, params, scale, out=o, workspace=ws,
                                       return_kept_per_row=True)
            l2_distance(o, full, sq_err=sq_err[c], sq_ref=sq_ref, workspace=l2_ws)
            kept[c] = per_row.sum(dim=1)
        err = sq_err.sum(dim=1).cpu().numpy()             # [C, heads]: over batch elements
        ref = sq_ref.sum(dim=0).cpu().numpy()             # [heads]
        kept_n = kept.cpu().numpy()
    nb = -(-n // block)
    loss = np.sqrt(err / np.where(ref > 0, ref, 1.0)).T   # [heads, C]
    sparsity = 1.0 - kept_n.T.astype(np.float64) / float(nb * nb)
    return HeadResults([list(c) for c in candidates], loss, sparsity)


def select(results, alpha):
    """Candidate index per head under loss threshold alpha (Algorithm 3)."""
    out = []
    for loss, sp in zip(results.loss, results.sparsity):
        order = np.argsort(loss, kind="stable")
        qualified = order[loss[order] <= alpha]
        if len(qualified) == 0:
            out.append(int(order[0]))
            continue
        # the first qualified candidate (in loss order) of the highest sparsity; it replaces the
        # lowest-loss candidate only if it is strictly sparser
        top = sp[qualified].max()
        pick = int(qualified[np.argmax(sp[qualified] == top)])
        out.append(pick if sp[pick] > sp[order[0]] else int(order[0]))
    return out


def select_target(results, target):
    """Candidate index per head for a target sparsity (the dual interface)."""
    out = []
    for loss, sp in zip(results.loss, results.sparsity):
        ok = np.nonzero(sp >= target)[0]
        if len(ok) == 0:
            ok = np.nonzero(sp == sp.max())[0]
        out.append(int(ok[np.argmin(loss[ok])]))       # argmin returns the first of equal losses
    return out


def strategy(results, picks):
    """The mask strategy map: the chosen stripe tuple of every head."""
    return [results.candidates[h][i] for h, i in enumerate(picks)]
