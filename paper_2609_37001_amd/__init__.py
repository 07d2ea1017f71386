"""PSA (Parameterized Stripe Attention) block-sparse attention forward for MI355X (gfx950).

Thin torch-facing wrapper around the C ABI of ``libpsa.so`` (``include/psa.h``): tensors are
only checked for dtype, device and layout, then their device pointers and the current HIP
stream are handed to the library.  Every computation runs in the library's HIP kernels; there
is no CPU or PyTorch fallback.

    params = [(T_w, T_o, T_s, S_w, S_o, S_s), ...]          # one 6-tuple per head
    o = attention_fwd(q, k, v, grid=(F, H, W, n_text), block=128, params=params)
    o_dense = dense_fwd(q, k, v, block=128)
    ws = plan(params, grid, block, batch=1)                   # plan once ...
    o = run(q, k, v, grid, block, ws)                         # ... run many times
    bmap, per_row, per_head = build_blockmap(params, (F, H, W, n_text), block=128)

3D PSABlocks with 3D padding (the paper's layout; q, k, v permuted once, e.g. for a whole DiT):

    pb = (3, 8, 16)
    qb, kb, vb = (to_blocks(x, grid, pb) for x in (q, k, v))
    ob = attention_fwd_3d(qb, kb, vb, grid, pb, params, tile=128)
    o = from_blocks(ob, grid, pb)
"""
import contextlib
import math

from . import _lib
from ._lib import STRIDE_INF, PsaError  # noqa: F401

__all__ = ["STRIDE_INF", "PsaError", "num_blocks", "workspace_size", "build_blockmap",
           "attention_fwd", "attention_fwd_noalloc", "plan", "run", "dense_fwd", "dense_workspace_size", "Workspace", "library_path",
           "blocked_tokens", "to_blocks", "from_blocks", "build_blockmap_3d", "plan_3d", "run_3d",
           "attention_fwd_3d", "l2_distance"]


def library_path():
    return _lib.LIB_PATH


def _grid(grid):
    g = tuple(int(x) for x in grid)
    if len(g) == 3:
        g = g + (0,)
    if len(g) != 4:
        raise ValueError("grid is (frames, height, width[, n_text])")
    return _lib.grid_of(*g)


def num_blocks(grid, block):
    return int(_lib.lib().psa_num_blocks(_grid(grid), int(block)))


def workspace_size(batch, n_heads, grid, block):
    return int(_lib.lib().psa_workspace_size(int(batch), int(n_heads), _grid(grid), int(block)))


def _torch():
    import torch
    return torch


def _stream(stream, device):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes_void(stream.cuda_stream)


def _on(stream):
    """Context for the allocations and the library call of one binding function: with a stream
    given, it becomes torch's current stream, so the tensors the function allocates (outputs,
    workspaces) belong to that stream's memory pool and are not handed to other work while the
    library still uses them there.  The caller orders the inputs onto that stream."""
    return contextlib.nullcontext() if stream is None else _torch().cuda.stream(stream)


def ctypes_void(x):
    import ctypes
    return ctypes.c_void_p(int(x)) if x else None


def _ptr(t):
    return ctypes_void(t.data_ptr()) if t is not None else None


def _check_qkv(*ts):
    torch = _torch()
    ref = ts[0]
    for t in ts:
        if t.dtype != torch.bfloat16:
            raise TypeError("q, k, v must be bfloat16")
        if not t.is_cuda:
            raise ValueError("q, k, v must be GPU tensors")
        if not t.is_contiguous():
            raise ValueError("q, k, v must be contiguous [batch, heads, N, head_dim]")
        if t.dim() != 4 or t.shape != ref.shape:
            raise ValueError("q, k, v must share the shape [batch, heads, N, head_dim]")
        if t.device != ref.device:
            raise ValueError("q, k, v must be on one device")


class Workspace:
    """Device workspace for attention_fwd / plan / run (a byte tensor on the given device).

    After plan() it also records the sizes and parameters of the plan it holds."""

    def __init__(self, batch, n_heads, grid, block, device):
        torch = _torch()
        self.nbytes = workspace_size(batch, n_heads, grid, block)
        if self.nbytes == 0:
            raise ValueError("invalid sizes for a workspace")
        self.tensor = torch.empty(self.nbytes, dtype=torch.uint8, device=device)
        self.sizes = (int(batch), int(n_heads), tuple(int(x) for x in _grid_tuple(grid)), int(block))
        self.params = None


def _grid_tuple(grid):
    g = tuple(int(x) for x in grid)
    return g + (0,) if len(g) == 3 else g


def _check_tokens(n, grid):
    """The library sees raw pointers: a tensor shorter than the grid would be read past its end."""
    f, h, w, nt = _grid_tuple(grid)
    if n != f * h * w + nt:
        raise ValueError("tensors hold %d tokens, the grid %s has %d" % (n, (f, h, w, nt), f * h * w + nt))


def build_blockmap(params, grid, block, device=None, blockmap=True, per_row=True, per_head=True,
                   stream=None):
    """Block map of the stripe parameters on the device.

    Returns (map uint8 [heads, nb, nb] | None, kept_per_row int32 [heads, nb] | None,
    kept_per_head int64 [heads] | None)."""
    torch = _torch()
    device = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    heads = len(params)
    nb = num_blocks(grid, block)
    if nb < 0:
        raise ValueError("invalid grid or block")
    with torch.cuda.device(device), _on(stream):
        bm = torch.empty((heads, nb, nb), dtype=torch.uint8, device=device) if blockmap else None
        pr = torch.empty((heads, nb), dtype=torch.int32, device=device) if per_row else None
        ph = torch.empty((heads,), dtype=torch.int64, device=device) if per_head else None
        _lib.check(_lib.lib().psa_build_blockmap(_lib.stripes(params), heads, _grid(grid), int(block),
                                                 _ptr(bm), _ptr(pr), _ptr(ph), _stream(None, device)))
    return bm, pr, ph


def attention_fwd(q, k, v, grid, block, params, scale=None, out=None, return_lse=False,
                  workspace=None, return_kept_per_row=False, stream=None):
    """PSA block-sparse attention forward.  q, k, v: bf16 [batch, heads, N, head_dim], contiguous.

    Returns o (and lse float32 [batch, heads, N], kept_per_row int32 [heads, nb] if asked)."""
    torch = _torch()
    _check_qkv(q, k, v)
    b, h, n, d = q.shape
    if len(params) != h:
        raise ValueError("one stripe tuple per head is required")
    _check_tokens(n, grid)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    nb = num_blocks(grid, block)
    with torch.cuda.device(q.device), _on(stream):
        o = torch.empty_like(q) if out is None else out
        _check_qkv(q, o)
        lse = torch.empty((b, h, n), dtype=torch.float32, device=q.device) if return_lse else None
        kept = torch.empty((h, max(nb, 1)), dtype=torch.int32, device=q.device) if return_kept_per_row else None
        ws = workspace if workspace is not None else Workspace(b, h, grid, block, q.device)
        _lib.check(_lib.lib().psa_attention_fwd(
            _ptr(q), _ptr(k), _ptr(v), _ptr(o), b, h, d, _grid(grid), int(block),
            _lib.stripes(params), scale, _ptr(ws.tensor), ws.nbytes, _ptr(lse), _ptr(kept),
            _stream(None, q.device)))
    ws.sizes = (b, h, _grid_tuple(grid), int(block))
    ws.params = [tuple(int(x) for x in m) for m in params]
    res = (o,)
    if return_lse:
        res += (lse,)
    if return_kept_per_row:
        res += (kept,)
    return res[0] if len(res) == 1 else res


def attention_fwd_noalloc(q, k, v, grid, block, params, out, scale=None, lse=None, kept_per_row=None,
                          stream=None):
    """attention_fwd with the plan in the library's static device scratch
    (psa_attention_fwd_noalloc): neither the library nor this wrapper allocates, so the caller
    passes the output `out` (bf16 like q) and, if wanted, `lse` (float32 [batch, heads, N]) and
    `kept_per_row` (int32 [heads, nb]).  Calls that overlap in time on one GPU must not be made."""
    torch = _torch()
    _check_qkv(q, k, v)
    _check_qkv(q, out)
    b, h, n, d = q.shape
    if len(params) != h:
        raise ValueError("one stripe tuple per head is required")
    _check_tokens(n, grid)
    nb = num_blocks(grid, block)
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (b, h, n) or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous float32 tensor [batch, heads, N]")
    if kept_per_row is not None and (kept_per_row.dtype != torch.int32 or tuple(kept_per_row.shape) != (h, nb)
                                     or not kept_per_row.is_contiguous()):
        raise ValueError("kept_per_row must be a contiguous int32 tensor [heads, nb]")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    with torch.cuda.device(q.device):
        _lib.check(_lib.lib().psa_attention_fwd_noalloc(
            _ptr(q), _ptr(k), _ptr(v), _ptr(out), b, h, d, _grid(grid), int(block), _lib.stripes(params),
            scale, _ptr(lse), _ptr(kept_per_row), _stream(stream, q.device)))
    return out


def plan(params, grid, block, batch=1, device=None, workspace=None, return_kept_per_row=False,
         stream=None):
    """Plan of the sparse attention for these stripes and sizes (psa_attention_plan).

    Returns the Workspace holding it (and kept_per_row int32 [heads, nb] if asked)."""
    torch = _torch()
    device = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    h = len(params)
    nb = num_blocks(grid, block)
    with torch.cuda.device(device), _on(stream):
        ws = workspace if workspace is not None else Workspace(batch, h, grid, block, device)
        kept = torch.empty((h, max(nb, 1)), dtype=torch.int32, device=device) if return_kept_per_row else None
        _lib.check(_lib.lib().psa_attention_plan(int(batch), h, _grid(grid), int(block),
                                                 _lib.stripes(params), _ptr(ws.tensor), ws.nbytes,
                                                 _ptr(kept), _stream(None, device)))
    ws.sizes = (int(batch), h, _grid_tuple(grid), int(block))
    ws.params = [tuple(int(x) for x in m) for m in params]
    return (ws, kept) if return_kept_per_row else ws


def run(q, k, v, grid, block, workspace, scale=None, out=None, return_lse=False, stream=None):
    """Sparse attention over a planned workspace (psa_attention_run)."""
    torch = _torch()
    _check_qkv(q, k, v)
    b, h, n, d = q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    _check_tokens(n, grid)
    ws = workspace
    if ws.params is None:
        raise ValueError("the workspace holds no plan: call plan() or attention_fwd() first")
    if ws.sizes != (b, h, _grid_tuple(grid), int(block)):
        raise ValueError("the workspace was planned for (batch, heads, grid, block) = %s, not %s"
                         % (ws.sizes, (b, h, _grid_tuple(grid), int(block))))
    with torch.cuda.device(q.device), _on(stream):
        o = torch.empty_like(q) if out is None else out
        _check_qkv(q, o)
        lse = torch.empty((b, h, n), dtype=torch.float32, device=q.device) if return_lse else None
        _lib.check(_lib.lib().psa_attention_run(
            _ptr(q), _ptr(k), _ptr(v), _ptr(o), b, h, d, _grid(grid), int(block), scale,
            _ptr(ws.tensor), ws.nbytes, _ptr(lse), _stream(None, q.device)))
    return (o, lse) if return_lse else o


def dense_workspace_size():
    return int(_lib.lib().psa_dense_workspace_size())


def dense_fwd(q, k, v, block, scale=None, out=None, return_lse=False, stream=None, workspace=None,
              balanced=True):
    """Dense attention forward with the same tile engine (the speedup baseline).

    balanced (default): a persistent grid takes the work items from per-XCD queues in a small
    workspace -- `workspace`, a uint8 device tensor of dense_workspace_size() bytes, or a fresh
    one -- so that XCDs holding different clocks finish together.  balanced=False runs the fixed
    grid (an equal share per XCD, no workspace).  Same output bits either way."""
    torch = _torch()
    _check_qkv(q, k, v)
    b, h, n, d = q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    with torch.cuda.device(q.device), _on(stream):
        o = torch.empty_like(q) if out is None else out
        _check_qkv(q, o)
        lse = torch.empty((b, h, n), dtype=torch.float32, device=q.device) if return_lse else None
        if not balanced:
            workspace = None
        elif workspace is None:
            workspace = torch.empty(dense_workspace_size(), dtype=torch.uint8, device=q.device)
        ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        _lib.check(_lib.lib().psa_dense_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), b, h, d, n, int(block),
                                            scale, _ptr(lse), _ptr(workspace), ws_bytes,
                                            _stream(None, q.device)))
    return (o, lse) if return_lse else o


# ---------------------------------------------------------------------------------------------
# 3D PSABlocks with 3D padding (include/psa.h, second part).
# ---------------------------------------------------------------------------------------------

def blocked_tokens(grid, pb):
    """Positions of the PSABlock-centric layout (T' H' W' bt bh bw + n_text)."""
    return int(_lib.lib().psa_blocked_tokens(_grid(grid), _lib.block3d_of(pb)))


def _layout(src, grid, pb, out, stream, to):
    torch = _torch()
    if src.dtype != torch.bfloat16 or not src.is_cuda or not src.is_contiguous() or src.dim() != 4:
        raise ValueError("expected a contiguous bf16 GPU tensor [batch, heads, tokens, head_dim]")
    b, h, n, d = src.shape
    g = _grid_tuple(grid)
    n_orig = g[0] * g[1] * g[2] + g[3]
    n_blk = blocked_tokens(grid, pb)
    if n_blk < 0:
        raise ValueError("invalid grid or PSABlock shape")
    if n != (n_orig if to else n_blk):
        raise ValueError("tensor has %d tokens, the %s layout has %d" % (n, "original" if to else "blocked",
                                                                        n_orig if to else n_blk))
    shape = (b, h, n_blk if to else n_orig, d)
    fn = _lib.lib().psa_to_blocks if to else _lib.lib().psa_from_blocks
    with torch.cuda.device(src.device), _on(stream):
        dst = torch.empty(shape, dtype=src.dtype, device=src.device) if out is None else out
        if tuple(dst.shape) != shape or not dst.is_contiguous() or dst.dtype != src.dtype:
            raise ValueError("out must be a contiguous bf16 tensor of shape %s" % (shape,))
        _lib.check(fn(_ptr(src), _ptr(dst), b * h, d, _grid(grid), _lib.block3d_of(pb),
                      _stream(None, src.device)))
    return dst


def to_blocks(x, grid, pb, out=None, stream=None):
    """[batch, heads, F*H*W + n_text, d] -> PSABlock-centric layout (psa_to_blocks)."""
    return _layout(x, grid, pb, out, stream, True)


def from_blocks(xb, grid, pb, out=None, stream=None):
    """PSABlock-centric layout -> [batch, heads, F*H*W + n_text, d] (psa_from_blocks)."""
    return _layout(xb, grid, pb, out, stream, False)


def build_blockmap_3d(params, grid, pb, device=None, blockmap=True, per_row=True, per_head=True,
                      stream=None):
    """PSABlock-level map: (uint8 [heads, G, G] | None, int32 [heads, G] | None,
    int64 [heads] | None), G = T'H'W' (+1 for the text group)."""
    torch = _torch()
    device = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    g = _grid_tuple(grid)
    (tp, hp, wp) = (-(-g[0] // pb[0]), -(-g[1] // pb[1]), -(-g[2] // pb[2]))
    groups = tp * hp * wp + (1 if g[3] > 0 else 0)
    heads = len(params)
    with torch.cuda.device(device), _on(stream):
        bm = torch.empty((heads, groups, groups), dtype=torch.uint8, device=device) if blockmap else None
        pr = torch.empty((heads, groups), dtype=torch.int32, device=device) if per_row else None
        ph = torch.empty((heads,), dtype=torch.int64, device=device) if per_head else None
        _lib.check(_lib.lib().psa_build_blockmap_3d(_lib.stripes(params), heads, _grid(grid),
                                                    _lib.block3d_of(pb), _ptr(bm), _ptr(pr), _ptr(ph),
                                                    _stream(None, device)))
    return bm, pr, ph


class Workspace3d(Workspace):
    """Workspace of plan_3d / run_3d."""

    def __init__(self, batch, n_heads, grid, pb, tile, device):
        torch = _torch()
        self.nbytes = int(_lib.lib().psa_workspace_size_3d(int(batch), int(n_heads), _grid(grid),
                                                            _lib.block3d_of(pb), int(tile)))
        if self.nbytes == 0:
            raise ValueError("invalid sizes for a 3D workspace")
        self.tensor = torch.empty(self.nbytes, dtype=torch.uint8, device=device)
        self.sizes = (int(batch), int(n_heads), _grid_tuple(grid), tuple(int(x) for x in pb), int(tile))
        self.params = None


def plan_3d(params, grid, pb, tile=128, batch=1, device=None, workspace=None,
            return_kept_per_tile=False, stream=None):
    """Plan over the PSABlock-centric layout (psa_attention_plan_3d)."""
    torch = _torch()
    device = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    h = len(params)
    n_tiles = -(-blocked_tokens(grid, pb) // int(tile))
    with torch.cuda.device(device), _on(stream):
        ws = workspace if workspace is not None else Workspace3d(batch, h, grid, pb, tile, device)
        kept = torch.empty((h, n_tiles), dtype=torch.int32, device=device) if return_kept_per_tile else None
        _lib.check(_lib.lib().psa_attention_plan_3d(int(batch), h, _grid(grid), _lib.block3d_of(pb),
                                                    int(tile), _lib.stripes(params), _ptr(ws.tensor),
                                                    ws.nbytes, _ptr(kept), _stream(None, device)))
    ws.sizes = (int(batch), h, _grid_tuple(grid), tuple(int(x) for x in pb), int(tile))
    ws.params = [tuple(int(x) for x in m) for m in params]
    return (ws, kept) if return_kept_per_tile else ws


def run_3d(q, k, v, grid, pb, tile, workspace, scale=None, out=None, return_lse=False, stream=None):
    """Sparse attention over a 3D plan; q, k, v, o in the PSABlock-centric layout."""
    torch = _torch()
    _check_qkv(q, k, v)
    b, h, n, d = q.shape
    if n != blocked_tokens(grid, pb):
        raise ValueError("q, k, v must be in the PSABlock-centric layout (%d tokens)" % blocked_tokens(grid, pb))
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = workspace
    if ws.params is None:
        raise ValueError("the workspace holds no plan: call plan_3d() first")
    if ws.sizes != (b, h, _grid_tuple(grid), tuple(int(x) for x in pb), int(tile)):
        raise ValueError("the workspace was planned for %s, not %s"
                         % (ws.sizes, (b, h, _grid_tuple(grid), tuple(pb), int(tile))))
    with torch.cuda.device(q.device), _on(stream):
        o = torch.empty_like(q) if out is None else out
        _check_qkv(q, o)
        lse = torch.empty((b, h, n), dtype=torch.float32, device=q.device) if return_lse else None
        _lib.check(_lib.lib().psa_attention_run_3d(
            _ptr(q), _ptr(k), _ptr(v), _ptr(o), b, h, d, _grid(grid), _lib.block3d_of(pb), int(tile),
            scale, _ptr(ws.tensor), ws.nbytes, _ptr(lse), _stream(None, q.device)))
    return (o, lse) if return_lse else o


def attention_fwd_3d(q, k, v, grid, pb, params, tile=128, scale=None, out=None, return_lse=False,
                     workspace=None, stream=None):
    """plan_3d then run_3d (q, k, v in the PSABlock-centric layout)."""
    b = q.shape[0]
    ws = plan_3d(params, grid, pb, tile, batch=b, device=q.device, workspace=workspace, stream=stream)
    return run_3d(q, k, v, grid, pb, tile, ws, scale, out, return_lse, stream)


# ---------------------------------------------------------------------------------------------
# PSA-Search scoring (include/psa.h, third part); the search itself is in .search.
# ---------------------------------------------------------------------------------------------

def l2_distance(o, ref, sq_err=None, sq_ref=None, workspace=None, stream=None):
    """Per (batch, head) sums of (o - ref)^2 and ref^2 (float64 [batch, heads] each)."""
    torch = _torch()
    _check_qkv(o, ref)
    b, h, n, d = o.shape
    nbytes = int(_lib.lib().psa_l2_workspace_size(b * h))
    with torch.cuda.device(o.device), _on(stream):
        err = torch.empty((b, h), dtype=torch.float64, device=o.device) if sq_err is None else sq_err
        rref = torch.empty((b, h), dtype=torch.float64, device=o.device) if sq_ref is None else sq_ref
        for t in (err, rref):
            if t.dtype != torch.float64 or t.numel() != b * h or not t.is_contiguous():
                raise ValueError("sq_err and sq_ref must be contiguous float64 tensors of %d elements" % (b * h))
        ws = torch.empty(nbytes, dtype=torch.uint8, device=o.device) if workspace is None else workspace
        if ws.numel() < nbytes:
            raise ValueError("l2 workspace needs %d bytes" % nbytes)
        _lib.check(_lib.lib().psa_l2_distance(_ptr(o), _ptr(ref), b * h, n, d, _ptr(err), _ptr(rref),
                                              _ptr(ws), ws.numel(), _stream(None, o.device)))
    return err, rref
