"""C ABI of libpsa.so on the CPU: the library loads, exports every call of include/psa.h, and
rejects invalid arguments with the documented status codes before touching the GPU."""
import ctypes
import os
import re

import pytest

from paper_2609_37001_amd import _lib
import paper_2609_37001_amd as psa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INF = _lib.STRIDE_INF


def header_functions():
    text = open(os.path.join(ROOT, "include", "psa.h")).read()
    return sorted(set(re.findall(r"^\s*(?:const char\*|int32_t|int64_t|size_t|psa_status_t)\s+(psa_\w+)\(", text, re.M)))


def test_header_declares_the_boundary():
    assert header_functions() == sorted(_lib.EXPORTS)


def test_library_exports_every_header_function():
    L = _lib.lib()
    for name in header_functions():
        assert hasattr(L, name), name


def test_num_blocks_and_workspace():
    L = _lib.lib()
    assert L.psa_num_blocks(_lib.grid_of(21, 45, 80), 128) == 591
    assert L.psa_num_blocks(_lib.grid_of(33, 45, 80, 256), 128) == 931
    assert L.psa_num_blocks(_lib.grid_of(4, 16, 16), 64) == 16
    assert L.psa_num_blocks(_lib.grid_of(2, 3, 4, 3), 5) == 6
    assert L.psa_num_blocks(_lib.grid_of(0, 3, 4), 5) == -1
    assert L.psa_num_blocks(_lib.grid_of(2, 3, 4), 0) == -1
    assert L.psa_num_blocks(_lib.grid_of(2, 3, 4, -1), 4) == -1
    ws = psa.workspace_size(1, 40, (21, 45, 80), 128)
    assert ws >= 2 * 4 * 40 * 591 and ws % 256 == 0
    assert psa.workspace_size(0, 40, (21, 45, 80), 128) == 0


def _attn(q=1, k=1, v=1, o=1, batch=1, heads=1, d=128, grid=(2, 8, 8, 0), block=128, params=None,
          ws=1, wsb=1 << 20, scale=0.1):
    L = _lib.lib()
    params = [(1, 0, INF, 1, 0, INF)] * heads if params is None else params
    vp = lambda x: ctypes.c_void_p(x) if x else None
    return L.psa_attention_fwd(vp(q * 256), vp(k * 256), vp(v * 256), vp(o * 256), batch, heads, d,
                               _lib.grid_of(*grid), block, _lib.stripes(params), scale, vp(ws * 256), wsb,
                               None, None, None)


def test_attention_validation_codes():
    assert _attn(q=0) == _lib.PSA_ERR_INVALID
    assert _attn(o=0) == _lib.PSA_ERR_INVALID
    assert _attn(batch=0) == _lib.PSA_ERR_INVALID
    assert _attn(d=96) == _lib.PSA_ERR_UNSUPPORTED
    assert _attn(block=32) == _lib.PSA_ERR_UNSUPPORTED
    assert _attn(grid=(0, 8, 8, 0)) == _lib.PSA_ERR_INVALID
    assert _attn(params=[(0, 0, 1, 1, 0, 1)]) == _lib.PSA_ERR_INVALID
    assert _attn(params=[(1, 0, 0, 1, 0, 1)]) == _lib.PSA_ERR_INVALID
    assert _attn(params=[(1, 1 << 25, 1, 1, 0, 1)]) == _lib.PSA_ERR_INVALID
    assert _attn(ws=0) == _lib.PSA_ERR_WORKSPACE
    assert _attn(wsb=16) == _lib.PSA_ERR_WORKSPACE
    assert _attn(grid=(100, 100, 128, 0)) == _lib.PSA_ERR_UNSUPPORTED        # 10000 blocks
    assert _attn(batch=1025) == _lib.PSA_ERR_UNSUPPORTED


def _noalloc(q=1, o=1, batch=1, heads=1, d=128, grid=(2, 8, 8, 0), block=128, params=None, lse=0, kept=0):
    L = _lib.lib()
    params = [(1, 0, INF, 1, 0, INF)] * heads if params is None else params
    vp = lambda x: ctypes.c_void_p(x) if x else None
    return L.psa_attention_fwd_noalloc(vp(q * 256), vp(256), vp(256), vp(o * 256), batch, heads, d,
                                       _lib.grid_of(*grid), block, _lib.stripes(params), 0.1, vp(lse), vp(kept),
                                       None)


def test_noalloc_validation_before_any_hip_call():
    """Invalid arguments and sizes whose plan exceeds the static scratch are rejected before the
    entry point touches the GPU (this container has none)."""
    assert _noalloc(q=0) == _lib.PSA_ERR_INVALID
    assert _noalloc(d=96) == _lib.PSA_ERR_UNSUPPORTED
    assert _noalloc(params=[(1, 0, 0, 1, 0, 1)]) == _lib.PSA_ERR_INVALID
    assert _noalloc(grid=(0, 8, 8, 0)) == _lib.PSA_ERR_INVALID
    assert _noalloc(lse=2) == _lib.PSA_ERR_INVALID                               # misaligned float
    assert _noalloc(kept=3) == _lib.PSA_ERR_INVALID                              # misaligned int32
    assert _noalloc(grid=(100, 100, 128, 0)) == _lib.PSA_ERR_UNSUPPORTED           # 10000 blocks
    # 1000 heads x 7936 blocks: the plan needs far more than the scratch holds
    big = (62, 128, 128, 0)
    need = psa.workspace_size(1, 1000, big, 128)
    assert need > _lib.NOALLOC_SCRATCH_BYTES
    assert _noalloc(heads=1000, grid=big) == _lib.PSA_ERR_WORKSPACE
    assert b"static scratch" in _lib.lib().psa_last_error()
    # 40 heads of the Wan 2.1 14B grid fit
    assert psa.workspace_size(1, 40, (21, 45, 80), 128) < _lib.NOALLOC_SCRATCH_BYTES


def test_error_messages():
    L = _lib.lib()
    assert _attn(params=[(1, 0, 0, 1, 0, 1)]) == _lib.PSA_ERR_INVALID
    assert b"stride" in L.psa_last_error()
    for s in range(5):
        assert L.psa_status_string(s).startswith(b"PSA_")
    with pytest.raises(_lib.PsaError) as e:
        _lib.check(_attn(d=80))
    assert e.value.status == _lib.PSA_ERR_UNSUPPORTED


def test_dense_validation_codes():
    L = _lib.lib()
    vp = ctypes.c_void_p
    args = lambda n, d, blk, q=256, ws=None, wsb=0: (vp(q), vp(256), vp(256), vp(256), 1, 1, d, n, blk, 0.1,
                                                     None, vp(ws), wsb, None)
    assert L.psa_dense_fwd(*args(0, 128, 128)) == _lib.PSA_ERR_INVALID
    assert L.psa_dense_fwd(*args(100, 48, 128)) == _lib.PSA_ERR_UNSUPPORTED
    assert L.psa_dense_fwd(*args(100, 64, 16)) == _lib.PSA_ERR_UNSUPPORTED
    assert L.psa_dense_fwd(*args(100, 64, 64, q=0)) == _lib.PSA_ERR_INVALID
    need = L.psa_dense_workspace_size()
    assert need >= 8 * 4 and need % 256 == 0
    assert L.psa_dense_fwd(*args(100, 64, 64, ws=512, wsb=need - 1)) == _lib.PSA_ERR_WORKSPACE
    assert L.psa_dense_fwd(*args(100, 64, 64, ws=512 + 128, wsb=need)) == _lib.PSA_ERR_WORKSPACE
    assert b"aligned" in L.psa_last_error()


def test_blockmap_validation_codes():
    L = _lib.lib()
    bad = L.psa_build_blockmap(_lib.stripes([(1, 0, 1, 0, 0, 1)]), 1, _lib.grid_of(2, 2, 2), 1,
                               None, None, None, None)
    assert bad == _lib.PSA_ERR_INVALID
    assert L.psa_build_blockmap(_lib.stripes([(1, 0, 1, 1, 0, 1)]), 0, _lib.grid_of(2, 2, 2), 1,
                                None, None, None, None) == _lib.PSA_ERR_INVALID
    assert L.psa_build_blockmap(_lib.stripes([(1, 0, 1, 1, 0, 1)]), 1, _lib.grid_of(2, 2, 0), 1,
                                None, None, None, None) == _lib.PSA_ERR_INVALID
    assert L.psa_build_blockmap(None, 1, _lib.grid_of(2, 2, 2), 1, None, None, None, None) == _lib.PSA_ERR_INVALID


def _plan(batch=1, heads=1, grid=(2, 8, 8, 0), block=128, params=None, ws=1, wsb=1 << 20):
    L = _lib.lib()
    params = [(1, 0, INF, 1, 0, INF)] * heads if params is None else params
    vp = lambda x: ctypes.c_void_p(x) if x else None
    return L.psa_attention_plan(batch, heads, _lib.grid_of(*grid), block, _lib.stripes(params),
                                vp(ws * 256), wsb, None, None)


def _run(q=1, o=1, batch=1, heads=1, d=128, grid=(2, 8, 8, 0), block=128, ws=1, wsb=1 << 20):
    L = _lib.lib()
    vp = lambda x: ctypes.c_void_p(x) if x else None
    return L.psa_attention_run(vp(q * 256), vp(256), vp(256), vp(o * 256), batch, heads, d,
                               _lib.grid_of(*grid), block, 0.1, vp(ws * 256), wsb, None, None)


def test_plan_validation_codes():
    assert _plan(batch=0) == _lib.PSA_ERR_INVALID
    assert _plan(heads=0, params=[(1, 0, 1, 1, 0, 1)]) == _lib.PSA_ERR_INVALID
    assert _plan(block=32) == _lib.PSA_ERR_UNSUPPORTED
    assert _plan(grid=(2, 8, 0, 0)) == _lib.PSA_ERR_INVALID
    assert _plan(params=[(1, 0, 1, 1, 0, 0)]) == _lib.PSA_ERR_INVALID
    assert _plan(ws=0) == _lib.PSA_ERR_WORKSPACE
    assert _plan(wsb=8) == _lib.PSA_ERR_WORKSPACE
    assert _plan(ws=1, wsb=1 << 20, grid=(100, 100, 128, 0)) == _lib.PSA_ERR_UNSUPPORTED
    assert _plan(batch=33, heads=32, params=[(1, 0, 1, 1, 0, 1)] * 32) == _lib.PSA_ERR_UNSUPPORTED


def test_run_validation_codes():
    assert _run(q=0) == _lib.PSA_ERR_INVALID
    assert _run(o=0) == _lib.PSA_ERR_INVALID
    assert _run(d=96) == _lib.PSA_ERR_UNSUPPORTED
    assert _run(block=16) == _lib.PSA_ERR_UNSUPPORTED
    assert _run(heads=0) == _lib.PSA_ERR_INVALID
    assert _run(ws=0) == _lib.PSA_ERR_WORKSPACE
    assert _run(wsb=100) == _lib.PSA_ERR_WORKSPACE



def _b3(t, h, w):
    return _lib.block3d_of((t, h, w))


def test_blocked_tokens_and_3d_workspace():
    L = _lib.lib()
    assert L.psa_blocked_tokens(_lib.grid_of(21, 45, 80), _b3(3, 8, 16)) == 21 * 48 * 80
    assert L.psa_blocked_tokens(_lib.grid_of(33, 45, 80, 256), _b3(3, 8, 16)) == 33 * 48 * 80 + 256
    assert L.psa_blocked_tokens(_lib.grid_of(30, 48, 80), _b3(6, 8, 8)) == 30 * 48 * 80
    assert L.psa_blocked_tokens(_lib.grid_of(3, 5, 7, 2), _b3(2, 2, 3)) == 4 * 6 * 9 + 2
    assert L.psa_blocked_tokens(_lib.grid_of(3, 5, 7), _b3(0, 2, 3)) == -1
    assert L.psa_blocked_tokens(_lib.grid_of(0, 5, 7), _b3(1, 2, 3)) == -1
    ws = L.psa_workspace_size_3d(1, 40, _lib.grid_of(21, 45, 80), _b3(3, 8, 16), 128)
    assert ws >= 16 * (21 * 48 * 80 // 128) and ws % 256 == 0
    assert L.psa_workspace_size_3d(1, 40, _lib.grid_of(21, 45, 80), _b3(3, 8, 5), 128) == 0   # 120 % 128
    assert L.psa_workspace_size_3d(1, 40, _lib.grid_of(21, 45, 80), _b3(3, 8, 16), 32) == 0


def test_layout_validation_codes():
    L = _lib.lib()
    vp = ctypes.c_void_p
    g = _lib.grid_of(3, 5, 7, 2)
    assert L.psa_to_blocks(None, vp(256), 1, 128, g, _b3(2, 2, 2), None) == _lib.PSA_ERR_INVALID
    assert L.psa_from_blocks(vp(256), None, 1, 128, g, _b3(2, 2, 2), None) == _lib.PSA_ERR_INVALID
    assert L.psa_to_blocks(vp(256), vp(256), 0, 128, g, _b3(2, 2, 2), None) == _lib.PSA_ERR_INVALID
    assert L.psa_to_blocks(vp(256), vp(256), 1, 96, g, _b3(2, 2, 2), None) == _lib.PSA_ERR_UNSUPPORTED
    assert L.psa_to_blocks(vp(256), vp(256), 1, 64, g, _b3(2, 0, 2), None) == _lib.PSA_ERR_INVALID
    assert L.psa_to_blocks(vp(256), vp(256), 70000, 64, g, _b3(2, 2, 2), None) == _lib.PSA_ERR_UNSUPPORTED
    assert L.psa_build_blockmap_3d(_lib.stripes([(1, 0, 0, 1, 0, 1)]), 1, g, _b3(2, 2, 2), None, None,
                                   None, None) == _lib.PSA_ERR_INVALID


def test_plan_and_run_3d_validation_codes():
    L = _lib.lib()
    vp = lambda x: ctypes.c_void_p(x) if x else None
    g = _lib.grid_of(4, 10, 20, 0)
    ok = [(1, 0, INF, 1, 0, INF)]

    def plan(pb=(2, 4, 16), tile=128, params=ok, ws=256, wsb=1 << 20, batch=1):
        return L.psa_attention_plan_3d(batch, len(params), g, _b3(*pb), tile, _lib.stripes(params),
                                       vp(ws), wsb, None, None)

    assert plan(tile=32) == _lib.PSA_ERR_UNSUPPORTED
    assert plan(pb=(3, 8, 5)) == _lib.PSA_ERR_UNSUPPORTED          # 120 positions: not whole tiles
    assert plan(pb=(1, 0, 16)) == _lib.PSA_ERR_INVALID
    assert plan(params=[(1, 0, 1, 1, 0, 0)]) == _lib.PSA_ERR_INVALID
    assert plan(ws=0) == _lib.PSA_ERR_WORKSPACE
    assert plan(wsb=64) == _lib.PSA_ERR_WORKSPACE
    assert plan(batch=0) == _lib.PSA_ERR_INVALID

    def run(q=256, d=128, tile=128, pb=(2, 4, 16)):
        return L.psa_attention_run_3d(vp(q), vp(256), vp(256), vp(256), 1, 1, d, g, _b3(*pb), tile,
                                      0.1, vp(256), 1 << 20, None, None)

    assert run(q=0) == _lib.PSA_ERR_INVALID
    assert run(d=80) == _lib.PSA_ERR_UNSUPPORTED
    assert run(tile=96) == _lib.PSA_ERR_UNSUPPORTED
    assert run(pb=(1, 3, 5)) == _lib.PSA_ERR_UNSUPPORTED


def test_misaligned_pointers_are_rejected():
    """The kernels move 16-byte vectors: a misaligned tensor is an argument error, checked before
    anything is enqueued (no GPU is needed to see it)."""
    L = _lib.lib()
    vp = lambda x: ctypes.c_void_p(x) if x else None
    params = _lib.stripes([(1, 0, INF, 1, 0, INF)])
    g = _lib.grid_of(2, 8, 8, 0)
    fwd = lambda q=256, k=256, v=256, o=256, lse=None, kept=None: L.psa_attention_fwd(
        vp(q), vp(k), vp(v), vp(o), 1, 1, 128, g, 128, params, 0.1, vp(256), 1 << 20, vp(lse), vp(kept), None)
    assert fwd(q=256 + 8) == _lib.PSA_ERR_INVALID
    assert fwd(k=256 + 2) == _lib.PSA_ERR_INVALID
    assert fwd(v=256 + 4) == _lib.PSA_ERR_INVALID
    assert fwd(o=256 + 12) == _lib.PSA_ERR_INVALID
    assert fwd(lse=256 + 2) == _lib.PSA_ERR_INVALID
    assert b"aligned" in L.psa_last_error()
    assert fwd(kept=256 + 1) == _lib.PSA_ERR_INVALID
    run = lambda q=256, o=256, lse=None: L.psa_attention_run(vp(q), vp(256), vp(256), vp(o), 1, 1, 128, g, 128,
                                                             0.1, vp(256), 1 << 20, vp(lse), None)
    assert run(q=264) == _lib.PSA_ERR_INVALID
    assert run(o=258) == _lib.PSA_ERR_INVALID
    assert run(lse=257) == _lib.PSA_ERR_INVALID
    dense = lambda q=256, lse=None: L.psa_dense_fwd(vp(q), vp(256), vp(256), vp(256), 1, 1, 128, 256, 128,
                                                    0.1, vp(lse), None, 0, None)
    assert dense(q=264) == _lib.PSA_ERR_INVALID
    assert dense(lse=258) == _lib.PSA_ERR_INVALID
    b3 = _b3(2, 4, 16)
    g3 = _lib.grid_of(4, 10, 20, 0)
    assert L.psa_attention_run_3d(vp(256), vp(256), vp(264), vp(256), 1, 1, 128, g3, b3, 128, 0.1, vp(256),
                                  1 << 20, None, None) == _lib.PSA_ERR_INVALID
    assert L.psa_to_blocks(vp(264), vp(256), 1, 128, g3, b3, None) == _lib.PSA_ERR_INVALID
    assert L.psa_from_blocks(vp(256), vp(260), 1, 128, g3, b3, None) == _lib.PSA_ERR_INVALID
    assert L.psa_build_blockmap(params, 1, g, 128, None, vp(258), None, None) == _lib.PSA_ERR_INVALID
    assert L.psa_build_blockmap(params, 1, g, 128, None, None, vp(260), None) == _lib.PSA_ERR_INVALID
    assert L.psa_build_blockmap_3d(params, 1, g3, b3, None, None, vp(260), None) == _lib.PSA_ERR_INVALID
    assert L.psa_attention_plan(1, 1, g, 128, params, vp(256), 1 << 20, vp(258), None) == _lib.PSA_ERR_INVALID
    assert L.psa_attention_plan_3d(1, 1, g3, b3, 128, params, vp(256), 1 << 20, vp(258),
                                   None) == _lib.PSA_ERR_INVALID
    l2 = lambda o=256, err=512, ws=1024: L.psa_l2_distance(vp(o), vp(256), 1, 64, 128, vp(err), None, vp(ws),
                                                           4096, None)
    assert l2(o=264) == _lib.PSA_ERR_INVALID
    assert l2(err=516) == _lib.PSA_ERR_INVALID
    assert l2(ws=1028) == _lib.PSA_ERR_WORKSPACE
