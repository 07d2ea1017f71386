"""ctypes binding of libpsa.so (include/psa.h).  Argument marshalling only: every step of the
attention path runs in the HIP kernels of the library; torch supplies device memory and streams.

The library is loaded from this package directory; if it is missing the import of the binding
functions raises, there is no fallback.
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
# PSA_LIBRARY selects another build of the library (the host-sanitized one of build.py --asan).
LIB_PATH = os.environ.get("PSA_LIBRARY") or os.path.join(PKG, "libpsa.so")

STRIDE_INF = 0x7FFFFFFF
MAX_OFFSET = 1 << 24
MAX_BLOCKS = 7936
MAX_BATCH_HEADS = 1024
NOALLOC_SCRATCH_BYTES = 16 << 20

PSA_OK = 0
PSA_ERR_INVALID = 1
PSA_ERR_UNSUPPORTED = 2
PSA_ERR_WORKSPACE = 3
PSA_ERR_HIP = 4

EXPORTS = ("psa_num_blocks", "psa_workspace_size", "psa_build_blockmap", "psa_attention_plan",
           "psa_attention_run", "psa_attention_fwd", "psa_attention_fwd_noalloc", "psa_dense_workspace_size", "psa_dense_fwd",
           "psa_blocked_tokens",
           "psa_to_blocks", "psa_from_blocks", "psa_build_blockmap_3d", "psa_workspace_size_3d",
           "psa_attention_plan_3d", "psa_attention_run_3d", "psa_l2_workspace_size", "psa_l2_distance",
           "psa_status_string", "psa_last_error")


class Stripe(ctypes.Structure):
    _fields_ = [("t_w", ctypes.c_int32), ("t_o", ctypes.c_int32), ("t_s", ctypes.c_int32),
                ("s_w", ctypes.c_int32), ("s_o", ctypes.c_int32), ("s_s", ctypes.c_int32)]


class Grid(ctypes.Structure):
    _fields_ = [("frames", ctypes.c_int32), ("height", ctypes.c_int32),
                ("width", ctypes.c_int32), ("n_text", ctypes.c_int32)]


class Block3d(ctypes.Structure):
    _fields_ = [("t", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32)]


class PsaError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__("%s (%s)" % (detail, _status_name(status)))
        self.status = status


_STATUS = {0: "PSA_OK", 1: "PSA_ERR_INVALID", 2: "PSA_ERR_UNSUPPORTED", 3: "PSA_ERR_WORKSPACE",
           4: "PSA_ERR_HIP"}


def _status_name(s):
    return _STATUS.get(s, str(s))


_lib = None


def lib():
    """The loaded libpsa.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libpsa.so is not built: run `python -m paper_2609_37001_amd.build`")
        # torch ships its own HIP runtime under the soname libamdhip64.so.7; whichever copy is
        # loaded first serves the whole process.  Loading torch first makes the library bind to
        # the runtime that owns the tensors and streams it is handed.
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.psa_num_blocks.argtypes = [Grid, i32]
        L.psa_num_blocks.restype = i32
        L.psa_workspace_size.argtypes = [i32, i32, Grid, i32]
        L.psa_workspace_size.restype = sz
        L.psa_build_blockmap.argtypes = [ctypes.POINTER(Stripe), i32, Grid, i32, vp, vp, vp, vp]
        L.psa_build_blockmap.restype = ctypes.c_int
        L.psa_attention_plan.argtypes = [i32, i32, Grid, i32, ctypes.POINTER(Stripe), vp, sz, vp, vp]
        L.psa_attention_plan.restype = ctypes.c_int
        L.psa_attention_run.argtypes = [vp, vp, vp, vp, i32, i32, i32, Grid, i32, ctypes.c_float, vp,
                                        sz, vp, vp]
        L.psa_attention_run.restype = ctypes.c_int
        L.psa_attention_fwd.argtypes = [vp, vp, vp, vp, i32, i32, i32, Grid, i32,
                                        ctypes.POINTER(Stripe), ctypes.c_float, vp, sz, vp, vp, vp]
        L.psa_attention_fwd.restype = ctypes.c_int
        L.psa_attention_fwd_noalloc.argtypes = [vp, vp, vp, vp, i32, i32, i32, Grid, i32,
                                                ctypes.POINTER(Stripe), ctypes.c_float, vp, vp, vp]
        L.psa_attention_fwd_noalloc.restype = ctypes.c_int
        L.psa_dense_workspace_size.argtypes = []
        L.psa_dense_workspace_size.restype = sz
        L.psa_dense_fwd.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, ctypes.c_float, vp, vp, sz,
                                    vp]
        L.psa_dense_fwd.restype = ctypes.c_int
        L.psa_blocked_tokens.argtypes = [Grid, Block3d]
        L.psa_blocked_tokens.restype = i64
        for name in ("psa_to_blocks", "psa_from_blocks"):
            getattr(L, name).argtypes = [vp, vp, i32, i32, Grid, Block3d, vp]
            getattr(L, name).restype = ctypes.c_int
        L.psa_build_blockmap_3d.argtypes = [ctypes.POINTER(Stripe), i32, Grid, Block3d, vp, vp, vp, vp]
        L.psa_build_blockmap_3d.restype = ctypes.c_int
        L.psa_workspace_size_3d.argtypes = [i32, i32, Grid, Block3d, i32]
        L.psa_workspace_size_3d.restype = sz
        L.psa_attention_plan_3d.argtypes = [i32, i32, Grid, Block3d, i32, ctypes.POINTER(Stripe), vp, sz,
                                            vp, vp]
        L.psa_attention_plan_3d.restype = ctypes.c_int
        L.psa_attention_run_3d.argtypes = [vp, vp, vp, vp, i32, i32, i32, Grid, Block3d, i32,
                                           ctypes.c_float, vp, sz, vp, vp]
        L.psa_attention_run_3d.restype = ctypes.c_int
        L.psa_l2_workspace_size.argtypes = [i32]
        L.psa_l2_workspace_size.restype = sz
        L.psa_l2_distance.argtypes = [vp, vp, i32, i32, i32, vp, vp, vp, sz, vp]
        L.psa_l2_distance.restype = ctypes.c_int
        L.psa_status_string.argtypes = [ctypes.c_int]
        L.psa_status_string.restype = ctypes.c_char_p
        L.psa_last_error.argtypes = []
        L.psa_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def check(status):
    if status != PSA_OK:
        raise PsaError(status, lib().psa_last_error().decode())
    return status


def stripes(params):
    """Host array of psa_stripe_t from a sequence of 6-tuples."""
    arr = (Stripe * max(1, len(params)))()
    for i, m in enumerate(params):
        arr[i] = Stripe(*[int(x) for x in m])
    return arr


def grid_of(frames, height, width, n_text=0):
    return Grid(int(frames), int(height), int(width), int(n_text))


def block3d_of(pb):
    t, h, w = (int(x) for x in pb)
    return Block3d(t, h, w)
