"""ctypes view of libssba.so (include/ssba.h).  Argument marshalling only.

Loading fails loudly (ImportError) when the library has not been built: there
is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libssba.so")

SSBA_OK = 0
SSBA_ERR_ARG = 1
SSBA_ERR_SHAPE = 2
SSBA_ERR_UNSUPPORTED = 3
SSBA_ERR_WORKSPACE = 4
SSBA_ERR_NONFINITE = 5
SSBA_ERR_HIP = 6

DT_BF16 = 0
DT_F32 = 1
GATE_TOPK = 0
GATE_WINDOW = 1
GATE_DENSE = 2
GATE_TOPK_SHARED = 3

EXPORTS = ("ssba_abi_version", "ssba_status_str", "ssba_workspace_size", "ssba_build_index",
           "ssba_forward", "ssba_forward_dense", "ssba_read_device_status",
           "ssba_forward_kernel", "ssba_forward_topk", "ssba_layers_workspace_size",
           "ssba_forward_layers", "ssba_haar_dwt", "ssba_haar_iwt", "ssba_haar_kernel_name",
           "ssba_forward_train", "ssba_backward_workspace_size", "ssba_backward",
           "ssba_probe_mfma", "ssba_build_index_ex", "ssba_forward_ex", "ssba_forward_topk_ex",
           "ssba_forward_train_ex", "ssba_backward_ex", "ssba_forward_layers_ex",
           "ssba_read_device_status_ex", "ssba_forward_topk_noalloc", "ssba_pool_keys_ex",
           "ssba_forward_gated_ex", "ssba_rope_pool_keys_ex", "ssba_forward_topk_rope_ex")

# Byte count that the binding passes for a buffer it cannot size (None).
UNSIZED = ctypes.c_size_t(-1).value


class SsbaDesc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32), ("tile", ctypes.c_int32),
        ("shift_y", ctypes.c_int32), ("shift_x", ctypes.c_int32),
        ("n_text", ctypes.c_int32), ("gate", ctypes.c_int32), ("keep", ctypes.c_int32),
        ("win_h", ctypes.c_int32), ("win_w", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("stride_b", ctypes.c_int64), ("stride_h", ctypes.c_int64), ("stride_t", ctypes.c_int64),
    ]


class SsbaLayer(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("o", ctypes.c_void_p), ("keep", ctypes.c_int32), ("skip", ctypes.c_int32)]


class HaarDesc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("c", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("levels", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class SsbaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} (status {status})")


_lib = None


def load(path: str = None) -> ctypes.CDLL:
    """Load libssba.so (or `path`) once.  Raises ImportError if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2605_15684_amd.build` "
                          "(the SSBA path has no CPU fallback)")
    # PyTorch ships its own HIP runtime under the same soname.  Importing it
    # first makes this library bind to that runtime, so kernels launched here
    # run on torch's streams and memory; loaded the other way round the
    # process would hold two runtimes.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    dp = ctypes.POINTER(SsbaDesc)
    lib.ssba_abi_version.restype = ctypes.c_int
    lib.ssba_abi_version.argtypes = []
    lib.ssba_status_str.restype = ctypes.c_char_p
    lib.ssba_status_str.argtypes = [ctypes.c_int]
    lib.ssba_workspace_size.restype = ctypes.c_int
    lib.ssba_workspace_size.argtypes = [dp, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    lib.ssba_build_index.restype = ctypes.c_int
    lib.ssba_build_index.argtypes = [dp, vp, vp, vp, vp, vp]
    lib.ssba_forward.restype = ctypes.c_int
    lib.ssba_forward.argtypes = [dp, vp, vp, vp, vp, vp, vp]
    lib.ssba_forward_dense.restype = ctypes.c_int
    lib.ssba_forward_dense.argtypes = [dp, vp, vp, vp, vp, vp]
    lib.ssba_forward_topk.restype = ctypes.c_int
    lib.ssba_forward_topk.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp]
    lib.ssba_forward_kernel.restype = ctypes.c_char_p
    lib.ssba_forward_kernel.argtypes = [dp, ctypes.c_int]
    lib.ssba_layers_workspace_size.restype = ctypes.c_int
    lib.ssba_layers_workspace_size.argtypes = [dp, ctypes.c_int, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    lib.ssba_forward_layers.restype = ctypes.c_int
    lib.ssba_forward_layers.argtypes = [dp, ctypes.POINTER(SsbaLayer), ctypes.c_int, vp, vp, vp]
    lib.ssba_forward_train.restype = ctypes.c_int
    lib.ssba_forward_train.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp]
    lib.ssba_backward_workspace_size.restype = ctypes.c_int
    lib.ssba_backward_workspace_size.argtypes = [dp, ctypes.POINTER(sz)]
    lib.ssba_backward.restype = ctypes.c_int
    lib.ssba_backward.argtypes = [dp] + [vp] * 12
    hp = ctypes.POINTER(HaarDesc)
    lib.ssba_haar_dwt.restype = ctypes.c_int
    lib.ssba_haar_dwt.argtypes = [hp, vp, ctypes.POINTER(vp), vp]
    lib.ssba_haar_iwt.restype = ctypes.c_int
    lib.ssba_haar_iwt.argtypes = [hp, ctypes.POINTER(vp), ctypes.POINTER(vp), vp, vp]
    lib.ssba_haar_kernel_name.restype = ctypes.c_char_p
    lib.ssba_haar_kernel_name.argtypes = [hp, ctypes.c_int]
    lib.ssba_read_device_status.restype = ctypes.c_int
    lib.ssba_read_device_status.argtypes = [dp, vp, ctypes.POINTER(ctypes.c_int), vp]
    lib.ssba_probe_mfma.restype = ctypes.c_int
    lib.ssba_probe_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, vp, vp]
    for name, args in (("ssba_build_index_ex", [dp, vp, vp, vp, sz, vp, sz, vp]),
                       ("ssba_forward_ex", [dp, vp, vp, vp, vp, sz, vp, vp]),
                       ("ssba_forward_topk_ex", [dp, vp, vp, vp, vp, sz, vp, sz, vp, vp]),
                       ("ssba_forward_train_ex", [dp, vp, vp, vp, vp, sz, vp, vp, vp]),
                       ("ssba_backward_ex", [dp, vp, vp, vp, vp, vp, vp, vp, sz, vp, vp, vp, vp, sz, vp]),
                       ("ssba_forward_layers_ex", [dp, ctypes.POINTER(SsbaLayer), ctypes.c_int, vp, sz, vp, sz,
                                                   vp]),
                       ("ssba_read_device_status_ex", [dp, vp, sz, ctypes.POINTER(ctypes.c_int), vp]),
                       ("ssba_forward_topk_noalloc", [dp, vp, vp, vp, vp, sz, vp, vp]),
                       ("ssba_pool_keys_ex", [dp, vp, vp, sz, vp]),
                       ("ssba_forward_gated_ex", [dp, vp, vp, vp, vp, sz, vp, sz, vp, vp]),
                       ("ssba_rope_pool_keys_ex", [dp, vp, vp, vp, vp, ctypes.c_float, vp, sz, vp]),
                       ("ssba_forward_topk_rope_ex", [dp, vp, vp, vp, vp, vp, ctypes.c_float, vp, sz, vp, sz,
                                                      vp, vp])):
        fn = getattr(lib, name)
        fn.restype = ctypes.c_int
        fn.argtypes = args
    _lib = lib
    return lib


def status_str(status: int) -> str:
    return load().ssba_status_str(int(status)).decode()


def check(status: int, where: str) -> None:
    if status != SSBA_OK:
        raise SsbaError(status, where)


def workspace_size(desc: SsbaDesc):
    ib, sb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    check(load().ssba_workspace_size(ctypes.byref(desc), ctypes.byref(ib), ctypes.byref(sb)),
          "ssba_workspace_size")
    return ib.value, sb.value


def _nb(n):
    return UNSIZED if n is None else int(n)


def build_index(desc, q_ptr, k_ptr, index_ptr, scratch_ptr, stream, index_bytes=None,
                scratch_bytes=None) -> int:
    """ssba_build_index_ex; a size of None is passed as unchecked."""
    return load().ssba_build_index_ex(ctypes.byref(desc), q_ptr, k_ptr, index_ptr, _nb(index_bytes),
                                      scratch_ptr, _nb(scratch_bytes), stream)


def forward(desc, q_ptr, k_ptr, v_ptr, index_ptr, o_ptr, stream, index_bytes=None) -> int:
    return load().ssba_forward_ex(ctypes.byref(desc), q_ptr, k_ptr, v_ptr, index_ptr, _nb(index_bytes),
                                  o_ptr, stream)


def forward_dense(desc, q_ptr, k_ptr, v_ptr, o_ptr, stream) -> int:
    return load().ssba_forward_dense(ctypes.byref(desc), q_ptr, k_ptr, v_ptr, o_ptr, stream)


def read_device_status(desc, scratch_ptr, stream, scratch_bytes=None):
    out = ctypes.c_int(0)
    check(load().ssba_read_device_status_ex(ctypes.byref(desc), scratch_ptr, _nb(scratch_bytes),
                                            ctypes.byref(out), stream), "ssba_read_device_status")
    return out.value


def forward_topk(desc, q_ptr, k_ptr, v_ptr, index_ptr, scratch_ptr, o_ptr, stream, index_bytes=None,
                 scratch_bytes=None) -> int:
    return load().ssba_forward_topk_ex(ctypes.byref(desc), q_ptr, k_ptr, v_ptr, index_ptr, _nb(index_bytes),
                                       scratch_ptr, _nb(scratch_bytes), o_ptr, stream)


def pool_keys(desc, k_ptr, scratch_ptr, stream, scratch_bytes=None) -> int:
    """ssba_pool_keys_ex: the pooling launch of the fused top-k form."""
    return load().ssba_pool_keys_ex(ctypes.byref(desc), k_ptr, scratch_ptr, _nb(scratch_bytes), stream)


def forward_gated(desc, q_ptr, k_ptr, v_ptr, index_ptr, scratch_ptr, o_ptr, stream, index_bytes=None,
                  scratch_bytes=None) -> int:
    """ssba_forward_gated_ex: the gated attention launch of the fused top-k form."""
    return load().ssba_forward_gated_ex(ctypes.byref(desc), q_ptr, k_ptr, v_ptr, index_ptr, _nb(index_bytes),
                                        scratch_ptr, _nb(scratch_bytes), o_ptr, stream)


def rope_pool_keys(desc, q_ptr, k_ptr, q_rope_ptr, k_rope_ptr, theta, scratch_ptr, stream,
                   scratch_bytes=None) -> int:
    """ssba_rope_pool_keys_ex: the rotary pre-pass of the fused call."""
    return load().ssba_rope_pool_keys_ex(ctypes.byref(desc), q_ptr, k_ptr, q_rope_ptr, k_rope_ptr,
                                         ctypes.c_float(theta), scratch_ptr, _nb(scratch_bytes), stream)


def forward_topk_rope(desc, q_ptr, k_ptr, v_ptr, q_rope_ptr, k_rope_ptr, theta, index_ptr, scratch_ptr, o_ptr,
                      stream, index_bytes=None, scratch_bytes=None) -> int:
    """ssba_forward_topk_rope_ex: the rotary pre-pass, then the gated attention."""
    return load().ssba_forward_topk_rope_ex(ctypes.byref(desc), q_ptr, k_ptr, v_ptr, q_rope_ptr, k_rope_ptr,
                                            ctypes.c_float(theta), index_ptr, _nb(index_bytes), scratch_ptr,
                                            _nb(scratch_bytes), o_ptr, stream)


NOALLOC_SCRATCH_BYTES = 8 << 20   # SSBA_NOALLOC_SCRATCH_BYTES


def forward_topk_noalloc(desc, q_ptr, k_ptr, v_ptr, index_ptr, o_ptr, stream, index_bytes=None) -> int:
    """ssba_forward_topk_noalloc: scratch from the library's fixed device array."""
    return load().ssba_forward_topk_noalloc(ctypes.byref(desc), q_ptr, k_ptr, v_ptr, index_ptr,
                                            _nb(index_bytes), o_ptr, stream)


def forward_kernel(desc, dense: bool = False, mode: int = None):
    """Name of the kernel ssba_forward (mode 0), ssba_forward_dense (mode 1,
    or dense=True) or ssba_forward_topk (mode 2) would launch."""
    m = (1 if dense else 0) if mode is None else mode
    name = load().ssba_forward_kernel(ctypes.byref(desc), m)
    return None if name is None else name.decode()


def layers_workspace_size(desc: SsbaDesc, n_layers: int):
    ib, sb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    check(load().ssba_layers_workspace_size(ctypes.byref(desc), int(n_layers), ctypes.byref(ib),
                                            ctypes.byref(sb)), "ssba_layers_workspace_size")
    return ib.value, sb.value


def forward_layers(desc, layers, index_ptr, scratch_ptr, stream, index_bytes=None, scratch_bytes=None) -> int:
    """`layers`: a ctypes array of SsbaLayer."""
    return load().ssba_forward_layers_ex(ctypes.byref(desc), layers, len(layers), index_ptr, _nb(index_bytes),
                                         scratch_ptr, _nb(scratch_bytes), stream)


def haar_dwt(desc, x_ptr, level_ptrs, stream) -> int:
    arr = (ctypes.c_void_p * max(1, len(level_ptrs)))(*level_ptrs)
    return load().ssba_haar_dwt(ctypes.byref(desc), x_ptr, arr, stream)


def haar_iwt(desc, level_ptrs, residual_ptrs, x_ptr, stream) -> int:
    arr = (ctypes.c_void_p * max(1, len(level_ptrs)))(*level_ptrs)
    res = None if residual_ptrs is None else (ctypes.c_void_p * max(1, len(residual_ptrs)))(*residual_ptrs)
    return load().ssba_haar_iwt(ctypes.byref(desc), arr, res, x_ptr, stream)


def haar_kernel_name(desc, inverse: bool):
    name = load().ssba_haar_kernel_name(ctypes.byref(desc), 1 if inverse else 0)
    return None if name is None else name.decode()


def probe_mfma(blocks: int, iters: int, sink_ptr, stream) -> int:
    return load().ssba_probe_mfma(blocks, iters, sink_ptr, stream)


def forward_train(desc, q_ptr, k_ptr, v_ptr, index_ptr, o_ptr, lse_ptr, stream, index_bytes=None) -> int:
    return load().ssba_forward_train_ex(ctypes.byref(desc), q_ptr, k_ptr, v_ptr, index_ptr, _nb(index_bytes),
                                        o_ptr, lse_ptr, stream)


def backward_workspace_size(desc) -> int:
    sb = ctypes.c_size_t(0)
    check(load().ssba_backward_workspace_size(ctypes.byref(desc), ctypes.byref(sb)), "ssba_backward_workspace_size")
    return sb.value


def backward(desc, q, k, v, o, dout, lse, index, dq, dk, dv, scratch, stream, index_bytes=None,
             scratch_bytes=None) -> int:
    return load().ssba_backward_ex(ctypes.byref(desc), q, k, v, o, dout, lse, index, _nb(index_bytes), dq, dk,
                                   dv, scratch, _nb(scratch_bytes), stream)
