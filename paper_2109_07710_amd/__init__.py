"""Masked convolution backward pass (ReLU-derived sparsity) on MI355X.

Thin ctypes binding over libconvbwd.so, the C-ABI declared in
include/convbwd.h.  It only marshals arguments: torch tensors (device memory,
streams) become pointers; every step of the computation runs in the HIP
kernels of the library.  A non-zero status becomes CbwError.  There is no
fallback: if the library is missing, importing the binding's functions
raises.

The operations are those of arXiv 2109.07710: the data gradient computed only
where the forward ReLU footprint is live (output sparsity, Sec. III-B), the
weight gradient skipping all-zero blocks of the incoming gradient (input
sparsity), and the dense data gradient.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libconvbwd.so")

CBW_OK, CBW_ERR_INVALID_ARG, CBW_ERR_UNSUPPORTED, CBW_ERR_WORKSPACE, CBW_ERR_HIP = 0, -1, -2, -3, -4
CBW_NCHW, CBW_NHWC = 0, 1
CBW_KCRS, CBW_KRSC = 0, 1
CBW_F32, CBW_BF16 = 0, 1
CBW_OP_BWD_DATA, CBW_OP_BWD_DATA_MASKED, CBW_OP_BWD_WEIGHT, CBW_OP_FWD, CBW_OP_BWD_DATA_ELEMENTWISE = 0, 1, 2, 3, 4
CBW_OP_BWD_BOTH = 5
CBW_FLAG_NO_SKIP = 1
CBW_FLAG_SKIP_X_BLOCKS = 2

EXPORTS = ("cbw_status_string", "cbw_validate_desc", "cbw_mask_words", "cbw_dy_mask_words",
           "cbw_workspace_size", "cbw_data_tiling", "cbw_relu_mask_pack", "cbw_nonzero_mask_pack", "conv_bwd_data",
           "conv_bwd_data_masked", "conv_bwd_data_masked_noalloc", "conv_fwd_relu_mask", "conv_bwd_weight_sparse", "conv_bwd_weight_sparse_x", "conv_bwd_sparse",
           "conv_bwd_data_elementwise", "cbw_read_pixel_counts", "cbw_read_weight_work", "cbw_read_stats",
           "cbw_read_live_lists",
           "cbw_read_occupancy", "cbw_set_profile_events")


class ConvDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("N", "C", "H", "W", "K", "R", "S", "P", "Q",
                 "stride_h", "stride_w", "pad_h", "pad_w", "act_layout", "w_layout", "dtype")]

    @classmethod
    def make(cls, N, C, H, W, K, R, S, stride=(1, 1), pad=(0, 0), dtype="bf16", w_layout="krsc",
             act_layout="nhwc"):
        if isinstance(stride, int):
            stride = (stride, stride)
        if isinstance(pad, int):
            pad = (pad, pad)
        P = (H + 2 * pad[0] - R) // stride[0] + 1
        Q = (W + 2 * pad[1] - S) // stride[1] + 1
        return cls(N, C, H, W, K, R, S, P, Q, stride[0], stride[1], pad[0], pad[1],
                   {"nhwc": CBW_NHWC, "nchw": CBW_NCHW}[act_layout],
                   {"krsc": CBW_KRSC, "kcrs": CBW_KCRS}[w_layout],
                   {"bf16": CBW_BF16, "f32": CBW_F32}[dtype])


class Stats(ctypes.Structure):
    _fields_ = [("rows_total", ctypes.c_int64), ("rows_live", ctypes.c_int64),
                ("blocks_total", ctypes.c_int64), ("blocks_skipped", ctypes.c_int64)]


class CbwError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (where, status_string(status), status))


_lib = None


def lib():
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libconvbwd.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    dp = ctypes.POINTER(ConvDesc)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    L.cbw_status_string.argtypes = [ctypes.c_int]
    L.cbw_status_string.restype = ctypes.c_char_p
    L.cbw_validate_desc.argtypes = [dp]
    L.cbw_mask_words.argtypes = [dp]
    L.cbw_mask_words.restype = sz
    L.cbw_dy_mask_words.argtypes = [dp]
    L.cbw_dy_mask_words.restype = sz
    L.cbw_workspace_size.argtypes = [dp, ctypes.c_int, ctypes.POINTER(sz)]
    i32p_ = ctypes.POINTER(ctypes.c_int32)
    L.cbw_data_tiling.argtypes = [dp, i32p_, i32p_, i32p_]
    L.cbw_relu_mask_pack.argtypes = [dp, vp, vp, vp]
    L.cbw_nonzero_mask_pack.argtypes = [ctypes.c_int32, ctypes.c_int64, vp, vp, vp]
    L.conv_bwd_data.argtypes = [dp, vp, vp, vp, vp, sz, vp]
    L.conv_bwd_data_masked.argtypes = [dp, vp, vp, vp, vp, vp, sz, ctypes.c_uint32, vp]
    L.conv_bwd_data_masked_noalloc.argtypes = [dp, vp, vp, vp, vp, ctypes.c_uint32, vp]
    L.conv_fwd_relu_mask.argtypes = [dp, vp, vp, vp, vp, vp, sz, vp]
    L.conv_bwd_weight_sparse.argtypes = [dp, vp, vp, vp, vp, vp, sz, ctypes.c_uint32, vp]
    L.conv_bwd_weight_sparse_x.argtypes = [dp, vp, vp, vp, vp, vp, vp, sz, ctypes.c_uint32, vp]
    L.conv_bwd_sparse.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, sz, ctypes.c_uint32, vp]
    L.conv_bwd_data_elementwise.argtypes = [dp, vp, vp, vp, vp, vp, sz, vp]
    L.cbw_read_pixel_counts.argtypes = [dp, vp, sz, vp, ctypes.POINTER(ctypes.c_int64), vp]
    L.cbw_read_weight_work.argtypes = [dp, vp, sz, vp, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32), vp]
    L.cbw_read_stats.argtypes = [dp, ctypes.c_int, vp, sz, ctypes.POINTER(Stats), vp]
    i32p = ctypes.POINTER(ctypes.c_int32)
    L.cbw_read_live_lists.argtypes = [dp, vp, sz, ctypes.c_int, vp, i32p, i32p, vp]
    L.cbw_read_occupancy.argtypes = [dp, vp, sz, vp, i32p, i32p, i32p, i32p, vp]
    L.cbw_set_profile_events.argtypes = [ctypes.c_int, vp, vp]
    for name in EXPORTS:
        if name != "cbw_status_string" and name not in ("cbw_mask_words", "cbw_dy_mask_words"):
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def status_string(status):
    return lib().cbw_status_string(status).decode()


def _check(status, where):
    if status != CBW_OK:
        raise CbwError(status, where)


def _ptr(t):
    """Device pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


# ---------------------------------------------------------------- host-only

def cbw_validate_desc(desc):
    return lib().cbw_validate_desc(ctypes.byref(desc))


def cbw_mask_words(desc):
    return lib().cbw_mask_words(ctypes.byref(desc))


def cbw_dy_mask_words(desc):
    return lib().cbw_dy_mask_words(ctypes.byref(desc))


def cbw_workspace_size(desc, op):
    n = ctypes.c_size_t(0)
    _check(lib().cbw_workspace_size(ctypes.byref(desc), op, ctypes.byref(n)), "cbw_workspace_size")
    return n.value


def cbw_data_tiling(desc):
    """(channels per tile, pixel-row capacity, pixel rows per tile) of the
    data-gradient GEMM in its dense and non-skipping modes (host only)."""
    a, b, c = ctypes.c_int32(0), ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().cbw_data_tiling(ctypes.byref(desc), ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)),
           "cbw_data_tiling")
    return a.value, b.value, c.value


def workspace(desc, op, device="cuda"):
    """A uint8 device tensor of the size `op` needs (allocated by torch)."""
    import torch
    return torch.empty(max(cbw_workspace_size(desc, op), 1), dtype=torch.uint8, device=device)


# ------------------------------------------------------------ device calls

def cbw_relu_mask_pack(desc, X, x_mask, stream=None):
    _check(lib().cbw_relu_mask_pack(ctypes.byref(desc), _ptr(X), _ptr(x_mask), _stream(stream)),
           "cbw_relu_mask_pack")


def cbw_nonzero_mask_pack(dtype, count, t, bits, stream=None):
    _check(lib().cbw_nonzero_mask_pack(dtype, count, _ptr(t), _ptr(bits), _stream(stream)),
           "cbw_nonzero_mask_pack")


def conv_bwd_data(desc, dY, W, dX, ws, stream=None):
    _check(lib().conv_bwd_data(ctypes.byref(desc), _ptr(dY), _ptr(W), _ptr(dX), _ptr(ws), _nbytes(ws),
                               _stream(stream)), "conv_bwd_data")


def conv_bwd_data_masked(desc, dY, W, x_mask, dX, ws, flags=0, stream=None):
    _check(lib().conv_bwd_data_masked(ctypes.byref(desc), _ptr(dY), _ptr(W), _ptr(x_mask), _ptr(dX),
                                      _ptr(ws), _nbytes(ws), flags, _stream(stream)), "conv_bwd_data_masked")


def conv_bwd_data_masked_noalloc(desc, dY, W, x_mask, dX, flags=0, stream=None):
    """conv_bwd_data_masked on the library's built-in scratch (no workspace)."""
    _check(lib().conv_bwd_data_masked_noalloc(ctypes.byref(desc), _ptr(dY), _ptr(W), _ptr(x_mask), _ptr(dX),
                                              flags, _stream(stream)), "conv_bwd_data_masked_noalloc")


def conv_fwd_relu_mask(desc, X, W, Y, y_mask, ws, stream=None):
    """Y = relu(conv(X, W)) and, when y_mask is given, its footprint bits."""
    _check(lib().conv_fwd_relu_mask(ctypes.byref(desc), _ptr(X), _ptr(W), _ptr(Y), _ptr(y_mask), _ptr(ws),
                                    _nbytes(ws), _stream(stream)), "conv_fwd_relu_mask")


def conv_bwd_weight_sparse(desc, X, dY, dy_mask, dW, ws, flags=0, stream=None):
    _check(lib().conv_bwd_weight_sparse(ctypes.byref(desc), _ptr(X), _ptr(dY), _ptr(dy_mask), _ptr(dW),
                                        _ptr(ws), _nbytes(ws), flags, _stream(stream)),
           "conv_bwd_weight_sparse")


def conv_bwd_weight_sparse_x(desc, X, dY, x_mask, dy_mask, dW, ws, flags=0, stream=None):
    _check(lib().conv_bwd_weight_sparse_x(ctypes.byref(desc), _ptr(X), _ptr(dY), _ptr(x_mask), _ptr(dy_mask),
                                          _ptr(dW), _ptr(ws), _nbytes(ws), flags, _stream(stream)),
           "conv_bwd_weight_sparse_x")


def conv_bwd_sparse(desc, X, dY, W, x_mask, dy_mask, dX, dW, ws, flags=0, stream=None):
    """Both gradients in one call (x_mask None: dense data gradient)."""
    _check(lib().conv_bwd_sparse(ctypes.byref(desc), _ptr(X), _ptr(dY), _ptr(W), _ptr(x_mask), _ptr(dy_mask),
                                 _ptr(dX), _ptr(dW), _ptr(ws), _nbytes(ws), flags, _stream(stream)),
           "conv_bwd_sparse")


def both_weight_offset(desc):
    """Byte offset of the weight-gradient part in a conv_bwd_sparse workspace."""
    return (cbw_workspace_size(desc, CBW_OP_BWD_DATA_MASKED) + 255) // 256 * 256


def conv_bwd_data_elementwise(desc, dY, W, x_mask, dX, ws, stream=None):
    _check(lib().conv_bwd_data_elementwise(ctypes.byref(desc), _ptr(dY), _ptr(W), _ptr(x_mask), _ptr(dX),
                                           _ptr(ws), _nbytes(ws), _stream(stream)), "conv_bwd_data_elementwise")


def cbw_read_pixel_counts(desc, ws, stream=None):
    """Per-pixel (tap, k) product counts of the last conv_bwd_data_elementwise
    call on ws (numpy int32 [N*H*W]) and their sum."""
    import numpy as np
    out = np.zeros(desc.N * desc.H * desc.W, np.int32)
    tot = ctypes.c_int64(0)
    _check(lib().cbw_read_pixel_counts(ctypes.byref(desc), _ptr(ws), _nbytes(ws),
                                       out.ctypes.data_as(ctypes.c_void_p), ctypes.byref(tot), _stream(stream)),
           "cbw_read_pixel_counts")
    return out, tot.value


def cbw_read_weight_work(desc, ws, stream=None):
    """Blocks executed per weight-gradient work item: numpy int32 [nsplit][ntiles]."""
    import numpy as np
    ns, nt = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().cbw_read_weight_work(ctypes.byref(desc), _ptr(ws), _nbytes(ws), None, ctypes.byref(ns),
                                      ctypes.byref(nt), _stream(stream)), "cbw_read_weight_work")
    out = np.zeros((ns.value, nt.value), np.int32)
    _check(lib().cbw_read_weight_work(ctypes.byref(desc), _ptr(ws), _nbytes(ws), out.ctypes.data_as(ctypes.c_void_p),
                                      ctypes.byref(ns), ctypes.byref(nt), _stream(stream)), "cbw_read_weight_work")
    return out


def cbw_read_stats(desc, op, ws, stream=None):
    st = Stats()
    _check(lib().cbw_read_stats(ctypes.byref(desc), op, _ptr(ws), _nbytes(ws), ctypes.byref(st),
                                _stream(stream)), "cbw_read_stats")
    return st


def cbw_read_live_lists(desc, ws, group, stream=None):
    """The compacted live-pixel list of one channel group (numpy int32) and the group width."""
    import numpy as np
    n, g = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().cbw_read_live_lists(ctypes.byref(desc), _ptr(ws), _nbytes(ws), group, None, ctypes.byref(n),
                                     ctypes.byref(g), _stream(stream)), "cbw_read_live_lists")
    out = np.zeros(max(n.value, 1), np.int32)
    _check(lib().cbw_read_live_lists(ctypes.byref(desc), _ptr(ws), _nbytes(ws), group,
                                     out.ctypes.data_as(ctypes.c_void_p), ctypes.byref(n), ctypes.byref(g),
                                     _stream(stream)), "cbw_read_live_lists")
    return out[: n.value], g.value


def cbw_read_occupancy(desc, ws, stream=None):
    """The dY block occupancy map [nchunks][ktiles] (numpy uint8), chunk pixels and k-tile width."""
    import numpy as np
    nc, kt, cp, kw = (ctypes.c_int32(0) for _ in range(4))
    args = (ctypes.byref(nc), ctypes.byref(kt), ctypes.byref(cp), ctypes.byref(kw))
    _check(lib().cbw_read_occupancy(ctypes.byref(desc), _ptr(ws), _nbytes(ws), None, *args, _stream(stream)),
           "cbw_read_occupancy")
    out = np.zeros((nc.value, kt.value), np.uint8)
    _check(lib().cbw_read_occupancy(ctypes.byref(desc), _ptr(ws), _nbytes(ws),
                                    out.ctypes.data_as(ctypes.c_void_p), *args, _stream(stream)),
           "cbw_read_occupancy")
    return out, cp.value, kw.value


def cbw_set_profile_events(op, start=None, stop=None):
    """Record events `start`/`stop` around the op's main GEMM kernel on every
    following call of this thread (None, None switches it off): torch.cuda.Event
    objects (recorded once, so that they exist) or raw hipEvent_t handles
    (int)."""
    def handle(e):
        if e is None:
            return None
        return ctypes.c_void_p(e if isinstance(e, int) else e.cuda_event)
    sp, tp = handle(start), handle(stop)
    _check(lib().cbw_set_profile_events(op, sp, tp), "cbw_set_profile_events")
