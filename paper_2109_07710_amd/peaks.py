"""ctypes binding of libcbwpeaks.so (include/cbw_peaks.h): the measured
matrix-core and HBM ceilings the benchmark quotes next to the published
MI355X peaks.  Argument marshalling only; the caller times the launches."""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcbwpeaks.so")

MFMA_16X16X32, MFMA_32X32X16 = 0, 1

_lib = None


def lib():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libcbwpeaks.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    L.cbw_peak_seed_bytes.argtypes = []
    L.cbw_peak_seed_bytes.restype = sz
    L.cbw_peak_sink_words.argtypes = [ctypes.c_int]
    L.cbw_peak_sink_words.restype = sz
    L.cbw_peak_mfma_flops.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
    L.cbw_peak_mfma_flops.restype = ctypes.c_double
    L.cbw_peak_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, vp, vp, vp]
    L.cbw_peak_mfma.restype = ctypes.c_int
    L.cbw_peak_hbm_read.argtypes = [vp, sz, vp, vp]
    L.cbw_peak_hbm_read.restype = ctypes.c_int
    L.cbw_peak_hbm_copy.argtypes = [vp, vp, sz, vp]
    L.cbw_peak_hbm_copy.restype = ctypes.c_int
    _lib = L
    return L


def _ptr(t):
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(st, where):
    if st != 0:
        raise RuntimeError("%s failed (%d)" % (where, st))


def seed_bytes():
    return lib().cbw_peak_seed_bytes()


def sink_words(blocks):
    return lib().cbw_peak_sink_words(blocks)


def mfma_flops(shape, blocks, iters):
    return lib().cbw_peak_mfma_flops(shape, blocks, iters)


def mfma(shape, blocks, iters, seed, sink, stream=None):
    _check(lib().cbw_peak_mfma(shape, blocks, iters, _ptr(seed), _ptr(sink), _stream(stream)), "cbw_peak_mfma")


def hbm_read(src, sink, stream=None):
    _check(lib().cbw_peak_hbm_read(_ptr(src), src.numel() * src.element_size(), _ptr(sink), _stream(stream)),
           "cbw_peak_hbm_read")


def hbm_copy(src, dst, stream=None):
    assert src.numel() * src.element_size() == dst.numel() * dst.element_size()
    _check(lib().cbw_peak_hbm_copy(_ptr(src), _ptr(dst), src.numel() * src.element_size(), _stream(stream)),
           "cbw_peak_hbm_copy")
