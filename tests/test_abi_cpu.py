"""C-ABI checks that need no GPU: the library loads, exports every function
include/convbwd.h declares, and its host-only validation and workspace
planning behave as documented.  No compute call is made here."""
import ctypes
import os
import re

import pytest

import paper_2109_07710_amd as cb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "convbwd.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "while")))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(cb.LIB_PATH):
        pytest.skip("library not built")
    return cb.lib()


def test_exports_every_declared_symbol(L):
    names = _declared_functions()
    assert len(names) >= 13
    assert set(names) == set(cb.EXPORTS)
    for n in names:
        assert hasattr(L, n), n


def test_status_strings(L):
    for s in (0, -1, -2, -3, -4):
        assert cb.status_string(s) != "unknown status"
    assert cb.status_string(5) == "unknown status"


def _desc(**kw):
    base = dict(N=2, C=64, H=10, W=12, K=32, R=3, S=3, stride=(1, 1), pad=(1, 1), dtype="bf16")
    base.update(kw)
    return cb.ConvDesc.make(**base)


def test_validation_codes(L):
    assert cb.cbw_validate_desc(_desc()) == cb.CBW_OK
    assert cb.cbw_validate_desc(_desc(stride=(2, 3), pad=(0, 2), R=5, S=1)) == cb.CBW_OK
    d = _desc()
    d.P += 1
    assert cb.cbw_validate_desc(d) == cb.CBW_ERR_INVALID_ARG
    d = _desc()
    d.N = 0
    assert cb.cbw_validate_desc(d) == cb.CBW_ERR_INVALID_ARG
    d = _desc()
    d.stride_h = 0
    assert cb.cbw_validate_desc(d) == cb.CBW_ERR_INVALID_ARG
    d = _desc()
    d.pad_w = -1
    assert cb.cbw_validate_desc(d) == cb.CBW_ERR_INVALID_ARG
    d = _desc()
    d.dtype = 7
    assert cb.cbw_validate_desc(d) == cb.CBW_ERR_INVALID_ARG
    assert cb.cbw_validate_desc(_desc(C=12)) == cb.CBW_ERR_UNSUPPORTED           # not a multiple of 8 (bf16)
    assert cb.cbw_validate_desc(_desc(C=12, K=8, dtype="f32")) == cb.CBW_OK     # multiple of 4 (fp32)
    assert cb.cbw_validate_desc(_desc(act_layout="nchw")) == cb.CBW_OK
    assert cb.cbw_validate_desc(_desc(w_layout="kcrs")) == cb.CBW_OK
    assert cb.cbw_validate_desc(_desc(N=4096, H=1024, W=1024, C=8)) == cb.CBW_ERR_UNSUPPORTED  # >= 2^31 elems
    # the fp32 weight gradient must stay below 2^31 bytes: 7680^2*9*4 fits, 8192^2*9*4 does not
    assert cb.cbw_validate_desc(_desc(N=1, H=4, W=4, C=7680, K=7680)) == cb.CBW_OK
    assert cb.cbw_validate_desc(_desc(N=1, H=4, W=4, C=8192, K=8192)) == cb.CBW_ERR_UNSUPPORTED
    assert L.cbw_validate_desc(None) == cb.CBW_ERR_INVALID_ARG
    assert cb.cbw_validate_desc(_desc(H=1, R=3, pad=(0, 1))) == cb.CBW_ERR_INVALID_ARG  # empty output


def test_mask_words(L):
    d = _desc()
    assert cb.cbw_mask_words(d) == (2 * 64 * 10 * 12 + 31) // 32
    assert cb.cbw_dy_mask_words(d) == (2 * 32 * 10 * 12 + 31) // 32
    bad = _desc()
    bad.P = 99
    assert cb.cbw_mask_words(bad) == 0


def test_workspace_sizes(L):
    d = cb.ConvDesc.make(32, 256, 56, 56, 256, 3, 3, 1, 1)
    dense = cb.cbw_workspace_size(d, cb.CBW_OP_BWD_DATA)
    masked = cb.cbw_workspace_size(d, cb.CBW_OP_BWD_DATA_MASKED)
    wgt = cb.cbw_workspace_size(d, cb.CBW_OP_BWD_WEIGHT)
    wt_bytes = 256 * 256 * 9 * 2
    assert dense >= wt_bytes + 256
    npix = 32 * 56 * 56
    assert masked >= dense + npix * 4              # at least one channel group of live-pixel lists
    assert wgt >= 2 * 256 * 9 * 256 * 4            # at least two split-K partials of dW
    assert all(x % 256 == 0 for x in (dense, masked))
    with pytest.raises(cb.CbwError):
        cb.cbw_workspace_size(d, 7)
    assert L.cbw_workspace_size(ctypes.byref(d), 0, None) == cb.CBW_ERR_INVALID_ARG


def test_forward_descriptor_rules(L):
    """The forward runs as the data-gradient GEMM with C and K, (H, W) and
    (P, Q) interchanged, flipped taps and padding R-1-pad: stride 1 only."""
    d = cb.ConvDesc.make(32, 256, 56, 56, 256, 3, 3, 1, 1)
    fwd = cb.cbw_workspace_size(d, cb.CBW_OP_FWD)
    assert fwd == cb.cbw_workspace_size(d, cb.CBW_OP_BWD_DATA)   # same shape with C = K
    assert fwd >= 256 * 256 * 9 * 2 + 256
    d2 = cb.ConvDesc.make(2, 64, 10, 12, 128, 3, 3, 1, 1)           # C != K: forward plans as (C, K) swapped
    swapped = cb.ConvDesc.make(2, 128, 10, 12, 64, 3, 3, 1, 1)
    assert cb.cbw_workspace_size(d2, cb.CBW_OP_FWD) == cb.cbw_workspace_size(swapped, cb.CBW_OP_BWD_DATA)
    assert cb.cbw_workspace_size(_desc(R=1, S=1, pad=(0, 0)), cb.CBW_OP_FWD) > 0
    n = ctypes.c_size_t(0)
    for bad in (_desc(stride=(2, 1)), _desc(stride=(1, 2)), _desc(R=3, S=3, pad=(3, 1)), _desc(R=1, S=3, pad=(1, 1))):
        assert L.cbw_workspace_size(ctypes.byref(bad), cb.CBW_OP_FWD, ctypes.byref(n)) == cb.CBW_ERR_UNSUPPORTED
        assert L.conv_fwd_relu_mask(ctypes.byref(bad), None, None, None, None, None, 0, None) == \
            cb.CBW_ERR_UNSUPPORTED
    fake = ctypes.c_void_p(1 << 20)
    assert L.conv_fwd_relu_mask(ctypes.byref(_desc()), None, fake, fake, None, None, 0, None) == \
        cb.CBW_ERR_INVALID_ARG
    assert L.conv_fwd_relu_mask(ctypes.byref(_desc()), fake, fake, fake, None, None, 0, None) == \
        cb.CBW_ERR_WORKSPACE
    misaligned = ctypes.c_void_p((1 << 20) + 4)
    assert L.conv_fwd_relu_mask(ctypes.byref(_desc()), fake, fake, fake, misaligned, None, 0, None) == \
        cb.CBW_ERR_UNSUPPORTED


def test_elementwise_descriptor_rules(L):
    """The per-element data gradient: bf16, KRSC, C in {64, 128, 256, 512},
    K < 65536; its workspace is one int32 count per output pixel."""
    for C in (64, 128, 256, 512):
        d = cb.ConvDesc.make(2, C, 10, 12, 40, 3, 3, 1, 1)
        assert cb.cbw_workspace_size(d, cb.CBW_OP_BWD_DATA_ELEMENTWISE) == (2 * 10 * 12 * 4 + 255) // 256 * 256
    n = ctypes.c_size_t(0)
    bad = [cb.ConvDesc.make(2, 96, 10, 12, 40, 3, 3, 1, 1), cb.ConvDesc.make(2, 1024, 4, 4, 8, 1, 1),
           cb.ConvDesc.make(2, 64, 10, 12, 40, 3, 3, 1, 1, dtype="f32"),
           cb.ConvDesc.make(2, 64, 10, 12, 40, 3, 3, 1, 1, w_layout="kcrs"),
           cb.ConvDesc.make(1, 64, 2, 2, 65536, 1, 1)]
    fake = ctypes.c_void_p(1 << 20)
    for d in bad:
        assert L.cbw_workspace_size(ctypes.byref(d), cb.CBW_OP_BWD_DATA_ELEMENTWISE, ctypes.byref(n)) == \
            cb.CBW_ERR_UNSUPPORTED
        assert L.conv_bwd_data_elementwise(ctypes.byref(d), fake, fake, fake, fake, fake, 1 << 20, None) == \
            cb.CBW_ERR_UNSUPPORTED
    good = cb.ConvDesc.make(2, 64, 10, 12, 40, 3, 3, 1, 1)
    assert L.conv_bwd_data_elementwise(ctypes.byref(good), fake, fake, None, fake, fake, 1 << 20, None) == \
        cb.CBW_ERR_INVALID_ARG
    assert L.conv_bwd_data_elementwise(ctypes.byref(good), fake, fake, fake, fake, fake, 16, None) == \
        cb.CBW_ERR_WORKSPACE


def test_null_arguments_rejected_without_gpu(L):
    d = _desc()
    n = ctypes.c_size_t(0)
    assert L.cbw_workspace_size(ctypes.byref(d), 1, ctypes.byref(n)) == 0
    # Null tensors are rejected by validation before any HIP call is made.
    assert L.conv_bwd_data_masked(ctypes.byref(d), None, None, None, None, None, 0, 0, None) == \
        cb.CBW_ERR_INVALID_ARG
    assert L.conv_bwd_data(ctypes.byref(d), None, None, None, None, 0, None) == cb.CBW_ERR_INVALID_ARG
    assert L.conv_bwd_weight_sparse(ctypes.byref(d), None, None, None, None, None, 0, 0, None) == \
        cb.CBW_ERR_INVALID_ARG
    assert L.cbw_relu_mask_pack(ctypes.byref(d), None, None, None) == cb.CBW_ERR_INVALID_ARG
    assert L.cbw_nonzero_mask_pack(1, 10, None, None, None) == cb.CBW_ERR_INVALID_ARG
    assert L.cbw_nonzero_mask_pack(1, 0, None, None, None) == cb.CBW_OK
    assert L.cbw_nonzero_mask_pack(9, 10, None, None, None) == cb.CBW_ERR_INVALID_ARG
    bad = _desc()
    bad.Q = 1
    assert L.conv_bwd_data(ctypes.byref(bad), None, None, None, None, 0, None) == cb.CBW_ERR_INVALID_ARG
    # Workspace check comes after the pointer checks: fake aligned pointers, no workspace.
    fake = ctypes.c_void_p(1 << 20)
    assert L.conv_bwd_data(ctypes.byref(d), fake, fake, fake, None, 0, None) == cb.CBW_ERR_WORKSPACE
    assert L.conv_bwd_weight_sparse(ctypes.byref(d), fake, fake, None, fake, None, 0, 0, None) == \
        cb.CBW_ERR_WORKSPACE
    misaligned = ctypes.c_void_p((1 << 20) + 2)
    assert L.conv_bwd_data(ctypes.byref(d), misaligned, fake, fake, None, 0, None) == cb.CBW_ERR_UNSUPPORTED


def _ws(d, op):
    n = ctypes.c_size_t(0)
    st = cb.lib().cbw_workspace_size(ctypes.byref(d), op, ctypes.byref(n))
    return st, n.value


def test_nchw_workspace_and_scope(L):
    """NCHW callers of the three backward operations get NHWC copies of their
    activations (and NHWC-order footprints) after every NHWC region: the
    workspace grows by exactly those buffers, 256-byte aligned; the forward
    and the per-element data gradient refuse NCHW."""
    al = lambda b: (b + 255) // 256 * 256
    a = cb.ConvDesc.make(4, 64, 10, 12, 32, 3, 3, 1, 1)
    b = cb.ConvDesc.make(4, 64, 10, 12, 32, 3, 3, 1, 1, act_layout="nchw")
    act_x, act_y = 4 * 10 * 12 * 64 * 2, 4 * 10 * 12 * 32 * 2
    bits_x, bits_y = (4 * 10 * 12 * 64 + 31) // 32 * 4, (4 * 10 * 12 * 32 + 31) // 32 * 4
    st, nh = _ws(a, cb.CBW_OP_BWD_DATA)
    st2, nc = _ws(b, cb.CBW_OP_BWD_DATA)
    assert st == st2 == cb.CBW_OK and nc == nh + al(act_y) + al(act_x)
    st, nh = _ws(a, cb.CBW_OP_BWD_DATA_MASKED)
    st2, nc = _ws(b, cb.CBW_OP_BWD_DATA_MASKED)
    assert st == st2 == cb.CBW_OK and nc == nh + al(act_y) + al(act_x) + al(bits_x)
    st, nh = _ws(a, cb.CBW_OP_BWD_WEIGHT)
    st2, nc = _ws(b, cb.CBW_OP_BWD_WEIGHT)
    assert st == st2 == cb.CBW_OK and nc == nh + al(act_x) + al(act_y) + al(bits_y)
    assert _ws(b, cb.CBW_OP_FWD)[0] == cb.CBW_ERR_UNSUPPORTED
    e = cb.ConvDesc.make(4, 64, 10, 12, 64, 3, 3, 1, 1, act_layout="nchw")
    assert _ws(e, cb.CBW_OP_BWD_DATA_ELEMENTWISE)[0] == cb.CBW_ERR_UNSUPPORTED


# (N, C, H, W) -> expected (channels, capacity, rows).  The rows follow from
# counting rounds by hand: with 256 resident tiles, T tiles take ceil(T / 256)
# rounds, and the pick minimises rounds x rows among capacity, capacity - 16
# and capacity - 32 (full capacity when T <= 128, where the reduction splits).
TILING_CASES = [
    # 100352 pixels, 256 channels: 448 / 483 / 523 tiles -> 2, 2, 3 rounds -> 208
    ((32, 256, 56, 56), (256, 224, 208)),
    # 49152 pixels: 220 / 237 / 256 tiles, one round each -> the smallest, 192
    ((12, 256, 64, 64), (256, 224, 192)),
    # 114688 pixels: 512 / 552 / 598 tiles -> 2, 3, 3 rounds -> 224
    ((28, 256, 64, 64), (256, 224, 224)),
    # 128 channels, 100352 pixels: 224 / 233 / 242 tiles, one round -> 416
    ((32, 128, 56, 56), (128, 448, 416)),
    # 110592 pixels: 247 / 256 / 266 tiles -> 1, 1, 2 rounds -> 432
    ((27, 128, 64, 64), (128, 448, 432)),
    # 64 channels, 100352 pixels: 196 / 203 / 210 tiles, one round -> 480
    ((2, 64, 224, 224), (64, 512, 480)),
    # 126976 pixels: 248 / 256 / 265 tiles -> 1, 1, 2 rounds -> 496
    ((31, 64, 64, 64), (64, 512, 496)),
    # 512 pixels: one tile, split reduction -> full capacity
    ((2, 16, 16, 16), (64, 512, 512)),
    # 28672 pixels: 128 tiles of 224 -> split regime -> 224
    ((8, 256, 56, 64), (256, 224, 224)),
]


@pytest.mark.parametrize("shape,expect", TILING_CASES, ids=lambda v: "x".join(map(str, v)))
def test_data_tile_rows(L, shape, expect):
    N, C, H, W = shape
    d = cb.ConvDesc.make(N, C, H, W, C, 3, 3, 1, 1)
    assert cb.cbw_data_tiling(d) == expect


def test_data_tiling_rejects_bad_descriptors(L):
    d = _desc()
    d.P += 1
    z = ctypes.c_int32(0)
    assert L.cbw_data_tiling(ctypes.byref(d), ctypes.byref(z), None, None) == cb.CBW_ERR_INVALID_ARG


def test_noalloc_rejects_descriptors_beyond_its_scratch(L):
    """The built-in-scratch data gradient refuses, before any device call, a
    layer whose workspace would exceed its 32 MiB: 64 channels at 224 x 224
    with 200 images needs 4 bytes of live list per pixel (40 MB).  (A 5 x 5
    layer: with a 3 x 3 or 1 x 1 filter the row-window or pointwise kernel
    would serve it, with no lists.)"""
    d = _desc(N=200, C=64, K=64, H=224, W=224, R=5, S=5, pad=(2, 2))
    assert cb.cbw_validate_desc(d) == cb.CBW_OK
    st = L.conv_bwd_data_masked_noalloc(ctypes.byref(d), None, None, None, None, 0, None)
    assert st == cb.CBW_ERR_WORKSPACE
    d = _desc(N=0)
    assert L.conv_bwd_data_masked_noalloc(ctypes.byref(d), None, None, None, None, 0, None) == cb.CBW_ERR_INVALID_ARG


def test_peaks_library_exports_its_header():
    import paper_2109_07710_amd.peaks as pk
    if not os.path.exists(pk.LIB_PATH):
        pytest.skip("library not built")
    text = open(os.path.join(ROOT, "include", "cbw_peaks.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M))
    assert names == {"cbw_peak_seed_bytes", "cbw_peak_sink_words", "cbw_peak_mfma_flops", "cbw_peak_mfma",
                     "cbw_peak_hbm_read", "cbw_peak_hbm_copy"}
    PL = pk.lib()
    for n in names:
        assert hasattr(PL, n), n
    # host-only queries and argument checks (nothing is launched on an error)
    assert pk.mfma_flops(pk.MFMA_16X16X32, 2, 3) == 2 * 16 * 16 * 32 * 8 * 3 * 2 * 4
    assert pk.mfma_flops(pk.MFMA_32X32X16, 1, 1) == 2 * 32 * 32 * 16 * 4 * 4
    assert PL.cbw_peak_mfma(7, 1, 1, None, None, None) == -1
    assert PL.cbw_peak_hbm_copy(None, None, 16, None) == -1


def test_both_gradients_workspace_and_validation(L):
    """conv_bwd_sparse: its workspace holds the masked data gradient's, then
    (from the next 256-byte boundary) the weight gradient's; every argument
    error is reported before anything is launched."""
    d = cb.ConvDesc.make(32, 256, 56, 56, 256, 3, 3, 1, 1)
    both = cb.cbw_workspace_size(d, cb.CBW_OP_BWD_BOTH)
    masked = cb.cbw_workspace_size(d, cb.CBW_OP_BWD_DATA_MASKED)
    wgt = cb.cbw_workspace_size(d, cb.CBW_OP_BWD_WEIGHT)
    off = cb.both_weight_offset(d)
    assert off % 256 == 0 and masked <= off < masked + 256
    assert both == off + wgt
    fake = ctypes.c_void_p(1 << 20)
    call = L.conv_bwd_sparse
    # null tensors, then unknown flags, then misaligned pointers, then the workspace
    assert call(ctypes.byref(d), None, fake, fake, None, None, fake, fake, None, 0, 0, None) == \
        cb.CBW_ERR_INVALID_ARG
    assert call(ctypes.byref(d), fake, fake, fake, None, None, fake, fake, None, 0, 4, None) == \
        cb.CBW_ERR_INVALID_ARG
    misaligned = ctypes.c_void_p((1 << 20) + 4)
    assert call(ctypes.byref(d), fake, fake, fake, misaligned, None, fake, fake, None, 0, 0, None) == \
        cb.CBW_ERR_UNSUPPORTED
    assert call(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, None, 0, 0, None) == \
        cb.CBW_ERR_WORKSPACE
    assert call(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, both - 1, 0, None) == \
        cb.CBW_ERR_WORKSPACE
    bad = cb.ConvDesc.make(32, 256, 56, 56, 256, 3, 3, 1, 1)
    bad.P += 1
    assert call(ctypes.byref(bad), fake, fake, fake, None, None, fake, fake, fake, both, 0, None) == \
        cb.CBW_ERR_INVALID_ARG
