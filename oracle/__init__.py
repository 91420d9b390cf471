"""Oracle for the masked convolution backward pass (dX, dW) and its helpers.

TEST INFRASTRUCTURE ONLY.  Only tests, the smoke check and the benchmark's
CPU-baseline leg may import this package.  It shares no code with the HIP
library (``paper_2109_07710_amd``) and never imports it.

Contents
--------
* fp64 direct-loop convolution forward / backward-data / backward-weight in
  C (``conv_ref.c``, loaded through ctypes), in the paper's logical order
  X[N][C][H][W], W[K][C][R][S], dY[N][K][P][Q] (Sec. II-A, Sec. IV-B);
* the ReLU mask bitmap (Sec. III-B, boxed derivative; Sec. IV-B output
  bitmap), the per-channel-group live-pixel lists that stand for the paper's
  non-zero indexing (Sec. IV-B), and the dY block occupancy, in numpy;
* 2x2 max-pool forward/backward, for the exactness of the pooled-footprint
  mask at MaxPool -> CONV boundaries;
* pure layout permutations between NHWC/KRSC storage and the logical order.

Parity pins for every function live in tests/test_oracle_pins.py.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")


class OracleShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("N", "C", "H", "W", "K", "R", "S", "P", "Q",
                 "stride_h", "stride_w", "pad_h", "pad_w")]


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("oracle library not built: %s (run __graft_entry__.build())" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    dp = ctypes.POINTER(ctypes.c_double)
    u8p = ctypes.POINTER(ctypes.c_uint8)
    i64p = ctypes.POINTER(ctypes.c_int64)
    i32p = ctypes.POINTER(ctypes.c_int32)
    sp = ctypes.POINTER(OracleShape)
    lib.oracle_conv_fwd.argtypes = [sp, dp, dp, dp]
    lib.oracle_conv_fwd.restype = None
    lib.oracle_conv_bwd_data.argtypes = [sp, dp, dp, u8p, dp, dp, i64p]
    lib.oracle_conv_bwd_data.restype = None
    lib.oracle_conv_bwd_weight.argtypes = [sp, dp, dp, dp, dp, i64p]
    lib.oracle_conv_bwd_weight.restype = None
    lib.oracle_bwd_data_macs.argtypes = [sp, dp, u8p, i64p]
    lib.oracle_bwd_data_macs.restype = ctypes.c_int64
    lib.oracle_conv_bwd_data_at.argtypes = [sp, dp, dp, i32p, ctypes.c_int64, dp, dp, i64p]
    lib.oracle_conv_bwd_data_at.restype = None
    lib.oracle_conv_bwd_weight_at.argtypes = [sp, dp, dp, i32p, ctypes.c_int64, dp, dp, i64p]
    lib.oracle_conv_bwd_weight_at.restype = None
    lib.oracle_conv_fwd_at.argtypes = [sp, dp, dp, i32p, ctypes.c_int64, dp, dp, i64p]
    lib.oracle_conv_fwd_at.restype = None
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def num_threads():
    """OpenMP threads the oracle uses."""
    return _load().oracle_num_threads()


def out_size(h, r, stride, pad):
    return (h + 2 * pad - r) // stride + 1


def make_shape(N, C, H, W, K, R, S, stride=(1, 1), pad=(0, 0)):
    P = out_size(H, R, stride[0], pad[0])
    Q = out_size(W, S, stride[1], pad[1])
    if P <= 0 or Q <= 0:
        raise ValueError("empty output")
    return OracleShape(N, C, H, W, K, R, S, P, Q, stride[0], stride[1], pad[0], pad[1])


def _dptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


# ---------------------------------------------------------------- convolution

def conv_fwd(x, w, stride=(1, 1), pad=(0, 0)):
    """Forward convolution (Sec. II-A).  x [N,C,H,W], w [K,C,R,S] -> y [N,K,P,Q]."""
    x, w = _f64(x), _f64(w)
    N, C, H, W_ = x.shape
    K, C2, R, S = w.shape
    assert C == C2
    sh = make_shape(N, C, H, W_, K, R, S, stride, pad)
    y = np.empty((N, K, sh.P, sh.Q), np.float64)
    _load().oracle_conv_fwd(ctypes.byref(sh), _dptr(x), _dptr(w), _dptr(y))
    return y


def relu(z):
    """The ReLU as the footprint definition reads it (Sec. III-B): z where
    z > 0, else +0.0 (so non-positive and NaN inputs give +0.0)."""
    z = np.asarray(z, dtype=np.float64)
    return np.where(z > 0, z, 0.0)


def conv_fwd_relu(x, w, stride=(1, 1), pad=(0, 0)):
    """Forward convolution followed by the ReLU (Sec. II-A; the ReLU output is
    the activation whose footprint the backward pass consumes, Sec. III-B).
    Returns (z, y, abs_sum, nterms): z = conv_fwd(x, w), y = relu(z), and per
    output the sum of |x*w| over its terms and their number (the
    conditioning of each sum, for error bounds)."""
    z = conv_fwd(x, w, stride, pad)
    a = conv_fwd(np.abs(_f64(x)), np.abs(_f64(w)), stride, pad)
    n = conv_fwd(np.ones(np.shape(x)), np.ones(np.shape(w)), stride, pad)
    return z, relu(z), a, np.rint(n).astype(np.int64)


def conv_fwd_at(x, w, coords, stride=(1, 1), pad=(0, 0)):
    """Forward convolution at sampled (n,k,p,q) coordinates.
    Returns (values, sum|X*W|, number of terms)."""
    x, w = _f64(x), _f64(w)
    N, C, H, W_ = x.shape
    K, _, R, S = w.shape
    sh = make_shape(N, C, H, W_, K, R, S, stride, pad)
    c, cp = _coords(coords)
    m = len(c)
    out, absd, nt = np.empty(m), np.empty(m), np.empty(m, np.int64)
    _load().oracle_conv_fwd_at(ctypes.byref(sh), _dptr(x), _dptr(w), cp, m, _dptr(out), _dptr(absd),
                               nt.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)))
    return out, absd, nt


def conv_bwd_data(dy, w, hw, stride=(1, 1), pad=(0, 0), mask=None, with_bound=False):
    """Data gradient, dense or masked (Sec. III-B output sparsity, Sec. IV-B).

    dy [N,K,P,Q], w [K,C,R,S], hw = (H, W).  mask: None or a bool/uint8 array
    [N,C,H,W]; killed outputs come back as +0.0.  with_bound: also return the
    per-output sum of |dY*W| and the number of terms.
    """
    dy, w = _f64(dy), _f64(w)
    N, K, P, Q = dy.shape
    K2, C, R, S = w.shape
    assert K == K2
    sh = make_shape(N, C, hw[0], hw[1], K, R, S, stride, pad)
    assert (sh.P, sh.Q) == (P, Q), "dY spatial size does not match stride/pad"
    dx = np.empty((N, C, hw[0], hw[1]), np.float64)
    mptr = None
    if mask is not None:
        m = np.ascontiguousarray(np.asarray(mask) != 0, dtype=np.uint8)
        assert m.shape == dx.shape
        mptr = m.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))
    absd = nt = None
    if with_bound:
        absd = np.empty_like(dx)
        nt = np.empty(dx.shape, np.int64)
    _load().oracle_conv_bwd_data(
        ctypes.byref(sh), _dptr(dy), _dptr(w), mptr, _dptr(dx),
        _dptr(absd) if with_bound else None,
        nt.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)) if with_bound else None)
    if with_bound:
        return dx, absd, nt
    return dx


def conv_bwd_weight(x, dy, rs, stride=(1, 1), pad=(0, 0), with_bound=False):
    """Weight gradient (Sec. IV-B).  x [N,C,H,W], dy [N,K,P,Q] -> dw [K,C,R,S]."""
    x, dy = _f64(x), _f64(dy)
    N, C, H, W_ = x.shape
    N2, K, P, Q = dy.shape
    assert N == N2
    sh = make_shape(N, C, H, W_, K, rs[0], rs[1], stride, pad)
    assert (sh.P, sh.Q) == (P, Q)
    dw = np.empty((K, C, rs[0], rs[1]), np.float64)
    absd = nt = None
    if with_bound:
        absd = np.empty_like(dw)
        nt = np.empty(dw.shape, np.int64)
    _load().oracle_conv_bwd_weight(
        ctypes.byref(sh), _dptr(x), _dptr(dy), _dptr(dw),
        _dptr(absd) if with_bound else None,
        nt.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)) if with_bound else None)
    if with_bound:
        return dw, absd, nt
    return dw


def bwd_data_macs(dy, hw, rs, C, stride=(1, 1), pad=(0, 0), mask=None, per_output=False):
    """MAC count of the data gradient under the paper's compute model
    (Sec. II-A; Fig. "Compaction" example, Sec. III-B): 0 for a killed
    output, one per in-range tap with a non-zero dY operand otherwise."""
    dy = _f64(dy)
    N, K, P, Q = dy.shape
    sh = make_shape(N, C, hw[0], hw[1], K, rs[0], rs[1], stride, pad)
    assert (sh.P, sh.Q) == (P, Q)
    mptr = None
    if mask is not None:
        m = np.ascontiguousarray(np.asarray(mask) != 0, dtype=np.uint8)
        assert m.shape == (N, C, hw[0], hw[1])
        mptr = m.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))
    per = np.empty((N, C, hw[0], hw[1]), np.int64) if per_output else None
    total = _load().oracle_bwd_data_macs(
        ctypes.byref(sh), _dptr(dy), mptr,
        per.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)) if per_output else None)
    return (total, per) if per_output else total


def _coords(coords):
    c = np.ascontiguousarray(np.asarray(coords, dtype=np.int32).reshape(-1, 4))
    return c, c.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def conv_bwd_data_at(dy, w, hw, coords, stride=(1, 1), pad=(0, 0)):
    """Dense data gradient at sampled (n,c,h,w) coordinates.
    Returns (values, sum|dY*W|, number of terms)."""
    dy, w = _f64(dy), _f64(w)
    N, K, P, Q = dy.shape
    _, C, R, S = w.shape
    sh = make_shape(N, C, hw[0], hw[1], K, R, S, stride, pad)
    assert (sh.P, sh.Q) == (P, Q)
    c, cp = _coords(coords)
    m = len(c)
    out, absd, nt = np.empty(m), np.empty(m), np.empty(m, np.int64)
    _load().oracle_conv_bwd_data_at(ctypes.byref(sh), _dptr(dy), _dptr(w), cp, m,
                                    _dptr(out), _dptr(absd),
                                    nt.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)))
    return out, absd, nt


def conv_bwd_weight_at(x, dy, rs, coords, stride=(1, 1), pad=(0, 0)):
    """Weight gradient at sampled (k,c,r,s) coordinates."""
    x, dy = _f64(x), _f64(dy)
    N, C, H, W_ = x.shape
    _, K, P, Q = dy.shape
    sh = make_shape(N, C, H, W_, K, rs[0], rs[1], stride, pad)
    assert (sh.P, sh.Q) == (P, Q)
    c, cp = _coords(coords)
    m = len(c)
    out, absd, nt = np.empty(m), np.empty(m), np.empty(m, np.int64)
    _load().oracle_conv_bwd_weight_at(ctypes.byref(sh), _dptr(x), _dptr(dy), cp, m,
                                      _dptr(out), _dptr(absd),
                                      nt.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)))
    return out, absd, nt


# ------------------------------------------------------- masks and indexing

def relu_mask(x):
    """ReLU derivative as used for output sparsity: live iff x > 0.

    The boxed derivative of Sec. III-B gives 1 at z >= 0 on the
    pre-activation, while the same section (and the introduction) says the
    gradient footprint is identical to that of the ReLU *output*; the two
    differ only where the pre-activation is exactly 0.  The reading taken
    here is the output footprint: live iff the ReLU output is > 0.
    """
    return np.asarray(x) > 0


def maxpool2x2(a):
    """2x2 max-pool, stride 2, over the spatial axes of an [N][C][H][W]
    tensor with even H and W (the pooling between the VGG-16 stages, the
    network of the paper's layer-wise results in Sec. VI).  Returns (pooled,
    arg): arg[n,c,i,j] in 0..3 is the row-major window position of the first
    maximum, the position max-pool backward routes the gradient to."""
    a = np.asarray(a, dtype=np.float64)
    N, C, H, W = a.shape
    assert H % 2 == 0 and W % 2 == 0
    pooled = np.empty((N, C, H // 2, W // 2))
    arg = np.empty((N, C, H // 2, W // 2), np.int64)
    for i in range(H // 2):
        for j in range(W // 2):
            win = np.stack([a[:, :, 2 * i, 2 * j], a[:, :, 2 * i, 2 * j + 1],
                            a[:, :, 2 * i + 1, 2 * j], a[:, :, 2 * i + 1, 2 * j + 1]], axis=-1)
            arg[:, :, i, j] = np.argmax(win, axis=-1)   # first maximum
            pooled[:, :, i, j] = np.max(win, axis=-1)
    return pooled, arg


def maxpool2x2_backward(g, arg):
    """Max-pool backward: each pooled gradient g[n,c,i,j] goes to window
    position arg[n,c,i,j] of the 2x2 window, every other position gets 0."""
    g = np.asarray(g, dtype=np.float64)
    N, C, h, w = g.shape
    out = np.zeros((N, C, 2 * h, 2 * w))
    for pos in range(4):
        sel = arg == pos
        out[:, :, pos // 2::2, pos % 2::2] = np.where(sel, g, 0.0)
    return out


def weight_block_liveness(x_live, dy_live, rs, stride, pad, chunk, ktile, ctile, tpg):
    """Which blocks of the weight-gradient GEMM have a non-zero in both of
    their operands (input sparsity in the weight-gradient phase: a block whose
    dY operand or whose X operand is entirely zero contributes only zero
    products, so it can be skipped; a live block may still have only zero
    products when the non-zeros of its two operands do not meet).

    x_live [N][C][H][W] and dy_live [N][K][P][Q] are boolean footprints.
    Output pixels are taken in (n, p, q) order and cut into chunks of
    `chunk`; output channels into tiles of `ktile`; input channels into
    tiles of `ctile`; filter taps (r*S + s) into groups of `tpg`.  Block
    (g, ct, kt, b) is live iff dY is non-zero somewhere in chunk b x k tile
    kt AND X is non-zero somewhere at the chunk's pixels shifted by one of
    the group's taps (inside the image) x channel tile ct.
    Returns bool [groups][ctiles][ktiles][chunks]."""
    x_live, dy_live = np.asarray(x_live, bool), np.asarray(dy_live, bool)
    N, C, H, W = x_live.shape
    _, K, P, Q = dy_live.shape
    R, S = rs
    npq = N * P * Q
    nch = -(-npq // chunk)
    nkt, nct, ngr = -(-K // ktile), -(-C // ctile), -(-(R * S) // tpg)
    n_i, p_i, q_i = np.meshgrid(np.arange(N), np.arange(P), np.arange(Q), indexing="ij")
    n_i, p_i, q_i = n_i.ravel(), p_i.ravel(), q_i.ravel()       # pixel order (n, p, q)
    blk = np.arange(npq) // chunk
    dy_pix = dy_live.transpose(0, 2, 3, 1).reshape(npq, K)
    dy_any = np.zeros((nch, nkt), bool)
    for kt in range(nkt):
        np.logical_or.at(dy_any[:, kt], blk, dy_pix[:, kt * ktile:(kt + 1) * ktile].any(axis=1))
    x_any = np.zeros((ngr, nct, nch), bool)
    for tap in range(R * S):
        r, s = divmod(tap, S)
        h = p_i * stride[0] - pad[0] + r
        w = q_i * stride[1] - pad[1] + s
        inside = (h >= 0) & (h < H) & (w >= 0) & (w < W)
        for ct in range(nct):
            v = np.zeros(npq, bool)
            sub = x_live[:, ct * ctile:(ct + 1) * ctile]
            v[inside] = sub[n_i[inside], :, h[inside], w[inside]].any(axis=1)
            np.logical_or.at(x_any[tap // tpg, ct], blk, v)
    return x_any[:, :, None, :] & dy_any.T[None, None, :, :]


def pack_bits(live_linear):
    """Bit i of 32-bit word i//32 = live_linear[i] (little-endian bit order),
    trailing bits of the last word 0.  This is the output bitmap of
    Sec. IV-B stored one bit per element in the tensor's own linear order."""
    b = np.asarray(live_linear, dtype=bool).reshape(-1)
    nwords = (b.size + 31) // 32
    padded = np.zeros(nwords * 32, dtype=bool)
    padded[: b.size] = b
    by = np.packbits(padded.reshape(-1, 8), axis=1, bitorder="little").reshape(-1)
    return by.view("<u4").astype(np.uint32)


def unpack_bits(words, count):
    by = np.asarray(words, dtype="<u4").view(np.uint8)
    return np.unpackbits(by, bitorder="little")[:count].astype(bool)


def relu_mask_bits(x_linear):
    """The packed ReLU bitmap of a tensor given in its storage order."""
    return pack_bits(relu_mask(x_linear).reshape(-1))


def live_pixel_lists(bits, npix, C, G):
    """Non-zero indexing of the output bitmap per channel group (the GPU
    analogue of the offset map of Sec. IV-B): for channel group g
    (channels [g*G, min((g+1)*G, C))) the ascending list of pixels with at
    least one live channel.  bits is in NHWC order (pixel-major).
    Returns a list of int32 arrays, one per group."""
    live = unpack_bits(bits, npix * C).reshape(npix, C)
    ngroups = (C + G - 1) // G
    out = []
    for g in range(ngroups):
        anyl = live[:, g * G: min((g + 1) * G, C)].any(axis=1)
        out.append(np.nonzero(anyl)[0].astype(np.int32))
    return out


def block_occupancy(dy_pixel_major, chunk, KG):
    """occ[j][g] = 1 iff some dY value in pixels [j*chunk, (j+1)*chunk) and
    channels [g*KG, (g+1)*KG) is non-zero (+0.0 and -0.0 both count as zero).
    dy_pixel_major: [npix, K] (NHWC flattened over N,P,Q).  These are the
    blocks whose products the weight gradient may skip (input sparsity,
    Sec. III-B and Sec. VI)."""
    d = np.asarray(dy_pixel_major)
    npix, K = d.shape
    nz = d != 0
    nchunks = (npix + chunk - 1) // chunk
    ngroups = (K + KG - 1) // KG
    occ = np.zeros((nchunks, ngroups), np.uint8)
    for j in range(nchunks):
        blk = nz[j * chunk: (j + 1) * chunk]
        for g in range(ngroups):
            occ[j, g] = 1 if blk[:, g * KG: (g + 1) * KG].any() else 0
    return occ


# ---------------------------------------------------------- layout helpers

def nhwc_to_nchw(a):
    return np.ascontiguousarray(np.asarray(a).transpose(0, 3, 1, 2))


def nchw_to_nhwc(a):
    return np.ascontiguousarray(np.asarray(a).transpose(0, 2, 3, 1))


def krsc_to_kcrs(a):
    return np.ascontiguousarray(np.asarray(a).transpose(0, 3, 1, 2))


def kcrs_to_krsc(a):
    return np.ascontiguousarray(np.asarray(a).transpose(0, 2, 3, 1))
