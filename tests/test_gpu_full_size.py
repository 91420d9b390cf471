"""GPU parity at the full sizes of the five workloads (the benchmark's layer
included, in the launch configuration bench.py times).

The oracle evaluates the definitions at sampled output coordinates (random
ones plus every image border); values are compared with the same normwise
and per-element bounds as the full-tensor tests.  Over the whole tensors:
the zero pattern of dX against the footprint (exact), the masked kernel
against the dense kernel at live outputs (bitwise), and the skipping weight
gradient against the non-skipping one (bitwise).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2109_07710_amd as cb
import workloads as wl
from parity import check_dw_regrouped, check_values, dx_as_nchw, dx_bits_nchw, gpu_backward, tol_for

pytestmark = pytest.mark.gpu

NSAMPLE = 3000


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


def _dx_coords(spec, rng):
    n = rng.integers(0, spec.N, NSAMPLE)
    c = rng.integers(0, spec.C, NSAMPLE)
    h = rng.integers(0, spec.H, NSAMPLE)
    w = rng.integers(0, spec.W, NSAMPLE)
    pts = [np.stack([n, c, h, w], 1)]
    # borders (padding taps) of one image, two channels
    for hh in range(spec.H):
        for ww in (0, spec.W - 1):
            pts.append(np.array([[spec.N - 1, 0, hh, ww], [0, spec.C - 1, hh, ww]]))
    for ww in range(spec.W):
        for hh in (0, spec.H - 1):
            pts.append(np.array([[0, spec.C // 2, hh, ww]]))
    return np.concatenate(pts).astype(np.int32)


def _dw_coords(spec, rng):
    k = rng.integers(0, spec.K, NSAMPLE)
    c = rng.integers(0, spec.C, NSAMPLE)
    r = rng.integers(0, spec.R, NSAMPLE)
    s = rng.integers(0, spec.S, NSAMPLE)
    corners = [[kk, cc, rr, ss] for kk in (0, spec.K - 1) for cc in (0, spec.C - 1)
               for rr in range(spec.R) for ss in range(spec.S)]
    return np.concatenate([np.stack([k, c, r, s], 1), np.array(corners)]).astype(np.int32)


def _check_full(spec, flags_pairs=True):
    print("\n[case] full size %s N=%d C=%d K=%d %dx%d R=%d" % (spec.name, spec.N, spec.C, spec.K, spec.H, spec.W,
                                                            spec.R), flush=True)
    t = wl.draw(spec)
    gpu = gpu_backward(spec, t, dy_mask=True)
    rng = np.random.default_rng(2109)
    st, pd = (spec.stride, spec.stride), (spec.pad, spec.pad)
    x64 = oracle.nhwc_to_nchw(t["x"].double().numpy())
    dy64 = oracle.nhwc_to_nchw(t["dy"].double().numpy())
    w64 = oracle.krsc_to_kcrs(t["w"].double().numpy())
    tol = tol_for(spec.dtype)
    if spec.need_dx:
        mask = oracle.relu_mask(x64)
        bits = dx_bits_nchw(gpu["dx"])
        if spec.masked:
            assert not (bits[~mask] != 0).any(), "killed outputs must be +0.0"
        cx = _dx_coords(spec, rng)
        o, absd, nt = oracle.conv_bwd_data_at(dy64, w64, (spec.H, spec.W), cx, st, pd)
        live = mask[cx[:, 0], cx[:, 1], cx[:, 2], cx[:, 3]] if spec.masked else np.ones(len(cx), bool)
        o = np.where(live, o, 0.0)
        absd, nt = np.where(live, absd, 0.0), np.where(live, nt, 0)
        g = gpu["dx"].float().cpu().numpy()[cx[:, 0], cx[:, 2], cx[:, 3], cx[:, 1]].astype(np.float64)
        e = check_values(g, o, absd, nt, tol, spec.dtype == "bf16", spec.name + " dX (sampled)")
        print("  dX sampled normwise error %.3e" % e, flush=True)
        if spec.masked and flags_pairs:
            dense = gpu_backward(spec, t, masked=False)
            bd = dx_bits_nchw(dense["dx"])
            stats = cb.cbw_read_stats(gpu["desc"], cb.CBW_OP_BWD_DATA_MASKED, gpu["ws_dx"])
            if stats.rows_live == stats.rows_total:
                # same rows, same reduction split: identical bits
                assert np.array_equal(bits[mask], bd[mask]), "masked kernel differs from dense at live outputs"
            else:
                # compaction removed rows, so the reduction may be split differently
                gm = dx_as_nchw(gpu["dx"])[mask]
                dm = dx_as_nchw(dense["dx"])[mask]
                assert np.max(np.abs(gm - dm)) <= 2.0 ** -7 * max(np.max(np.abs(dm)), 1e-30)
    cw = _dw_coords(spec, rng)
    o, absw, ntw = oracle.conv_bwd_weight_at(x64, dy64, (spec.R, spec.S), cw, st, pd)
    g = gpu["dw"].cpu().numpy()[cw[:, 0], cw[:, 2], cw[:, 3], cw[:, 1]].astype(np.float64)
    e = check_values(g, o, absw, ntw, tol, False, spec.name + " dW (sampled)")
    print("  dW sampled normwise error %.3e" % e, flush=True)
    if flags_pairs:
        g2 = gpu_backward(spec, t, flags=cb.CBW_FLAG_NO_SKIP, dy_mask=True)
        sk = cb.cbw_read_stats(gpu["desc"], cb.CBW_OP_BWD_WEIGHT, gpu["ws_dw"]).blocks_skipped
        check_dw_regrouped(gpu["dw"], g2["dw"], sk, spec.name + " dW, skipping against not skipping")


def test_full_config2_bench_layer():
    _check_full(wl.config2()[0])


@pytest.mark.parametrize("layer", [0, 1, 2])
def test_full_config3_bottleneck(layer):
    _check_full(wl.config3()[layer])


@pytest.mark.parametrize("kind,d", [("bernoulli", 0.1), ("bernoulli", 0.9), ("clustered", 0.5),
                                    ("channel_shared", 0.3)])
def test_full_config4_sweep_points(kind, d):
    _check_full(wl.config4(d, kind)[0])


@pytest.mark.parametrize("layer", [3, 4, 7, 12])
def test_full_config5_vgg_layers(layer):
    _check_full(wl.config5()[layer - 1])


@pytest.mark.parametrize("layer", [3, 11])
def test_full_config5_pooled_mask(layer):
    """conv2_1 and conv5_1 at full size with the pooled > 0 mask."""
    _check_full(wl.config5(pooled_mask=True)[layer - 1])


def test_full_spatial_config5_conv1_2():
    """conv1_2 at its full 224 x 224 size (64 -> 64 channels) with 4 of the 32
    images, to keep input generation short."""
    _check_full(wl.config5(N=4)[1], flags_pairs=False)


def test_full_config5_first_layer_padded_image():
    """conv1_1 reads the 3-channel image.  C = 3 is not a multiple of the
    16-byte vector, which the library reports instead of computing; the
    workload stores the image with its channels zero-padded to 8, and the
    weight gradient of the padding must come out exactly zero.  Full 224 x 224
    size with 4 of the 32 images."""
    spec = wl.config5(N=4)[0]
    d3 = cb.ConvDesc.make(spec.N, 3, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad)
    assert cb.cbw_validate_desc(d3) == cb.CBW_ERR_UNSUPPORTED
    assert spec.C == 8 and spec.extra["true_c"] == 3 and not spec.need_dx
    _check_full(spec, flags_pairs=False)
    t = wl.draw(spec)
    gpu = gpu_backward(spec, t, dy_mask=True)
    assert not gpu["dw"][..., 3:].any().item(), "weight gradient of the zero channels"
