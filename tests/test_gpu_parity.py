"""GPU parity: the HIP path through the C-ABI against the fp64 oracle.

Full-tensor comparisons run at sizes the oracle finishes in seconds but that
span several tiles and a ragged tail; the full-size layers the benchmark
times are checked on sampled outputs (see test_gpu_full_size.py).  Every test
prints its case before the first GPU call.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
import paper_2109_07710_amd as cb
import workloads as wl
from parity import (check_layer, check_values, check_zero_pattern, desc_of, dw_as_kcrs, dx_as_nchw,
                    dx_bits_nchw, gpu_backward, oracle_backward, tol_for)

pytestmark = pytest.mark.gpu


def _case(msg):
    print("\n[case] " + msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


def _run_and_check(spec, **kw):
    _case("%s N=%d C=%d K=%d %dx%d R=%d stride=%d pad=%d %s %s" % (
        spec.name, spec.N, spec.C, spec.K, spec.H, spec.W, spec.R, spec.stride, spec.pad, spec.dtype, kw))
    t = wl.draw(spec)
    gpu = gpu_backward(spec, t, **{k: v for k, v in kw.items() if k in ("flags", "masked", "dy_mask", "w_layout")})
    ref = oracle_backward(spec, t, masked=kw.get("masked"))
    return check_layer(spec, t, gpu, ref, masked=kw.get("masked"), w_layout=kw.get("w_layout", "krsc")), gpu, t


# ----------------------------------------------------------------- configs

def test_config1_fp32():
    spec = wl.config1()[0]
    errs, _, _ = _run_and_check(spec)
    print(errs)


@pytest.mark.parametrize("flags", [0, cb.CBW_FLAG_NO_SKIP])
def test_config2_reduced(flags):
    spec = wl.config2(N=2, H=20)[0]  # 800 pixels: 7 pixel tiles, ragged tail of 32; 2 channel tiles
    errs, _, _ = _run_and_check(spec, flags=flags, dy_mask=(flags == 0))
    print(errs)


def test_config2_dense_path():
    spec = wl.config2(N=1, H=18)[0]
    errs, _, _ = _run_and_check(spec, masked=False)
    print(errs)


@pytest.mark.parametrize("layer", [0, 1, 2])
def test_config3_bottleneck_reduced(layer):
    spec = wl.config3(N=2, H=12)[layer]
    errs, _, _ = _run_and_check(spec, dy_mask=True)
    print(errs)


@pytest.mark.parametrize("kind,d", [("bernoulli", 0.1), ("bernoulli", 0.5), ("clustered", 0.3),
                                    ("clustered", 0.9), ("channel_shared", 0.2)])
def test_config4_sweep_reduced(kind, d):
    spec = wl.config4(d, kind, N=2, H=14)[0]
    errs, _, _ = _run_and_check(spec)
    print(errs)


@pytest.mark.parametrize("layer", [2, 3, 4, 9, 12])
def test_config5_vgg_layers_reduced(layer):
    spec = wl.config5(N=1, scale=8)[layer - 1]
    errs, _, _ = _run_and_check(spec)
    print(errs)


@pytest.mark.parametrize("layer", [3, 5, 8, 11])
def test_config5_pooled_mask_reduced(layer):
    """The four layers after a max-pool with their data gradient masked by
    pooled > 0 (the pooled ReLU output is the conv's X)."""
    spec = wl.config5(N=2, scale=8, pooled_mask=True)[layer - 1]
    assert spec.masked and spec.x_kind == "pooled_gauss"
    errs, _, _ = _run_and_check(spec)
    print(errs)


# ------------------------------------------------------- shapes / strides

def _shape_cases():
    out = []
    for (R, S), st, pad, (C, K), dt in itertools.product([(1, 1), (3, 3), (5, 5), (3, 1)], [1, 2, 3], [0, 1, 2],
                                                          [(16, 24), (136, 8)], ["bf16", "f32"]):
        H, W = 11, 9
        if (H + 2 * pad - R) // st + 1 <= 0 or (W + 2 * pad - S) // st + 1 <= 0:
            continue
        out.append((R, S, st, pad, C, K, dt))
    return out[::5]


@pytest.mark.parametrize("R,S,st,pad,C,K,dt", _shape_cases())
def test_strides_pads_shapes(R, S, st, pad, C, K, dt):
    spec = wl.LayerSpec("shape_sweep", 9, 0, N=2, C=C, H=11, W=9, K=K, R=R, S=S, stride=st, pad=pad, dtype=dt,
                        x_kind="shifted_gauss", x_param=0.1, dy_kind="bernoulli", dy_param=0.5)
    _run_and_check(spec)


@pytest.mark.parametrize("C,K,R,S", [(8, 64, 3, 3), (24, 72, 3, 3), (96, 136, 3, 3), (16, 200, 5, 5),
                                     (128, 64, 3, 3), (40, 128, 3, 2), (64, 64, 1, 1)])
def test_narrow_channel_tilings(C, K, R, S):
    """Layer widths that select the narrow tiles: channel tiles of 64 or 128,
    output-channel tiles of 64 or 128 in the weight gradient, and filter taps
    packed into one channel tile (C <= 128, with columns past the packed taps
    left empty, e.g. C = 96 or 40)."""
    spec = wl.LayerSpec("narrow", 9, 1, N=2, C=C, H=13, W=11, K=K, R=R, S=S, stride=1, pad=R // 2,
                        dtype="bf16", x_kind="shifted_gauss", x_param=0.1, dy_kind="bernoulli", dy_param=0.5)
    _run_and_check(spec)


def test_kcrs_filter_layout():
    spec = wl.config2(N=1, H=10)[0]
    _run_and_check(spec, w_layout="kcrs")


# ------------------------------------------------------- exact properties

def test_masked_equals_dense_times_mask_bitwise():
    """Output sparsity changes which outputs are computed, not their values:
    the gathered kernel reproduces the dense kernel's bits at live outputs."""
    spec = wl.config4(0.3, "clustered", N=2, H=14)[0]
    _case(spec.name)
    t = wl.draw(spec)
    g_m = gpu_backward(spec, t, masked=True)
    g_d = gpu_backward(spec, t, masked=False)
    g_s = gpu_backward(spec, t, masked=True, flags=cb.CBW_FLAG_NO_SKIP)
    mask = oracle.relu_mask(oracle.nhwc_to_nchw(t["x"].float().numpy()))
    bm, bd, bs = dx_bits_nchw(g_m["dx"]), dx_bits_nchw(g_d["dx"]), dx_bits_nchw(g_s["dx"])
    assert np.array_equal(bm[mask], bd[mask])
    assert np.array_equal(bm, bs)
    assert np.all(bm[~mask] == 0)
    assert torch.equal(g_m["dw"], g_s["dw"])


def test_run_twice_bitwise_deterministic():
    spec = wl.config2(N=1, H=16)[0]
    _case(spec.name)
    t = wl.draw(spec)
    a = gpu_backward(spec, t, dy_mask=True)
    b = gpu_backward(spec, t, dy_mask=True)
    assert torch.equal(a["dx"].view(torch.int16), b["dx"].view(torch.int16))
    assert torch.equal(a["dw"].view(torch.int32), b["dw"].view(torch.int32))


def test_relu_mask_pack_exact():
    _case("mask pack special values")
    vals = [0.0, -0.0, 1.0, -1.0, float("nan"), float("inf"), -float("inf"), 1e-40, -1e-40, 3e-38]
    for dtype, tdt in (("bf16", torch.bfloat16), ("f32", torch.float32)):
        for n in (1, 8, 31, 32, 33, 1000, 4099):
            base = torch.tensor(vals * (n // len(vals) + 1), dtype=torch.float32)[:n]
            # NHWC tensor with C = 8: pad the element count up to whole pixels
            C = 8
            npx = (n + C - 1) // C
            x = torch.zeros(npx * C, dtype=torch.float32)
            x[:n] = base
            x = x.to(tdt)
            desc = cb.ConvDesc.make(1, C, 1, npx, 8, 1, 1, dtype=dtype)
            xm = torch.full((cb.cbw_mask_words(desc),), -1, dtype=torch.int32, device="cuda")
            cb.cbw_relu_mask_pack(desc, x.view(1, 1, npx, C).cuda(), xm)
            ref = oracle.relu_mask_bits(x.float().numpy())
            assert np.array_equal(xm.cpu().numpy().view(np.uint32), ref), (dtype, n)
            bits = torch.full((cb.cbw_mask_words(desc),), -1, dtype=torch.int32, device="cuda")
            cb.cbw_nonzero_mask_pack(desc.dtype, x.numel(), x.cuda(), bits)
            ref_nz = oracle.pack_bits(x.float().numpy() != 0)
            assert np.array_equal(bits.cpu().numpy().view(np.uint32), ref_nz), (dtype, n)


@pytest.mark.parametrize("C", [256, 128, 64])
@pytest.mark.parametrize("kind,d", [("bernoulli", 0.01), ("clustered", 0.2), ("channel_shared", 0.3)])
def test_compaction_lists_exact(kind, d, C):
    """Live lists per channel group (the group is the tile's channel width:
    256, 128 or 64 channels) equal the oracle's, and so do the row counts."""
    spec = wl.config4(d, kind, N=2, H=14)[0]
    spec.C = spec.K = C
    _case("compaction %s d=%.2f C=%d" % (kind, d, C))
    t = wl.draw(spec)
    gpu = gpu_backward(spec, t)
    desc = gpu["desc"]
    npix = spec.N * spec.H * spec.W
    bits = gpu["xmask"].cpu().numpy().view(np.uint32)
    assert np.array_equal(bits, oracle.relu_mask_bits(t["x"].float().numpy()))
    lst0, G = cb.cbw_read_live_lists(desc, gpu["ws_dx"], 0)
    ref = oracle.live_pixel_lists(bits, npix, spec.C, G)
    for g in range(len(ref)):
        got, _ = cb.cbw_read_live_lists(desc, gpu["ws_dx"], g)
        assert np.array_equal(got, ref[g]), g
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_DATA_MASKED, gpu["ws_dx"])
    assert st.rows_live == sum(len(r) for r in ref)
    assert st.rows_total == len(ref) * npix


@pytest.mark.parametrize("use_bits", [False, True])
def test_occupancy_and_block_skip(use_bits):
    """A dY with whole zero blocks: the occupancy map equals the oracle's and
    the skipped blocks do not change dW."""
    spec = wl.config2(N=2, H=16)[0]
    _case("occupancy bits=%s" % use_bits)
    t = wl.draw(spec)
    dy = t["dy"].clone()
    npq = spec.N * spec.P * spec.Q
    flat = dy.view(npq, spec.K)
    flat[0:300, 0:128] = 0        # zero blocks in the first k tile
    flat[260:512, :] = 0          # and whole chunks
    t["dy"] = dy
    gpu = gpu_backward(spec, t, dy_mask=use_bits)
    occ, chunk, kw = cb.cbw_read_occupancy(gpu["desc"], gpu["ws_dw"])
    ref = oracle.block_occupancy(flat.float().numpy(), chunk, kw)
    assert np.array_equal(occ, ref)
    st = cb.cbw_read_stats(gpu["desc"], cb.CBW_OP_BWD_WEIGHT, gpu["ws_dw"])
    assert st.blocks_total == ref.size and st.blocks_skipped == int((ref == 0).sum()) > 0
    ref_full = oracle_backward(spec, t)
    check_values(dw_as_kcrs(gpu["dw"]), ref_full["dw"], ref_full["dw_abs"], ref_full["dw_n"], tol_for("bf16"),
                 False, "dW with skipped blocks")
    g2 = gpu_backward(spec, t, flags=cb.CBW_FLAG_NO_SKIP)
    assert torch.equal(gpu["dw"], g2["dw"])


def test_guard_bands_untouched():
    """Outputs are written only inside their extent."""
    spec = wl.config2(N=1, H=13)[0]
    _case(spec.name + " guard bands")
    t = wl.draw(spec)
    desc = desc_of(spec)
    pad = 4096
    d = {k: v.cuda() for k, v in t.items()}
    xm = torch.zeros(cb.cbw_mask_words(desc), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, d["x"], xm)
    nx = d["x"].numel()
    buf = torch.full((nx + 2 * pad,), float("nan"), dtype=torch.bfloat16, device="cuda")
    dx = buf[pad:pad + nx].view(d["x"].shape)
    ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED)
    cb.conv_bwd_data_masked(desc, d["dy"], d["w"], xm, dx, ws)
    nw = spec.K * spec.R * spec.S * spec.C
    wbuf = torch.full((nw + 2 * pad,), float("nan"), dtype=torch.float32, device="cuda")
    dw = wbuf[pad:pad + nw]
    ws2 = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT)
    cb.conv_bwd_weight_sparse(desc, d["x"], d["dy"], None, dw, ws2)
    torch.cuda.synchronize()
    assert torch.isnan(buf[:pad].float()).all() and torch.isnan(buf[pad + nx:].float()).all()
    assert torch.isnan(wbuf[:pad]).all() and torch.isnan(wbuf[pad + nw:]).all()
    assert not torch.isnan(dx.float()).any() and not torch.isnan(dw).any()


def test_errors_raise_before_launch():
    spec = wl.config2(N=1, H=8)[0]
    _case("error paths")
    desc = desc_of(spec)
    t = {k: v.cuda() for k, v in wl.draw(spec).items()}
    xm = torch.zeros(cb.cbw_mask_words(desc), dtype=torch.int32, device="cuda")
    dx = torch.full_like(t["x"], 7.0)
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(cb.CbwError) as e:
        cb.conv_bwd_data_masked(desc, t["dy"], t["w"], xm, dx, small)
    assert e.value.status == cb.CBW_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert (dx.float() == 7.0).all()
    bad = desc_of(spec)
    bad.P += 1
    ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED)
    with pytest.raises(cb.CbwError) as e:
        cb.conv_bwd_data_masked(bad, t["dy"], t["w"], xm, dx, ws)
    assert e.value.status == cb.CBW_ERR_INVALID_ARG
    with pytest.raises(cb.CbwError) as e:
        cb.conv_bwd_data_masked(desc, t["dy"], t["w"], None, dx, ws)
    assert e.value.status == cb.CBW_ERR_INVALID_ARG
    mis = torch.empty(t["x"].numel() + 8, dtype=torch.bfloat16, device="cuda")[1:1 + t["x"].numel()]
    with pytest.raises(cb.CbwError) as e:
        cb.conv_bwd_data_masked(desc, t["dy"], t["w"], xm, mis, ws)
    assert e.value.status == cb.CBW_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert (dx.float() == 7.0).all()
