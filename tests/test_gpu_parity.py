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
from parity import (check_dw_regrouped, check_layer, check_values, check_zero_pattern, desc_of, dw_as_kcrs,
                    dx_as_nchw, dx_bits_nchw, gpu_backward, oracle_backward, oracle_inputs, to_dev, tol_for)

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
    sk = cb.cbw_read_stats(g_m["desc"], cb.CBW_OP_BWD_WEIGHT, g_m["ws_dw"]).blocks_skipped
    check_dw_regrouped(g_m["dw"], g_s["dw"], sk, "dW")


def test_run_twice_bitwise_deterministic():
    spec = wl.config2(N=1, H=16)[0]
    _case(spec.name)
    t = wl.draw(spec)
    a = gpu_backward(spec, t, dy_mask=True)
    b = gpu_backward(spec, t, dy_mask=True)
    assert torch.equal(a["dx"].view(torch.int16), b["dx"].view(torch.int16))
    assert torch.equal(a["dw"].view(torch.int32), b["dw"].view(torch.int32))


def test_gather_sequence_shared_workspace():
    """One workspace over calls whose footprints alternate between every
    pixel live and some pixels dead, starting from a zeroed and from a
    0xff-filled workspace: each call's data gradient equals the dense
    kernel's bits at live outputs and zero elsewhere, whatever the previous
    call left behind (the per-group dead-pixel flags it raised or lowered)."""
    spec = wl.config4(0.3, "clustered", N=2, H=14)[0]
    _case("gather sequence " + spec.name)
    t = wl.draw(spec)
    desc = desc_of(spec)
    d = to_dev(t)
    x_live = d["x"].abs() + 0.125   # every element positive: every pixel live
    dx_ref = torch.empty_like(d["x"])
    cb.conv_bwd_data(desc, d["dy"], d["w"], dx_ref, cb.workspace(desc, cb.CBW_OP_BWD_DATA, "cuda"))
    ref_bits = dx_bits_nchw(dx_ref)
    dw = torch.empty((spec.K, spec.R, spec.S, spec.C), dtype=torch.float32, device="cuda")
    for fill in (0, 255):
        ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED, "cuda")
        ws_b = cb.workspace(desc, cb.CBW_OP_BWD_BOTH, "cuda")
        ws.fill_(fill)
        ws_b.fill_(fill)
        for i, x in enumerate((x_live, d["x"], x_live, d["x"], d["x"], x_live)):
            xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
            cb.cbw_relu_mask_pack(desc, x, xm)
            mask = oracle.relu_mask(oracle.nhwc_to_nchw(x.float().cpu().numpy()))
            for both in (False, True):
                dx = torch.full_like(d["x"], float("nan"))
                if both:
                    cb.conv_bwd_sparse(desc, x, d["dy"], d["w"], xm, None, dx, dw, ws_b, 0)
                else:
                    cb.conv_bwd_data_masked(desc, d["dy"], d["w"], xm, dx, ws, 0)
                torch.cuda.synchronize()
                bits = dx_bits_nchw(dx)
                assert np.array_equal(bits[mask], ref_bits[mask]), (fill, i, both)
                assert np.all(bits[~mask] == 0), (fill, i, both)


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
    spec.C, spec.K = C, 2 * C   # K != 64 when C = 64: the 3 x 3 layers with C = K = 64 list nothing
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
    tiles = spec.R * spec.S          # C = 256: one tap per tile, one channel tile
    assert st.blocks_total == ref.size * tiles and st.blocks_skipped == int((ref == 0).sum()) * tiles > 0
    # work redistribution: tile t (k tile t % ktiles) executes each live block
    # once, no split more than ceil(live / nsplit)
    work = cb.cbw_read_weight_work(gpu["desc"], gpu["ws_dw"])
    nsplit, ntiles = work.shape
    live_t = np.array([int(ref[:, t % ref.shape[1]].sum()) for t in range(ntiles)])
    assert np.array_equal(work.sum(axis=0), live_t)
    assert np.array_equal(work.max(axis=0), -(-live_t // nsplit))
    ref_full = oracle_backward(spec, t)
    check_values(dw_as_kcrs(gpu["dw"]), ref_full["dw"], ref_full["dw_abs"], ref_full["dw_n"], tol_for("bf16"),
                 False, "dW with skipped blocks")
    g2 = gpu_backward(spec, t, flags=cb.CBW_FLAG_NO_SKIP)
    check_dw_regrouped(gpu["dw"], g2["dw"], st.blocks_skipped, "dW with skipped blocks")


@pytest.mark.parametrize("pattern", ["last_image_live", "first_image_live", "odd_images_live"])
def test_balanced_split_long_dead_runs(pattern):
    """Configuration 2's layer with dY zero over whole images: runs of dead
    chunks far longer than one split (and than the cached liveness window of
    1024 chunks) open or close the balanced ranges.  Each tile's live blocks
    are executed once, shared so no split runs more than ceil(live / nsplit);
    dW agrees with the unskipped run and, at sampled entries, the oracle."""
    spec = wl.config2()[0]
    _case("balanced split " + pattern)
    t = wl.draw(spec)
    dy = t["dy"].clone()
    keep = {"last_image_live": [spec.N - 1], "first_image_live": [0],
            "odd_images_live": list(range(1, spec.N, 2))}[pattern]
    dead = torch.ones(spec.N, dtype=torch.bool)
    dead[keep] = False
    dy[dead] = 0
    t["dy"] = dy
    gpu = gpu_backward(spec, t, dy_mask=True)
    desc = gpu["desc"]
    occ, chunk, kw = cb.cbw_read_occupancy(desc, gpu["ws_dw"])
    npq = spec.N * spec.P * spec.Q
    ref = oracle.block_occupancy(dy.view(npq, spec.K).float().numpy(), chunk, kw)
    assert np.array_equal(occ, ref)
    work = cb.cbw_read_weight_work(desc, gpu["ws_dw"])
    nsplit, ntiles = work.shape
    live_t = np.array([int(ref[:, j % ref.shape[1]].sum()) for j in range(ntiles)])
    assert np.array_equal(work.sum(axis=0), live_t)
    assert np.array_equal(work.max(axis=0), -(-live_t // nsplit))
    if pattern != "odd_images_live":      # a dead run longer than the cached window
        assert occ.shape[0] - live_t.max() > 1024
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, gpu["ws_dw"])
    assert st.blocks_skipped == int((ref == 0).sum()) * (ntiles // ref.shape[1])
    g2 = gpu_backward(spec, t, flags=cb.CBW_FLAG_NO_SKIP)
    check_dw_regrouped(gpu["dw"], g2["dw"], st.blocks_skipped, "balanced dW against no skipping")
    # sampled entries against the oracle over the live images only (dead
    # images contribute exact zeros)
    sub = {k: t[k][keep] if k != "w" else t[k] for k in ("x", "w", "dy")}
    x64, _, dy64 = oracle_inputs(sub)
    rng = np.random.default_rng(5)
    m = 1500
    co = np.stack([rng.integers(0, spec.K, m), rng.integers(0, spec.C, m), rng.integers(0, 3, m),
                   rng.integers(0, 3, m)], 1).astype(np.int32)
    o, a, nt = oracle.conv_bwd_weight_at(x64, dy64, (3, 3), co, (1, 1), (1, 1))
    g = gpu["dw"].cpu().numpy()[co[:, 0], co[:, 2], co[:, 3], co[:, 1]].astype(np.float64)
    check_values(g, o, a, nt, tol_for("bf16"), False, "balanced dW (sampled)")


@pytest.mark.parametrize("pattern", ["last_image_live", "odd_images_live"])
def test_balanced_split_past_staged_tile(pattern):
    """Configuration 2's layer at N = 336: 16464 chunks, more than a tile
    stages in LDS (16384), so the ranking reads its segments from global
    memory.  dY is zero over whole images; the occupancy, the per-tile work
    and dW (against the unskipped run) are checked as for the smaller
    batch.  A chunk is live exactly when it holds a pixel of a live image
    (a live image's 64 x 256 dY blocks are never all zero at density 0.4)."""
    spec = wl.config2(N=336)[0]
    _case("balanced split past the staged tile, " + pattern)
    d = wl.draw_on_device(spec)
    keep = [spec.N - 1] if pattern == "last_image_live" else list(range(1, spec.N, 2))
    dead = torch.ones(spec.N, dtype=torch.bool, device="cuda")
    dead[keep] = False
    d["dy"][dead] = 0
    desc = desc_of(spec)
    dym = torch.zeros(cb.cbw_dy_mask_words(desc), dtype=torch.int32, device="cuda")
    cb.cbw_nonzero_mask_pack(desc.dtype, d["dy"].numel(), d["dy"], dym)
    ws = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT)
    dw = torch.empty((spec.K, spec.R, spec.S, spec.C), dtype=torch.float32, device="cuda")
    cb.conv_bwd_weight_sparse(desc, d["x"], d["dy"], dym, dw, ws)
    occ, chunk, kw = cb.cbw_read_occupancy(desc, ws)
    work = cb.cbw_read_weight_work(desc, ws)
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, ws)
    dw_n = torch.empty_like(dw)
    cb.conv_bwd_weight_sparse(desc, d["x"], d["dy"], dym, dw_n, ws, cb.CBW_FLAG_NO_SKIP)
    torch.cuda.synchronize()
    nch = occ.shape[0]
    assert nch > 16384
    ppi = spec.P * spec.Q
    live_img = np.zeros(spec.N, bool)
    live_img[keep] = True
    first = np.arange(nch) * chunk // ppi
    last = np.minimum(np.arange(nch) * chunk + chunk, spec.N * ppi) - 1
    expect = np.array([live_img[a:b + 1].any() for a, b in zip(first, last // ppi)])
    assert np.array_equal(occ.astype(bool), np.repeat(expect[:, None], occ.shape[1], axis=1))
    nsplit, ntiles = work.shape
    live_t = np.full(ntiles, int(expect.sum()))
    assert np.array_equal(work.sum(axis=0), live_t)
    assert np.array_equal(work.max(axis=0), -(-live_t // nsplit))
    assert st.blocks_skipped == int((~expect).sum()) * ntiles
    check_dw_regrouped(dw, dw_n, st.blocks_skipped, "balanced dW past the staged tile against no skipping")


def _x_skip_case(N, C, H, W, K, R, S, stride, pad, dtype, seed):
    """Inputs with whole zero regions in both operands: X dead over a band of
    rows of every image and over the upper channel tile of a few pixels, dY
    dead over chunks and over one output-channel tile."""
    rng = np.random.default_rng(seed)
    spec = wl.LayerSpec("xskip", 0, 0, N=N, C=C, H=H, W=W, K=K, R=R, S=S, stride=stride, pad=pad, dtype=dtype)
    x = np.maximum(rng.standard_normal((N, H, W, C), dtype=np.float32) - 0.25, 0)
    x[:, 2:H // 2 + 3] = 0
    x[0, H - 2:, :, C // 2:] = 0
    dy = rng.standard_normal((N, spec.P, spec.Q, K), dtype=np.float32) * (rng.random((N, spec.P, spec.Q, K)) < 0.4)
    flat = dy.reshape(-1, K)
    flat[: flat.shape[0] // 3, : K // 2] = 0
    flat[-flat.shape[0] // 4:] = 0
    w = rng.standard_normal((K, R, S, C), dtype=np.float32) * 0.1
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    t = {"x": torch.from_numpy(x).to(tdt), "dy": torch.from_numpy(dy).to(tdt), "w": torch.from_numpy(w).to(tdt)}
    return spec, t


@pytest.mark.parametrize("case", [
    (2, 256, 16, 16, 256, 3, 3, 1, 1, "bf16"),     # one tap per tile
    (2, 64, 12, 14, 64, 3, 3, 1, 1, "bf16"),       # three taps packed per tile (3 + 3 + 3)
    (2, 48, 13, 11, 40, 3, 3, 2, 1, "bf16"),       # stride 2, five taps packed, ragged tiles
    (2, 320, 9, 9, 72, 1, 1, 1, 0, "bf16"),        # 1x1, two channel tiles
    (2, 32, 10, 10, 24, 3, 3, 1, 1, "f32"),        # float32 kernel
], ids=["c256", "c64_packed", "stride2", "c320_1x1", "f32"])
@pytest.mark.parametrize("use_bits", [True, False])
def test_x_block_skip(case, use_bits):
    """conv_bwd_weight_sparse_x: blocks whose dY or X operand is all zero are
    skipped; the number skipped equals the oracle's count of dead blocks
    (exact), dW matches the oracle and equals the non-skipping result."""
    N, C, H, W, K, R, S, st, pd, dt = case
    spec, t = _x_skip_case(N, C, H, W, K, R, S, st, pd, dt, seed=C + K)
    _case("x-skip %s bits=%s" % (case, use_bits))
    desc = desc_of(spec)
    d = to_dev(t, "cuda")
    xm = dym = None
    if use_bits:
        xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
        cb.cbw_nonzero_mask_pack(desc.dtype, d["x"].numel(), d["x"], xm)
        dym = torch.zeros(max(cb.cbw_dy_mask_words(desc), 1), dtype=torch.int32, device="cuda")
        cb.cbw_nonzero_mask_pack(desc.dtype, d["dy"].numel(), d["dy"], dym)
    ws = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT, "cuda")
    dw = torch.empty((K, R, S, C), dtype=torch.float32, device="cuda")
    cb.conv_bwd_weight_sparse_x(desc, d["x"], d["dy"], xm, dym, dw, ws)
    st_x = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, ws)
    work_x = cb.cbw_read_weight_work(desc, ws)
    occ, chunk, kw = cb.cbw_read_occupancy(desc, ws)
    dw_y = torch.empty_like(dw)
    cb.conv_bwd_weight_sparse(desc, d["x"], d["dy"], dym, dw_y, ws)
    st_y = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, ws)
    # the dY-only call may run the row-window kernel (narrow stride-1 layers),
    # whose skip chunks are whole output rows: its own occupancy and tiling
    occ_y, chunk_y, kw_y = cb.cbw_read_occupancy(desc, ws)
    ntiles_y = cb.cbw_read_weight_work(desc, ws).shape[1]
    dw_n = torch.empty_like(dw)
    cb.conv_bwd_weight_sparse_x(desc, d["x"], d["dy"], xm, dym, dw_n, ws, cb.CBW_FLAG_NO_SKIP)
    torch.cuda.synchronize()
    # the tiling: filter taps packed side by side for bf16 when two or more
    # channel tiles fit in 256 columns (as few groups as fit, the taps spread
    # evenly over them), else one tap per 256-channel tile
    packed = dt == "bf16" and R * S > 1 and 2 * C <= 256
    groups = -(-(R * S) // (256 // C)) if packed else R * S
    tpg = -(-(R * S) // groups) if packed else 1
    ctile = C if packed else 256
    x64, _, dy64 = oracle_inputs(t)
    live = oracle.weight_block_liveness(x64 != 0, dy64 != 0, (R, S), (st, st), (pd, pd), chunk, kw, ctile, tpg)
    ref_y = oracle.block_occupancy(t["dy"].float().numpy().reshape(-1, K), chunk_y, kw_y)
    assert np.array_equal(occ_y, ref_y)
    per_block_y = ntiles_y // ref_y.shape[1]      # tiles sharing one (chunk, k tile) block of dY
    assert st_x.blocks_total == live.size
    assert st_y.blocks_total == ref_y.size * per_block_y
    # work redistribution: every tile's live blocks are executed exactly once,
    # shared so that no split runs more than ceil(live / nsplit) of them
    nsplit, ntiles = work_x.shape
    per_tile = live.reshape(ntiles, -1).sum(axis=1)          # tiles in (group, channel tile, k tile) order
    assert np.array_equal(work_x.sum(axis=0), per_tile)
    assert np.array_equal(work_x.max(axis=0), -(-per_tile // nsplit))
    assert st_x.blocks_skipped == int((~live).sum())
    assert st_y.blocks_skipped == int((ref_y == 0).sum()) * per_block_y > 0
    if (C, st) in ((256, 1), (64, 1), (32, 1)) and chunk_y == chunk:
        # cases where the zero band empties whole X windows (same chunking)
        assert st_x.blocks_skipped > st_y.blocks_skipped
    ref_dw, ref_abs, ref_n = oracle.conv_bwd_weight(x64, dy64, (R, S), (st, st), (pd, pd), with_bound=True)
    check_values(dw_as_kcrs(dw), ref_dw, ref_abs, ref_n, tol_for(dt), False, "dW with X-block skipping")
    check_dw_regrouped(dw, dw_n, st_x.blocks_skipped, "X-skipping dW against no skipping")
    check_dw_regrouped(dw_y, dw_n, st_y.blocks_skipped, "dY-skipping dW against no skipping")


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
