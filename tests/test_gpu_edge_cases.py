"""GPU edge cases: degenerate footprints, degenerate spatial sizes and the
largest tensors a buffer descriptor can address.

Degenerate footprints have exact answers: an all-dead footprint gives a dX of
+0.0 bit patterns with no row computed; an all-live one reproduces the dense
kernel bit for bit; an all-zero dY gives exact zeros everywhere with every
weight-gradient block skipped.  The largest case (configuration 2's layer at
N = 1280, 2.06 GB per activation tensor, just under the 2^31-byte limit of a
buffer descriptor) is checked against the oracle at sampled outputs of three
images, and over the whole tensors by exact properties (the zero pattern of
dX, and dW as the sum of the weight gradients of four quarter batches).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2109_07710_amd as cb
import workloads as wl
from parity import (check_layer, check_values, desc_of, dx_bits_nchw, gpu_backward, oracle_backward, oracle_inputs,
                    tol_for)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


def _case(name):
    print("\n[case] " + name, flush=True)


def _layer(N=2, C=64, H=10, W=12, K=48, dtype="bf16"):
    return wl.LayerSpec("edge", 0, 0, N=N, C=C, H=H, W=W, K=K, R=3, S=3, dtype=dtype,
                        x_kind="shifted_gauss", x_param=0.25, dy_kind="bernoulli", dy_param=0.4)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_all_dead_footprint(dtype):
    """X = 0 everywhere (a ReLU output with no live unit): the masked dX is
    the +0.0 pattern with no row computed, dW is exactly zero, and the X-block
    skip removes every weight-gradient block."""
    spec = _layer(dtype=dtype)
    _case("all-dead footprint " + dtype)
    t = wl.draw(spec)
    t["x"] = torch.zeros_like(t["x"])
    gpu = gpu_backward(spec, t, dy_mask=True)
    assert not dx_bits_nchw(gpu["dx"]).any()
    st = cb.cbw_read_stats(gpu["desc"], cb.CBW_OP_BWD_DATA_MASKED, gpu["ws_dx"])
    assert st.rows_live == 0 and st.rows_total > 0
    assert not gpu["dw"].view(torch.int32).any(), "dW must be +0.0 everywhere"
    desc = gpu["desc"]
    d = {k: v.cuda() for k, v in t.items()}
    dw = torch.full_like(gpu["dw"], 7.0)
    ws = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT)
    cb.conv_bwd_weight_sparse_x(desc, d["x"], d["dy"], None, None, dw, ws)
    stw = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, ws)
    assert stw.blocks_skipped == stw.blocks_total > 0
    assert not dw.view(torch.int32).any()


def test_all_live_footprint_equals_dense():
    """X > 0 everywhere: every row is live and the masked kernel reproduces
    the dense kernel bit for bit."""
    spec = _layer()
    _case("all-live footprint")
    t = wl.draw(spec)
    t["x"] = t["x"].float().abs().add(0.5).to(torch.bfloat16)
    g_m = gpu_backward(spec, t, masked=True)
    g_d = gpu_backward(spec, t, masked=False)
    st = cb.cbw_read_stats(g_m["desc"], cb.CBW_OP_BWD_DATA_MASKED, g_m["ws_dx"])
    assert st.rows_live == st.rows_total
    assert torch.equal(g_m["dx"].view(torch.int16), g_d["dx"].view(torch.int16))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_zero_gradient(dtype):
    """dY = 0: dX (masked and dense) and dW are +0.0 everywhere, and every
    weight-gradient block is skipped."""
    spec = _layer(dtype=dtype)
    _case("zero dY " + dtype)
    t = wl.draw(spec)
    t["dy"] = torch.zeros_like(t["dy"])
    for masked in (True, False):
        gpu = gpu_backward(spec, t, masked=masked, dy_mask=True)
        assert not dx_bits_nchw(gpu["dx"]).any()
        assert not gpu["dw"].view(torch.int32).any()
    st = cb.cbw_read_stats(gpu["desc"], cb.CBW_OP_BWD_WEIGHT, gpu["ws_dw"])
    assert st.blocks_skipped == st.blocks_total > 0


@pytest.mark.parametrize("N,H,W,C,K", [(5, 1, 1, 16, 24), (3, 1, 7, 8, 8), (2, 2, 2, 8, 264), (1, 3, 1, 272, 8)])
def test_tiny_images_and_widths(N, H, W, C, K):
    """Images of one pixel or one row (only some taps inside), the minimum
    channel width (one 16-byte vector) and widths just past a tile."""
    spec = _layer(N=N, C=C, H=H, W=W, K=K)
    _case("tiny N=%d %dx%d C=%d K=%d" % (N, H, W, C, K))
    t = wl.draw(spec)
    gpu = gpu_backward(spec, t, dy_mask=True)
    check_layer(spec, t, gpu, oracle_backward(spec, t))


def test_largest_addressable_tensors():
    """Configuration 2's layer at N = 1280: X, dY and dX are 2.06 GB each, just
    under the 2^31-byte limit of one buffer descriptor, so every 32-bit
    offset in the kernels is exercised near its top."""
    spec = wl.config2(N=1280)[0]
    desc = desc_of(spec)
    nbytes = spec.N * spec.H * spec.W * spec.C * 2
    assert 2 ** 31 - nbytes < 100 * 2 ** 20 and nbytes < 2 ** 31
    _case("largest tensors N=%d (%.2f GB per activation)" % (spec.N, nbytes / 1e9))
    d = wl.draw_on_device(spec)
    xm = torch.zeros(cb.cbw_mask_words(desc), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, d["x"], xm)
    dym = torch.zeros(cb.cbw_dy_mask_words(desc), dtype=torch.int32, device="cuda")
    cb.cbw_nonzero_mask_pack(desc.dtype, d["dy"].numel(), d["dy"], dym)
    dx = torch.empty_like(d["x"])
    ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED)
    cb.conv_bwd_data_masked(desc, d["dy"], d["w"], xm, dx, ws)
    dw = torch.empty((spec.K, spec.R, spec.S, spec.C), dtype=torch.float32, device="cuda")
    wsw = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT)
    cb.conv_bwd_weight_sparse(desc, d["x"], d["dy"], dym, dw, wsw)
    torch.cuda.synchronize()
    del ws, wsw
    # the zero pattern over the whole tensor (exact): dead outputs are +0.0
    dead = d["x"] <= 0
    assert not (dx.view(torch.int16)[dead] != 0).any().item()
    print("  zero pattern ok", flush=True)
    # sampled dX of three images against the oracle (an image's dX depends on that image only)
    imgs = [0, 641, spec.N - 1]
    rng = np.random.default_rng(7)
    for n in imgs:
        t = {"x": d["x"][n:n + 1].cpu(), "w": d["w"].cpu(), "dy": d["dy"][n:n + 1].cpu()}
        x64, w64, dy64 = oracle_inputs(t)
        m = 1500
        co = np.stack([np.zeros(m, np.int64), rng.integers(0, spec.C, m), rng.integers(0, spec.H, m),
                       rng.integers(0, spec.W, m)], 1).astype(np.int32)
        o, a, nt = oracle.conv_bwd_data_at(dy64, w64, (spec.H, spec.W), co, (1, 1), (1, 1))
        live = oracle.relu_mask(x64)[co[:, 0], co[:, 1], co[:, 2], co[:, 3]]
        o, a, nt = np.where(live, o, 0.0), np.where(live, a, 0.0), np.where(live, nt, 0)
        g = dx[n].float().cpu().numpy()[co[:, 2], co[:, 3], co[:, 1]].astype(np.float64)
        check_values(g, o, a, nt, tol_for("bf16"), True, "largest dX image %d (sampled)" % n)
    print("  sampled dX ok", flush=True)
    # dW: the sum of the weight gradients of four quarter batches, each a
    # separate call on its own slice (linearity of dW in the batch)
    q = spec.N // 4
    qspec = wl.config2(N=q)[0]
    qdesc = desc_of(qspec)
    acc = torch.zeros((spec.K, spec.R, spec.S, spec.C), dtype=torch.float64, device="cuda")
    part = torch.empty_like(dw)
    wsq = cb.workspace(qdesc, cb.CBW_OP_BWD_WEIGHT)
    for i in range(4):
        xs, dys = d["x"][i * q:(i + 1) * q], d["dy"][i * q:(i + 1) * q]
        cb.conv_bwd_weight_sparse(qdesc, xs, dys, None, part, wsq)
        acc += part.double()
    torch.cuda.synchronize()
    err = (dw.double() - acc).abs().max().item() / acc.abs().max().item()
    print("  dW vs quarter batches: normwise %.2e" % err, flush=True)
    assert err < 1e-4
    # and the dW of the first 16 images at sampled entries against the oracle
    sub = 16
    t = {"x": d["x"][:sub].cpu(), "w": d["w"].cpu(), "dy": d["dy"][:sub].cpu()}
    sspec = wl.config2(N=sub)[0]
    sdesc = desc_of(sspec)
    wss = cb.workspace(sdesc, cb.CBW_OP_BWD_WEIGHT)
    cb.conv_bwd_weight_sparse(sdesc, d["x"][:sub], d["dy"][:sub], None, part, wss)
    torch.cuda.synchronize()
    x64, _, dy64 = oracle_inputs(t)
    m = 2000
    co = np.stack([rng.integers(0, spec.K, m), rng.integers(0, spec.C, m), rng.integers(0, 3, m),
                   rng.integers(0, 3, m)], 1).astype(np.int32)
    o, a, nt = oracle.conv_bwd_weight_at(x64, dy64, (3, 3), co, (1, 1), (1, 1))
    g = part.cpu().numpy()[co[:, 0], co[:, 2], co[:, 3], co[:, 1]].astype(np.float64)
    check_values(g, o, a, nt, tol_for("bf16"), False, "dW of 16 images (sampled)")


# Live-row counts that differ between channel groups, so the skipping call's
# tile order (round by round across groups) runs past the rounds every group
# fills: one group all live and one all dead; one group all live and one with
# a third of its pixels live; three groups with 100%, 60% and 5% of their
# pixels live.  With 8 images the few tiles split their reduction; with 32
# images (112 tiles per full group) the last two cases run unsplit.
UNEVEN = [("live_dead", 512, (1.0, 0.0)), ("live_third", 512, (1.0, 0.33)), ("three_groups", 768, (1.0, 0.6, 0.05))]


@pytest.mark.parametrize("N", [8, 32])
@pytest.mark.parametrize("name,C,fracs", UNEVEN, ids=[u[0] for u in UNEVEN])
def test_uneven_group_counts(name, C, fracs, N):
    _case("uneven group counts %s C=%d %s N=%d" % (name, C, fracs, N))
    H, W, K = 28, 28, 64
    rng = np.random.default_rng(41)
    desc = cb.ConvDesc.make(N, C, H, W, K, 3, 3, 1, 1)
    x = torch.from_numpy(np.abs(rng.standard_normal((N, H, W, C), dtype=np.float32))).to(torch.bfloat16)
    # per group, a pixel is either live on every channel of the group or dead
    # on all of them (each group is 256 channels wide)
    live_px = np.stack([rng.random((N, H, W)) < f for f in fracs], -1)
    keep = np.repeat(live_px, 256, axis=-1)
    x = x * torch.from_numpy(keep)
    w = torch.from_numpy(rng.standard_normal((K, 3, 3, C), dtype=np.float32) * 0.05).to(torch.bfloat16)
    dy = torch.from_numpy(rng.standard_normal((N, H, W, K), dtype=np.float32)).to(torch.bfloat16)
    xd, wd, dyd = x.cuda(), w.cuda(), dy.cuda()
    xm = torch.zeros(cb.cbw_mask_words(desc), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, xd, xm)
    dense, gat = torch.empty_like(xd), torch.full_like(xd, float("nan"))
    cb.conv_bwd_data(desc, dyd, wd, dense, cb.workspace(desc, cb.CBW_OP_BWD_DATA))
    ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED)
    cb.conv_bwd_data_masked(desc, dyd, wd, xm, gat, ws, 0)
    torch.cuda.synchronize()
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_DATA_MASKED, ws)
    assert st.rows_live == int(live_px.sum()), "live rows counted by the compaction"
    live = xd > 0
    gb, db = gat.view(torch.int16), dense.view(torch.int16)
    assert not (gb[~live] != 0).any(), "killed outputs must be +0.0"
    # values against the oracle at sampled live outputs (a split reduction sums
    # in another order than the dense call, so only tolerance applies there)
    lv = np.argwhere(live.cpu().numpy())
    pick = lv[rng.choice(len(lv), size=min(3000, len(lv)), replace=False)]
    coords = pick[:, [0, 3, 1, 2]].astype(np.int32)          # (n, c, h, w)
    dy64 = oracle.nhwc_to_nchw(dy.double().numpy())
    w64 = oracle.krsc_to_kcrs(w.double().numpy())
    o, absd, nt = oracle.conv_bwd_data_at(dy64, w64, (H, W), coords, (1, 1), (1, 1))
    g = gat.float().cpu().numpy()[pick[:, 0], pick[:, 1], pick[:, 2], pick[:, 3]].astype(np.float64)
    check_values(g, o, absd, nt, tol_for("bf16"), True, name + " skipping dX (sampled live outputs)")
    if N == 32 and name != "live_dead":
        # neither call splits its reduction here (more than 128 tiles each):
        # the same per-output summation order, so the same bits
        assert torch.equal(gb[live], db[live]), "skipping call differs from the dense call at live outputs"
