"""GPU parity of conv_bwd_sparse, the call that computes both gradients of a
layer: against the separate calls it stands for (bitwise where their
reductions are grouped alike) and against the fp64 oracle, for skipping,
non-skipping and dense data gradients, layers whose data-gradient reduction
is split, X-block skipping, fp32, KCRS filters and NCHW tensors, and the
weight gradient's dead-block flag over a workspace shared by calls.  Every test
prints its case before the first GPU call."""
import numpy as np
import pytest
import torch

import paper_2109_07710_amd as cb
import workloads as wl
from parity import check_layer, desc_of, oracle_backward, to_dev

pytestmark = pytest.mark.gpu


def _case(msg):
    print("\n[case] " + msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


def _both(spec, d, desc, w, flags, masked, dy_mask, dev="cuda"):
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device=dev)
    cb.cbw_relu_mask_pack(desc, d["x"], xm)
    dym = None
    if dy_mask:
        dym = torch.zeros(max(cb.cbw_dy_mask_words(desc), 1), dtype=torch.int32, device=dev)
        cb.cbw_nonzero_mask_pack(desc.dtype, d["dy"].numel(), d["dy"], dym)
    dx = torch.full_like(d["x"], 7.0)          # every element must be overwritten
    shape = tuple(w.shape) if w.dtype == torch.float32 else tuple(w.shape)
    dw = torch.full(shape, 7.0, dtype=torch.float32, device=dev)
    ws = cb.workspace(desc, cb.CBW_OP_BWD_BOTH, dev)
    cb.conv_bwd_sparse(desc, d["x"], d["dy"], w, xm if masked else None, dym, dx, dw, ws, flags)
    torch.cuda.synchronize()
    return dx, dw, ws, xm, dym


def _separate(desc, d, w, xm, dym, flags, masked, x_skip, dw_shape, dev="cuda"):
    dx = torch.empty_like(d["x"])
    if masked:
        ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED, dev)
        cb.conv_bwd_data_masked(desc, d["dy"], w, xm, dx, ws, flags & cb.CBW_FLAG_NO_SKIP)
    else:
        ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA, dev)
        cb.conv_bwd_data(desc, d["dy"], w, dx, ws)
    dw = torch.empty(dw_shape, dtype=torch.float32, device=dev)
    ws2 = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT, dev)
    if x_skip:
        cb.conv_bwd_weight_sparse_x(desc, d["x"], d["dy"], xm, dym, dw, ws2, flags & cb.CBW_FLAG_NO_SKIP)
    else:
        cb.conv_bwd_weight_sparse(desc, d["x"], d["dy"], dym, dw, ws2, flags & cb.CBW_FLAG_NO_SKIP)
    torch.cuda.synchronize()
    return dx, dw


CASES = [
    # (name, spec factory, flags, masked, dy_mask, w_layout, act_layout)
    ("config1 fp32", lambda: wl.config1()[0], 0, True, True, "krsc", "nhwc"),
    ("config2 reduced, skipping", lambda: wl.config2(N=2, H=20)[0], 0, True, True, "krsc", "nhwc"),
    ("config2 reduced, no skip", lambda: wl.config2(N=2, H=20)[0], cb.CBW_FLAG_NO_SKIP, True, False, "krsc", "nhwc"),
    ("config2 reduced, dense dX", lambda: wl.config2(N=1, H=18)[0], cb.CBW_FLAG_NO_SKIP, False, False, "krsc", "nhwc"),
    ("config2 reduced, dY values for occupancy", lambda: wl.config2(N=2, H=16)[0], 0, True, False, "krsc", "nhwc"),
    ("config3 L1 1x1", lambda: wl.config3(N=2, H=20)[0], 0, True, True, "krsc", "nhwc"),
    ("config3 L2 3x3 64", lambda: wl.config3(N=2, H=20)[1], 0, True, True, "krsc", "nhwc"),
    ("config4 channel-shared d=0.1 (split data-gradient reduction)",
     lambda: wl.config4(0.1, "channel_shared", N=8)[0], 0, True, True, "krsc", "nhwc"),
    ("config4 clustered d=0.3", lambda: wl.config4(0.3, "clustered", N=4)[0], 0, True, True, "krsc", "nhwc"),
    ("config4 channel-shared d=0.2, X blocks skipped",
     lambda: wl.config4(0.2, "channel_shared", N=8)[0], cb.CBW_FLAG_SKIP_X_BLOCKS, True, True, "krsc", "nhwc"),
    ("config2 reduced, KCRS filters", lambda: wl.config2(N=1, H=20)[0], 0, True, True, "kcrs", "nhwc"),
    # the weight gradient's reduction in the data GEMM's tail workgroups with
    # 16 threads per output (row-window dW, 224 splits), and with a data
    # gradient whose dense tiling is split (its own reduction launch)
    ("VGG conv2_2 at 28x28, tail reduction", lambda: wl.config5(N=32, scale=4)[3], 0, True, True, "krsc", "nhwc"),
    ("VGG conv5_2, split data gradient", lambda: wl.config5(N=8)[11], 0, True, True, "krsc", "nhwc"),
    ("VGG conv5_2, split data gradient, no skip", lambda: wl.config5(N=8)[11], cb.CBW_FLAG_NO_SKIP, True, False,
     "kcrs", "nhwc"),
    ("config2 reduced, NCHW", lambda: wl.config2(N=1, H=20)[0], 0, True, True, "krsc", "nchw"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_both_gradients(case):
    name, make, flags, masked, dy_mask, w_layout, act_layout = case
    spec = make()
    _case("%s: %s N=%d C=%d K=%d %dx%d flags=%d masked=%s" % (name, spec.name, spec.N, spec.C, spec.K, spec.H,
                                                              spec.W, flags, masked, ))
    t = wl.draw(spec)
    d = to_dev(t)
    desc = desc_of(spec, w_layout)
    w = d["w"] if w_layout == "krsc" else d["w"].permute(0, 3, 1, 2).contiguous()
    dw_shape = (spec.K, spec.R, spec.S, spec.C) if w_layout == "krsc" else (spec.K, spec.C, spec.R, spec.S)
    if act_layout == "nchw":
        desc.act_layout = cb.CBW_NCHW
        d = {"x": d["x"].permute(0, 3, 1, 2).contiguous(), "dy": d["dy"].permute(0, 3, 1, 2).contiguous()}
    dx, dw, ws, xm, dym = _both(spec, d, desc, w, flags, masked, dy_mask)
    x_skip = bool(flags & cb.CBW_FLAG_SKIP_X_BLOCKS) and masked
    sdx, sdw = _separate(desc, d, w, xm, dym, flags, masked, x_skip, dw_shape)
    # the same kernels and splits as the separate calls: identical bits
    assert torch.equal(dx.view(torch.int16 if dx.dtype == torch.bfloat16 else torch.int32),
                       sdx.view(torch.int16 if sdx.dtype == torch.bfloat16 else torch.int32)), "dX differs"
    assert torch.equal(dw, sdw), "dW differs"
    # and the oracle
    if act_layout == "nchw":
        dx = dx.permute(0, 2, 3, 1).contiguous()
    gpu = {"dx": dx, "dw": dw}
    ref = oracle_backward(spec, t, masked=masked)
    errs = check_layer(spec, t, gpu, ref, masked=masked, w_layout=w_layout)
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_BOTH, ws)
    print(errs, st.rows_live, st.rows_total, st.blocks_skipped, st.blocks_total)
    if not masked or flags & cb.CBW_FLAG_NO_SKIP:
        assert st.rows_live == st.rows_total
    if flags & cb.CBW_FLAG_NO_SKIP:
        assert st.blocks_skipped == 0


def test_both_gradients_live_lists_and_occupancy():
    """The data-gradient part of the workspace holds the compaction lists the
    oracle defines (channel-shared footprint: whole rows dead), and the
    weight-gradient part the block occupancy of a dY with zero blocks."""
    import oracle
    spec = wl.config4(0.3, "channel_shared", N=4)[0]
    _case("lists and occupancy through conv_bwd_sparse: %s" % spec.name)
    t = wl.draw(spec)
    npq = spec.N * spec.P * spec.Q
    flat = t["dy"].view(npq, spec.K)
    flat[0:300, 0:256] = 0        # zero blocks in the first k tile
    flat[260:512, :] = 0          # and whole chunks
    d = to_dev(t)
    desc = desc_of(spec)
    dx, dw, ws, xm, dym = _both(spec, d, desc, d["w"], 0, True, True)
    npix = spec.N * spec.H * spec.W
    bits = xm.cpu().numpy().view(np.uint32)
    _, G = cb.cbw_read_live_lists(desc, ws, 0)
    ref = oracle.live_pixel_lists(bits, npix, spec.C, G)
    assert any(len(r) < npix for r in ref)
    for g in range(len(ref)):
        got, _ = cb.cbw_read_live_lists(desc, ws, g)
        assert np.array_equal(got, ref[g]), g
    off = cb.both_weight_offset(desc)
    occ, chunk, kw = cb.cbw_read_occupancy(desc, ws[off:])
    ref_occ = oracle.block_occupancy(flat.float().numpy(), chunk, kw)
    assert np.array_equal(occ, ref_occ) and (ref_occ == 0).any()
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_BOTH, ws)
    assert st.rows_live == sum(len(r) for r in ref)
    assert st.blocks_skipped > 0
    res = oracle_backward(spec, t)
    check_layer(spec, t, {"dx": dx, "dw": dw}, res)


def test_weight_gradient_alone():
    """dX = NULL: the weight gradient alone, equal to conv_bwd_weight_sparse."""
    spec = wl.config2(N=2, H=16)[0]
    _case("conv_bwd_sparse without dX: %s" % spec.name)
    t = wl.draw(spec)
    d = to_dev(t)
    desc = desc_of(spec)
    dym = torch.zeros(max(cb.cbw_dy_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.cbw_nonzero_mask_pack(desc.dtype, d["dy"].numel(), d["dy"], dym)
    dw = torch.full((spec.K, spec.R, spec.S, spec.C), 7.0, dtype=torch.float32, device="cuda")
    ws = cb.workspace(desc, cb.CBW_OP_BWD_BOTH)
    cb.conv_bwd_sparse(desc, d["x"], d["dy"], None, None, dym, None, dw, ws, 0)
    dw2 = torch.empty_like(dw)
    cb.conv_bwd_weight_sparse(desc, d["x"], d["dy"], dym, dw2, cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT), 0)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw2)


@pytest.mark.parametrize("layer", ["tiled", "rows"])
def test_weight_dead_block_flag_sequence_shared_workspace(layer):
    """One workspace over weight-gradient calls whose dY alternates between
    every block live and whole images of zeros, starting from a zeroed and
    from a 0xff-filled workspace, through conv_bwd_weight_sparse and
    conv_bwd_sparse: each call's dW and skip counts equal those of the same
    call on a fresh workspace, whatever dead-block flag the previous call
    (or the fill) left in the header.  The skipping GEMM takes the unskipped
    ranges unless the occupancy pass of the same call stored its number."""
    spec = wl.config2(N=3, H=14)[0] if layer == "tiled" else wl.config3(N=3, H=14)[1]
    _case("dW dead-block flag sequence %s %s N=%d C=%d K=%d %dx%d" % (layer, spec.name, spec.N, spec.C, spec.K,
                                                                   spec.H, spec.W))
    t = wl.draw(spec)
    d = to_dev(t)
    desc = desc_of(spec)
    dy_live = d["dy"].clone()
    dy_live[dy_live == 0] = 0.5          # every dY entry non-zero: no dead block
    dy_dead = d["dy"].clone()
    dy_dead[1] = 0                       # image 1 entirely zero: its blocks are dead
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, d["x"], xm)

    def dym_of(dy):
        m = torch.zeros(max(cb.cbw_dy_mask_words(desc), 1), dtype=torch.int32, device="cuda")
        cb.cbw_nonzero_mask_pack(desc.dtype, dy.numel(), dy, m)
        return m

    def run(dy, ws, both):
        dw = torch.full((spec.K, spec.R, spec.S, spec.C), 7.0, dtype=torch.float32, device="cuda")
        if both:
            dx = torch.empty_like(d["x"])
            cb.conv_bwd_sparse(desc, d["x"], dy, d["w"], xm, dym_of(dy), dx, dw, ws, 0)
            st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_BOTH, ws)
        else:
            cb.conv_bwd_weight_sparse(desc, d["x"], dy, dym_of(dy), dw, ws, 0)
            st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, ws)
        torch.cuda.synchronize()
        return dw, st.blocks_skipped, st.blocks_total

    for both in (False, True):
        op = cb.CBW_OP_BWD_BOTH if both else cb.CBW_OP_BWD_WEIGHT
        fresh = {}
        for name, dy in (("live", dy_live), ("dead", dy_dead)):
            fresh[name] = run(dy, cb.workspace(desc, op, "cuda").zero_(), both)
        assert fresh["live"][1] == 0
        assert fresh["dead"][1] > 0
        for fill in (0, 255):
            ws = cb.workspace(desc, op, "cuda")
            ws.fill_(fill)
            for i, name in enumerate(("live", "dead", "live", "dead", "dead", "live")):
                dw, skipped, total = run(dy_live if name == "live" else dy_dead, ws, both)
                ref, ref_skipped, ref_total = fresh[name]
                assert torch.equal(dw, ref), (both, fill, i, name)
                assert (skipped, total) == (ref_skipped, ref_total), (both, fill, i, name)
