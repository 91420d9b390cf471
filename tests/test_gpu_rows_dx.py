"""GPU parity of the row-window data gradient (3 x 3, stride-1 layers with 64
input and 64 output channels, bf16), which the data-gradient entry points
choose for those layers: dense and masked dX against the fp64 oracle on
shapes with ragged and multiple column segments, strips that cross image
boundaries, pads 0 to 2 and NCHW/KCRS boundaries; the row skip (output rows
whose footprint is empty cost no matrix work and come back as +0.0, counted
in the statistics); masked = dense x mask bitwise; run-twice determinism and
the combined call.  Every test prints its case before the first GPU call."""
import numpy as np
import pytest
import torch

import oracle
import paper_2109_07710_amd as cb
from parity import check_values, check_zero_pattern, dx_bits_nchw, tol_for

pytestmark = pytest.mark.gpu


def _case(msg):
    print("\n[case] " + msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


def _layer(N, H, W, pad, seed, dead_rows=None):
    rng = np.random.default_rng(seed)
    desc = cb.ConvDesc.make(N, 64, H, W, 64, 3, 3, (1, 1), pad)
    x = (rng.standard_normal((N, H, W, 64), dtype=np.float32) - 0.25)
    if dead_rows is not None:
        dead_rows(x)
    dy = rng.standard_normal((N, desc.P, desc.Q, 64), dtype=np.float32) * (rng.random((N, desc.P, desc.Q, 64)) < 0.5)
    w = rng.standard_normal((64, 3, 3, 64), dtype=np.float32) * 0.1
    t = {"x": torch.from_numpy(x).to(torch.bfloat16), "dy": torch.from_numpy(dy).to(torch.bfloat16),
         "w": torch.from_numpy(w).to(torch.bfloat16)}
    return desc, t


def _oracle(desc, t, masked):
    x64 = oracle.nhwc_to_nchw(t["x"].double().numpy())
    dy64 = oracle.nhwc_to_nchw(t["dy"].double().numpy())
    w64 = oracle.krsc_to_kcrs(t["w"].double().numpy())
    mask = oracle.relu_mask(x64)
    dx, absb, n = oracle.conv_bwd_data(dy64, w64, (desc.H, desc.W), (1, 1), (desc.pad_h, desc.pad_w),
                                       mask=mask if masked else None, with_bound=True)
    return dx, absb, n, mask


def _run(desc, t, masked, flags=0):
    d = {k: v.cuda() for k, v in t.items()}
    dx = torch.full_like(d["x"], float("nan"))
    if masked:
        xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
        cb.cbw_relu_mask_pack(desc, d["x"], xm)
        ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED)
        cb.conv_bwd_data_masked(desc, d["dy"], d["w"], xm, dx, ws, flags)
        st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_DATA_MASKED, ws)
    else:
        ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA)
        cb.conv_bwd_data(desc, d["dy"], d["w"], dx, ws)
        st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_DATA, ws)
    torch.cuda.synchronize()
    return dx, st


def _check(desc, t, dx, masked):
    o, absb, n, mask = _oracle(desc, t, masked)
    g = oracle.nhwc_to_nchw(dx.float().cpu().numpy())
    if masked:
        check_zero_pattern(dx_bits_nchw(dx), mask, "row-window dX")
    check_values(g, o, absb, n, tol_for("bf16"), True, "row-window dX")
    return mask


SHAPES = [
    # N, H, W, pad
    (2, 9, 14, (1, 1)),      # one segment of one 16-column block
    (3, 7, 56, (1, 1)),      # strips of one row: 21 rows over 21 workgroups
    (2, 13, 230, (1, 1)),    # two segments, the second 6 columns
    (1, 6, 449, (1, 1)),     # three segments, the last one column
    (2, 11, 37, (0, 0)),     # no padding: P = H - 2, Q = W - 2
    (2, 8, 40, (2, 2)),      # pad 2: P = H + 2
    (1, 10, 24, (2, 0)),     # unequal pads
    (100, 13, 12, (1, 1)),   # strips of 6 rows across 13-row images, prefetch 8 rows deep
    (6, 90, 150, (1, 1)),    # strips of 3 rows, prefetch 4 rows deep (150-column rings)
]


@pytest.mark.parametrize("masked", [False, True])
@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_rows_dx_against_oracle(shape, masked):
    N, H, W, pad = shape
    desc, t = _layer(N, H, W, pad, seed=N * 1000 + H * 10 + W)
    _case("row-window dX %s masked=%s P=%d Q=%d" % (shape, masked, desc.P, desc.Q))
    dx, st = _run(desc, t, masked)
    _check(desc, t, dx, masked)
    assert st.rows_total == N * H * W
    assert st.rows_live == st.rows_total   # random footprints: no row is dead


def test_rows_dx_strips_cross_images():
    """rows_per_strip does not divide H: a workgroup's strip runs into the
    next image and reloads its three dY rows there."""
    desc, t = _layer(60, 7, 20, (1, 1), seed=5)
    _case("row-window dX strips across images N=60 H=7 (420 rows: strips of 2; "
          "and N=300 H=3 -> strips of 4)")
    dx, _ = _run(desc, t, True)
    _check(desc, t, dx, True)
    desc, t = _layer(300, 3, 8, (1, 1), seed=6)
    dx, _ = _run(desc, t, True)
    _check(desc, t, dx, True)


def _computed_pixels(live, W):
    """Pixels the row-window kernel computes: per output row, each of its 8
    waves (2 channel halves x 4 column groups of 16-column blocks) runs its
    matrix work unless all its outputs are dead; a pixel counts once per
    channel half, the total is halved.  live: bool [rows, W, 64]."""
    nwb = (W + 15) // 16
    base, rem = divmod(nwb, 4)
    total = 0
    for wg in range(4):
        cnt = base + (1 if wg < rem else 0)
        b0 = wg * base + min(wg, rem)
        c0, c1 = 16 * b0, min(16 * (b0 + cnt), W)
        if c1 <= c0:
            continue
        for half in range(2):
            any_live = live[:, c0:c1, 32 * half:32 * half + 32].any(axis=(1, 2))
            total += int(any_live.sum()) * (c1 - c0)
    return total // 2


def test_rows_dx_dead_rows_skipped():
    """A wave whose outputs in a row are all dead skips that row's matrix
    work (those outputs are +0.0); the statistics count only the computed
    pixels; NO_SKIP computes everything (same values)."""
    def kill(x):
        x[0, 2:5] = -1.0     # three dead rows of image 0
        x[1, :, :] = -1.0    # image 1 entirely dead
        x[2, 7, :100] = -1.0 # a row with a live tail: only the waves over columns 80.. compute
        x[2, 3, :, :32] = -1.0   # one channel half dead along a row

    desc, t = _layer(3, 9, 130, (1, 1), seed=11, dead_rows=kill)
    _case("row-window dX dead rows N=3 H=9 W=130")
    dx, st = _run(desc, t, True)
    _check(desc, t, dx, True)
    live = (t["x"].float().numpy() > 0).reshape(3 * 9, 130, 64)
    expect = _computed_pixels(live, 130)
    assert expect < (3 * 9 - 3 - 9) * 130
    assert st.rows_live == expect
    dx2, st2 = _run(desc, t, True, cb.CBW_FLAG_NO_SKIP)
    assert torch.equal(dx.view(torch.int16), dx2.view(torch.int16))
    assert st2.rows_live == st2.rows_total
    # everything dead: no matrix work at all, every output +0.0
    t0 = dict(t)
    t0["x"] = -t["x"].abs() - 1
    dx0, st0 = _run(desc, t0, True)
    assert st0.rows_live == 0
    assert int(dx0.view(torch.int16).abs().sum()) == 0


def test_rows_dx_masked_equals_dense_times_mask():
    desc, t = _layer(2, 12, 100, (1, 1), seed=3)
    _case("row-window dX masked vs dense bitwise")
    dm, _ = _run(desc, t, True)
    dd, _ = _run(desc, t, False)
    mask = oracle.relu_mask(oracle.nhwc_to_nchw(t["x"].float().numpy()))
    bm, bd = dx_bits_nchw(dm), dx_bits_nchw(dd)
    assert np.array_equal(bm[mask], bd[mask])
    assert np.all(bm[~mask] == 0)
    dm2, _ = _run(desc, t, True)
    assert torch.equal(dm.view(torch.int16), dm2.view(torch.int16))


def test_rows_dx_lists_not_available():
    desc, t = _layer(1, 4, 16, (1, 1), seed=1)
    _case("row-window dX: the live-list reader reports unsupported")
    d = {k: v.cuda() for k, v in t.items()}
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, d["x"], xm)
    ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED)
    cb.conv_bwd_data_masked(desc, d["dy"], d["w"], xm, torch.empty_like(d["x"]), ws, 0)
    with pytest.raises(RuntimeError):
        cb.cbw_read_live_lists(desc, ws, 0)


@pytest.mark.parametrize("layout", ["nchw", "kcrs"])
def test_rows_dx_layouts(layout):
    desc, t = _layer(2, 10, 30, (1, 1), seed=21)
    _case("row-window dX boundary layout %s" % layout)
    d = {k: v.cuda() for k, v in t.items()}
    if layout == "kcrs":
        desc = cb.ConvDesc.make(2, 64, 10, 30, 64, 3, 3, (1, 1), (1, 1), w_layout="kcrs")
        w = d["w"].permute(0, 3, 1, 2).contiguous()
        xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
        cb.cbw_relu_mask_pack(desc, d["x"], xm)
        dx = torch.empty_like(d["x"])
        cb.conv_bwd_data_masked(desc, d["dy"], w, xm, dx, cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED), 0)
        torch.cuda.synchronize()
        _check(desc, t, dx, True)
    else:
        desc = cb.ConvDesc.make(2, 64, 10, 30, 64, 3, 3, (1, 1), (1, 1), act_layout="nchw")
        x_nchw = d["x"].permute(0, 3, 1, 2).contiguous()
        dy_nchw = d["dy"].permute(0, 3, 1, 2).contiguous()
        xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
        cb.cbw_relu_mask_pack(desc, x_nchw, xm)
        dx = torch.empty_like(x_nchw)
        cb.conv_bwd_data_masked(desc, dy_nchw, d["w"], xm, dx, cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED), 0)
        torch.cuda.synchronize()
        _check(desc, t, dx.permute(0, 2, 3, 1).contiguous(), True)


def test_rows_dx_combined_call_matches():
    desc, t = _layer(2, 14, 60, (1, 1), seed=8)
    _case("row-window dX through conv_bwd_sparse")
    d = {k: v.cuda() for k, v in t.items()}
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, d["x"], xm)
    dx = torch.empty_like(d["x"])
    dw = torch.empty((64, 3, 3, 64), dtype=torch.float32, device="cuda")
    ws = cb.workspace(desc, cb.CBW_OP_BWD_BOTH)
    cb.conv_bwd_sparse(desc, d["x"], d["dy"], d["w"], xm, None, dx, dw, ws, 0)
    ref, _ = _run(desc, t, True)
    assert torch.equal(dx.view(torch.int16), ref.view(torch.int16))
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_BOTH, ws)
    assert st.rows_live == st.rows_total
