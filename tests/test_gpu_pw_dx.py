"""GPU parity of the pointwise data gradient (1 x 1, stride-1, unpadded
layers with C and K in {64, 128, 256}, C * K <= 16384, bf16), which the
data-gradient entry points choose for those layers: dense and masked dX
against the fp64 oracle for every channel pair, pixel counts that leave a
ragged last block, several blocks per wave with an odd count and a short
last wave; the block skip (16-pixel blocks whose footprint is empty cost no
matrix work, come back as +0.0 and are left out of the statistics); masked =
dense x mask bitwise; run-twice determinism; NCHW/KCRS boundaries and the
combined call.  Every test prints its case before the first GPU call."""
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


def _layer(N, H, W, C, K, seed, dead=None):
    rng = np.random.default_rng(seed)
    desc = cb.ConvDesc.make(N, C, H, W, K, 1, 1, (1, 1), (0, 0))
    x = rng.standard_normal((N, H, W, C), dtype=np.float32) - 0.25
    if dead is not None:
        dead(x)
    dy = rng.standard_normal((N, H, W, K), dtype=np.float32) * (rng.random((N, H, W, K)) < 0.5)
    w = rng.standard_normal((K, 1, 1, C), dtype=np.float32) * 0.1
    t = {"x": torch.from_numpy(x).to(torch.bfloat16), "dy": torch.from_numpy(dy).to(torch.bfloat16),
         "w": torch.from_numpy(w).to(torch.bfloat16)}
    return desc, t


def _oracle(desc, t, masked):
    x64 = oracle.nhwc_to_nchw(t["x"].double().numpy())
    dy64 = oracle.nhwc_to_nchw(t["dy"].double().numpy())
    w64 = oracle.krsc_to_kcrs(t["w"].double().numpy())
    mask = oracle.relu_mask(x64)
    dx, absb, n = oracle.conv_bwd_data(dy64, w64, (desc.H, desc.W), (1, 1), (0, 0),
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
        check_zero_pattern(dx_bits_nchw(dx), mask, "pointwise dX")
    check_values(g, o, absb, n, tol_for("bf16"), True, "pointwise dX")
    return mask


SHAPES = [
    # N, H, W, C, K
    (3, 7, 9, 64, 64),        # 189 pixels: 11 blocks and a 13-pixel tail
    (2, 5, 21, 64, 128),
    (2, 17, 13, 64, 256),     # the bottleneck expansion's pair
    (1, 31, 7, 128, 64),
    (4, 6, 6, 128, 128),      # 144 pixels: whole blocks only
    (2, 11, 11, 256, 64),     # the bottleneck reduction's pair
    (2, 128, 130, 256, 64),   # 2080 blocks: two per wave
    (4, 128, 130, 64, 256),   # 4160 blocks: three per wave, the last wave two
]


@pytest.mark.parametrize("masked", [False, True])
@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_pw_dx_against_oracle(shape, masked):
    N, H, W, C, K = shape
    desc, t = _layer(N, H, W, C, K, seed=N * 1000 + H * 10 + W + C + K)
    _case("pointwise dX %s masked=%s" % (shape, masked))
    dx, st = _run(desc, t, masked)
    _check(desc, t, dx, masked)
    assert st.rows_total == N * H * W
    assert st.rows_live == st.rows_total   # random footprints: no block is dead


def _computed_pixels(live, npix):
    """Pixels of the 16-pixel blocks with a live output.  live: bool [npix, C]."""
    total = 0
    for b0 in range(0, npix, 16):
        if live[b0:b0 + 16].any():
            total += min(16, npix - b0)
    return total


@pytest.mark.parametrize("ck", [(256, 64), (64, 256)])
def test_pw_dx_dead_blocks_skipped(ck):
    """A 16-pixel block whose footprint is empty skips its matrix work (its
    outputs are +0.0) and is left out of the statistics; NO_SKIP computes
    everything (same values)."""
    C, K = ck

    def kill(x):
        x[0, 0:3] = -1.0          # three dead rows of 20 pixels: blocks 0-2 dead, block 3 partly
        x[1] = -1.0               # image 1 entirely dead
        x[2, 5, 4:] = -1.0        # a row with a live head
        x[2, 9, :, : C // 2] = -1.0   # half the channels dead along a row

    desc, t = _layer(3, 12, 20, C, K, seed=11, dead=kill)
    _case("pointwise dX dead blocks N=3 H=12 W=20 C=%d K=%d" % (C, K))
    dx, st = _run(desc, t, True)
    _check(desc, t, dx, True)
    live = (t["x"].float().numpy() > 0).reshape(-1, C)
    expect = _computed_pixels(live, live.shape[0])
    assert expect < live.shape[0] - 12 * 20
    assert st.rows_live == expect
    dx2, st2 = _run(desc, t, True, cb.CBW_FLAG_NO_SKIP)
    assert torch.equal(dx.view(torch.int16), dx2.view(torch.int16))
    assert st2.rows_live == st2.rows_total
    t0 = dict(t)
    t0["x"] = -t["x"].abs() - 1
    dx0, st0 = _run(desc, t0, True)
    assert st0.rows_live == 0
    assert int(dx0.view(torch.int16).abs().sum()) == 0


def test_pw_dx_masked_equals_dense_times_mask():
    desc, t = _layer(2, 19, 23, 256, 64, seed=3)
    _case("pointwise dX masked vs dense bitwise")
    dm, _ = _run(desc, t, True)
    dd, _ = _run(desc, t, False)
    mask = oracle.relu_mask(oracle.nhwc_to_nchw(t["x"].float().numpy()))
    bm, bd = dx_bits_nchw(dm), dx_bits_nchw(dd)
    assert np.array_equal(bm[mask], bd[mask])
    assert np.all(bm[~mask] == 0)
    dm2, _ = _run(desc, t, True)
    assert torch.equal(dm.view(torch.int16), dm2.view(torch.int16))


def test_pw_dx_lists_not_available():
    desc, t = _layer(1, 4, 16, 64, 256, seed=1)
    _case("pointwise dX: the live-list reader reports unsupported")
    d = {k: v.cuda() for k, v in t.items()}
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, d["x"], xm)
    ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED)
    cb.conv_bwd_data_masked(desc, d["dy"], d["w"], xm, torch.empty_like(d["x"]), ws, 0)
    with pytest.raises(RuntimeError):
        cb.cbw_read_live_lists(desc, ws, 0)


@pytest.mark.parametrize("layout", ["nchw", "kcrs"])
def test_pw_dx_layouts(layout):
    N, H, W, C, K = 2, 10, 30, 64, 256
    desc, t = _layer(N, H, W, C, K, seed=21)
    _case("pointwise dX boundary layout %s" % layout)
    d = {k: v.cuda() for k, v in t.items()}
    if layout == "kcrs":
        desc = cb.ConvDesc.make(N, C, H, W, K, 1, 1, (1, 1), (0, 0), w_layout="kcrs")
        w = d["w"].permute(0, 3, 1, 2).contiguous()
        xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
        cb.cbw_relu_mask_pack(desc, d["x"], xm)
        dx = torch.empty_like(d["x"])
        cb.conv_bwd_data_masked(desc, d["dy"], w, xm, dx, cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED), 0)
        torch.cuda.synchronize()
        _check(desc, t, dx, True)
    else:
        desc = cb.ConvDesc.make(N, C, H, W, K, 1, 1, (1, 1), (0, 0), act_layout="nchw")
        x_nchw = d["x"].permute(0, 3, 1, 2).contiguous()
        dy_nchw = d["dy"].permute(0, 3, 1, 2).contiguous()
        xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
        cb.cbw_relu_mask_pack(desc, x_nchw, xm)
        dx = torch.empty_like(x_nchw)
        cb.conv_bwd_data_masked(desc, dy_nchw, d["w"], xm, dx, cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED), 0)
        torch.cuda.synchronize()
        _check(desc, t, dx.permute(0, 2, 3, 1).contiguous(), True)


@pytest.mark.parametrize("ck", [(256, 64), (64, 256)])
def test_pw_dx_combined_call_matches(ck):
    C, K = ck
    desc, t = _layer(2, 14, 60, C, K, seed=8)
    _case("pointwise dX through conv_bwd_sparse C=%d K=%d" % (C, K))
    d = {k: v.cuda() for k, v in t.items()}
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, d["x"], xm)
    dx = torch.empty_like(d["x"])
    dw = torch.empty((K, 1, 1, C), dtype=torch.float32, device="cuda")
    ws = cb.workspace(desc, cb.CBW_OP_BWD_BOTH)
    cb.conv_bwd_sparse(desc, d["x"], d["dy"], d["w"], xm, None, dx, dw, ws, 0)
    ref, _ = _run(desc, t, True)
    assert torch.equal(dx.view(torch.int16), ref.view(torch.int16))
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_BOTH, ws)
    assert st.rows_live == st.rows_total
