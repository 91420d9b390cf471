"""GPU parity of the row-window weight gradient (narrow stride-1 layers: 64
or 128 channels in and out, filters of at most 3 x 3), which the weight
gradient entry points choose for those layers: against the fp64 oracle on
shapes with ragged column segments, unequal pads, non-square and 1 x 1
filters; the row occupancy and the balanced row ranges when whole output
rows of dY are zero; run-twice determinism.  Every test prints its case
before the first GPU call."""
import numpy as np
import pytest
import torch

import oracle
import paper_2109_07710_amd as cb
from parity import check_dw_regrouped, check_values, dw_as_kcrs

pytestmark = pytest.mark.gpu


def _case(msg):
    print("\n[case] " + msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


def _layer(N, C, K, H, W, R, S, pad, seed, dead_rows=None):
    rng = np.random.default_rng(seed)
    desc = cb.ConvDesc.make(N, C, H, W, K, R, S, (1, 1), pad)
    P, Q = desc.P, desc.Q
    x = np.maximum(rng.standard_normal((N, H, W, C), dtype=np.float32) - 0.25, 0)
    dy = rng.standard_normal((N, P, Q, K), dtype=np.float32) * (rng.random((N, P, Q, K)) < 0.4)
    if dead_rows is not None:
        dead_rows(dy)
    t = {"x": torch.from_numpy(x).to(torch.bfloat16), "dy": torch.from_numpy(dy).to(torch.bfloat16)}
    return desc, t


def _run(desc, t, flags=0, dy_mask=True):
    d = {k: v.cuda() for k, v in t.items()}
    dym = None
    if dy_mask:
        dym = torch.zeros(max(cb.cbw_dy_mask_words(desc), 1), dtype=torch.int32, device="cuda")
        cb.cbw_nonzero_mask_pack(desc.dtype, d["dy"].numel(), d["dy"], dym)
    dw = torch.full((desc.K, desc.R, desc.S, desc.C), 7.0, dtype=torch.float32, device="cuda")
    ws = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT)
    cb.conv_bwd_weight_sparse(desc, d["x"], d["dy"], dym, dw, ws, flags)
    torch.cuda.synchronize()
    return dw, ws


def _oracle(desc, t):
    x64 = oracle.nhwc_to_nchw(t["x"].double().numpy())
    dy64 = oracle.nhwc_to_nchw(t["dy"].double().numpy())
    return oracle.conv_bwd_weight(x64, dy64, (desc.R, desc.S), (1, 1), (desc.pad_h, desc.pad_w), with_bound=True)


SHAPES = [
    # N, C, K, H, W, R, S, pad
    (2, 64, 64, 20, 150, 3, 3, (1, 1)),     # two column segments, the second ragged (22 columns)
    (1, 64, 128, 17, 40, 3, 3, (1, 1)),     # two k tiles
    (2, 128, 128, 9, 30, 3, 3, (1, 1)),     # two channel and two k tiles
    (2, 128, 64, 8, 33, 3, 3, (0, 0)),      # no padding: P = H - 2
    (1, 64, 64, 12, 20, 2, 3, (0, 1)),      # 2 x 3 filter, unequal pads
    (1, 64, 64, 11, 26, 3, 1, (1, 0)),      # 3 x 1 filter
    (2, 64, 64, 10, 12, 1, 1, (0, 0)),      # 1 x 1
    (1, 64, 64, 5, 260, 3, 3, (2, 1)),      # three segments, pad 2 rows (P = H + 2)
]


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_rows_kernel_against_oracle(shape):
    N, C, K, H, W, R, S, pad = shape
    desc, t = _layer(N, C, K, H, W, R, S, pad, seed=C + K + H + W)
    _case("row-window dW %s P=%d Q=%d" % (shape, desc.P, desc.Q))
    dw, ws = _run(desc, t)
    occ, chunk, kw = cb.cbw_read_occupancy(desc, ws)
    assert chunk == desc.Q and kw == 64, "the row-window kernel runs for this layer"
    ref, absb, nterms = _oracle(desc, t)
    err = check_values(dw_as_kcrs(dw), ref, absb, nterms, 2e-2, False, "row-window dW")
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, ws)
    segments = -(-desc.Q // 128)
    assert st.blocks_total == N * desc.P * (K // 64) * segments * (C // 64)
    dw_n, _ = _run(desc, t, flags=cb.CBW_FLAG_NO_SKIP, dy_mask=False)
    check_dw_regrouped(dw, dw_n, st.blocks_skipped, "row-window dW against no skipping")
    print(err, st.blocks_skipped, st.blocks_total)


def _kill_rows(dy):
    # whole output rows zero: the first image's first half, and every third row of the second image
    N, P = dy.shape[0], dy.shape[1]
    dy[0, : P // 2] = 0
    if N > 1:
        dy[1, ::3] = 0


@pytest.mark.parametrize("use_bits", [True, False])
def test_rows_kernel_skips_dead_rows(use_bits):
    """Output rows whose dY is zero are skipped exactly (the oracle's row
    occupancy), the live rows are shared out in balanced ranges, and dW
    matches the oracle and the non-skipping run."""
    desc, t = _layer(2, 64, 64, 24, 56, 3, 3, (1, 1), seed=5, dead_rows=_kill_rows)
    _case("row-window dW, dead rows, bits=%s" % use_bits)
    dw, ws = _run(desc, t, dy_mask=use_bits)
    occ, chunk, kw = cb.cbw_read_occupancy(desc, ws)
    ref_occ = oracle.block_occupancy(t["dy"].float().numpy().reshape(-1, desc.K), chunk, kw)
    assert np.array_equal(occ, ref_occ) and (ref_occ == 0).any()
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, ws)
    work = cb.cbw_read_weight_work(desc, ws)
    nsplit, ntiles = work.shape
    live = int(ref_occ.sum())
    assert st.blocks_skipped == (ref_occ.size - live) * ntiles
    assert np.array_equal(work.sum(axis=0), np.full(ntiles, live))
    assert work.max() == -(-live // nsplit)
    ref, absb, nterms = _oracle(desc, t)
    check_values(dw_as_kcrs(dw), ref, absb, nterms, 2e-2, False, "row-window dW with dead rows")
    dw_n, _ = _run(desc, t, flags=cb.CBW_FLAG_NO_SKIP, dy_mask=False)
    check_dw_regrouped(dw, dw_n, st.blocks_skipped, "row-window dW with dead rows against no skipping")


def test_rows_kernel_run_twice_bitwise():
    desc, t = _layer(2, 64, 128, 14, 70, 3, 3, (1, 1), seed=9)
    _case("row-window dW run twice")
    a, _ = _run(desc, t)
    b, _ = _run(desc, t)
    assert torch.equal(a, b)
