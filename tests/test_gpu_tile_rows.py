"""GPU parity of the data-gradient GEMM (dense, non-skipping masked, skipping
masked) and of the forward at every pixel-row choice of every tile shape.

A tile covers its full pixel-row capacity or 16 or 32 rows less, and its
pixel blocks are then shared unevenly among the waves' pixel columns (for
example 7 + 6 blocks of 16 pixels).  The shapes below make the planner pick
each choice (checked through cbw_data_tiling; the skipping call makes the same
pick on the device because every pixel is live at these densities).  Values
at sampled outputs (random ones plus image borders, tile-boundary rows
included through the random draw) are compared with the fp64 oracle with the
normwise and per-element bounds of the other parity tests; over the whole
tensor, killed outputs must be +0.0 and the masked calls must equal the dense
call bit for bit at live outputs.  (With C = K = 64 the data gradient runs
the row-window kernel instead of the GEMM; the forward of those cases still
runs the 64-channel tile at its row choices.)
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2109_07710_amd as cb
import workloads as wl
from parity import check_values, tol_for

pytestmark = pytest.mark.gpu

NSAMPLE = 4000

# name, N, C (= K), H, W, expected (channels, capacity, rows)
CASES = [
    ("c256_rows208", 32, 256, 56, 56, (256, 224, 208)),
    ("c256_rows192", 12, 256, 64, 64, (256, 224, 192)),
    ("c128_rows416", 32, 128, 56, 56, (128, 448, 416)),
    ("c128_rows432", 27, 128, 64, 64, (128, 448, 432)),
    ("c64_rows480", 2, 64, 224, 224, (64, 512, 480)),
    ("c64_rows496", 31, 64, 64, 64, (64, 512, 496)),
    ("c256_rows192_f32", 12, 256, 64, 64, (256, 224, 192)),
    ("c256_rows208_f32", 32, 256, 56, 56, (256, 224, 208)),
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


def _coords(N, C, H, W, rng):
    n = rng.integers(0, N, NSAMPLE)
    c = rng.integers(0, C, NSAMPLE)
    h = rng.integers(0, H, NSAMPLE)
    w = rng.integers(0, W, NSAMPLE)
    pts = [np.stack([n, c, h, w], 1)]
    for hh in range(H):
        pts.append(np.array([[N - 1, C - 1, hh, 0], [0, 0, hh, W - 1]]))
    return np.concatenate(pts).astype(np.int32)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_tile_rows_parity(case):
    name, N, C, H, W, expect = case
    dtype = "f32" if name.endswith("_f32") else "bf16"
    print("\n[case] tile rows %s N=%d C=K=%d %dx%d %s" % (name, N, C, H, W, dtype), flush=True)
    spec = wl.LayerSpec(name, 2, 200 + CASES.index(case), N=N, C=C, H=H, W=W, K=C, R=3, S=3, dtype=dtype,
                        x_kind="shifted_gauss", x_param=0.25, dy_kind="bernoulli", dy_param=0.4)
    desc = cb.ConvDesc.make(N, C, H, W, C, 3, 3, 1, 1, dtype=dtype)
    assert cb.cbw_data_tiling(desc) == expect
    t = wl.draw(spec)
    x, w, dy = (t[k].cuda() for k in ("x", "w", "dy"))
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, x, xm)
    dense, sel, gat = torch.empty_like(x), torch.empty_like(x), torch.empty_like(x)
    cb.conv_bwd_data(desc, dy, w, dense, cb.workspace(desc, cb.CBW_OP_BWD_DATA))
    ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED)
    cb.conv_bwd_data_masked(desc, dy, w, xm, sel, ws, cb.CBW_FLAG_NO_SKIP)
    cb.conv_bwd_data_masked(desc, dy, w, xm, gat, ws, 0)
    y = torch.empty_like(x)
    ym = torch.zeros(max(cb.cbw_dy_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.conv_fwd_relu_mask(desc, x, w, y, ym, cb.workspace(desc, cb.CBW_OP_FWD))
    torch.cuda.synchronize()

    live = (x > 0)
    ity = torch.int16 if dtype == "bf16" else torch.int32
    db, sb, gb = (a.view(ity) for a in (dense, sel, gat))
    for what, m in (("non-skipping", sb), ("skipping", gb)):
        assert not (m[~live] != 0).any(), "%s masked call: killed outputs must be +0.0" % what
        assert torch.equal(m[live], db[live]), "%s masked call differs from the dense call at live outputs" % what

    rng = np.random.default_rng(77)
    cx = _coords(N, C, H, W, rng)
    x64 = oracle.nhwc_to_nchw(t["x"].double().numpy())
    w64 = oracle.krsc_to_kcrs(t["w"].double().numpy())
    dy64 = oracle.nhwc_to_nchw(t["dy"].double().numpy())
    tol = tol_for(dtype)
    o, absd, nt = oracle.conv_bwd_data_at(dy64, w64, (H, W), cx, (1, 1), (1, 1))
    g = dense.float().cpu().numpy()[cx[:, 0], cx[:, 2], cx[:, 3], cx[:, 1]].astype(np.float64)
    e1 = check_values(g, o, absd, nt, tol, dtype == "bf16", name + " dense dX (sampled)")
    z, a, n = oracle.conv_fwd_at(x64, w64, cx, (1, 1), (1, 1))
    gy = y.float().cpu().numpy()[cx[:, 0], cx[:, 2], cx[:, 3], cx[:, 1]].astype(np.float64)
    e2 = check_values(gy, np.maximum(z, 0.0), a, n, tol, dtype == "bf16", name + " forward (sampled)")
    print("  dX normwise %.3e, forward normwise %.3e" % (e1, e2), flush=True)
