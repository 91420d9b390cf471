"""GPU parity of the per-element data gradient (conv_bwd_data_elementwise)
against the fp64 oracle.

Values are compared with the normwise and per-element bounds of the other
parity tests.  Exact checks: every killed output is +0.0, and the number of
(tap, k) products each pixel executed equals the oracle's input-and-output
sparsity count (Sec. II-A compute model, one product per in-range tap with a
non-zero dY) for any live output of that pixel, and 0 for a pixel with no
live output.  The result agrees with the matrix-core masked path within the
same bounds (the summation orders differ).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2109_07710_amd as cb
import workloads as wl
from parity import check_values, desc_of, gpu_backward, oracle_inputs, tol_for, dx_as_nchw

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


def _spec(N, C, H, W, K, R, S, st, pd, dx, ddy, kind="bernoulli"):
    if kind == "bernoulli":
        return wl.LayerSpec("ew", 0, 1, N=N, C=C, H=H, W=W, K=K, R=R, S=S, stride=st, pad=pd,
                            x_kind="shifted_gauss", x_param=wl.threshold_for_density(dx),
                            dy_kind="bernoulli", dy_param=ddy)
    return wl.LayerSpec("ew", 0, 2, N=N, C=C, H=H, W=W, K=K, R=R, S=S, stride=st, pad=pd,
                        x_kind=kind, x_param=dx, dy_kind=kind, dy_param=ddy)


def _run(spec, t):
    desc = desc_of(spec)
    d = {k: v.cuda() for k, v in t.items()}
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, d["x"], xm)
    dx = torch.full_like(d["x"], float("nan"))
    ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_ELEMENTWISE)
    cb.conv_bwd_data_elementwise(desc, d["dy"], d["w"], xm, dx, ws)
    counts, total = cb.cbw_read_pixel_counts(desc, ws)
    torch.cuda.synchronize()
    return dx, counts, total


CASES = [
    # N, C, H, W, K, R, S, stride, pad, mask density, dY density
    (2, 64, 9, 11, 40, 3, 3, 1, 1, 0.4, 0.4),
    (2, 128, 7, 6, 8, 3, 3, 1, 1, 0.5, 0.3),
    (1, 256, 8, 8, 264, 3, 3, 1, 1, 0.1, 0.1),
    (1, 512, 6, 5, 520, 3, 3, 1, 1, 0.05, 0.05),     # two 512-k passes
    (2, 64, 11, 9, 24, 5, 5, 2, 2, 0.6, 0.5),        # stride 2: taps off the stride grid
    (2, 128, 10, 10, 16, 1, 1, 1, 0, 0.3, 0.7),      # 1x1
    (2, 256, 7, 9, 48, 3, 1, 2, 0, 0.2, 0.9),        # 3x1, stride 2, no padding
    (3, 64, 5, 5, 8, 3, 3, 3, 2, 0.9, 0.02),         # stride 3, very sparse dY
]


@pytest.mark.parametrize("case", CASES, ids=["c64", "c128", "c256_k264", "c512_k520", "s2_5x5", "1x1", "3x1_s2",
                                             "s3"])
def test_elementwise_parity(case):
    N, C, H, W, K, R, S, st, pd, dx_d, dy_d = case
    spec = _spec(*case)
    print("\n[case] elementwise %s" % (case,), flush=True)
    t = wl.draw(spec)
    dx, counts, total = _run(spec, t)
    x64, w64, dy64 = oracle_inputs(t)
    mask = oracle.relu_mask(x64)
    ref, ab, nt = oracle.conv_bwd_data(dy64, w64, (H, W), (st, st), (pd, pd), mask=mask, with_bound=True)
    g = dx_as_nchw(dx)
    check_values(g, ref, ab, nt, tol_for("bf16"), True, "elementwise dX")
    # killed outputs are +0.0 (bit pattern), live outputs finite
    bits = dx.view(torch.int16).cpu().numpy()
    assert not (oracle.nchw_to_nhwc(~mask) & (bits != 0)).any()
    assert torch.isfinite(dx.float()).all()
    # executed products per pixel: the oracle's IN+OUT count at any live output of the pixel
    _, per = oracle.bwd_data_macs(dy64, (H, W), (R, S), C, (st, st), (pd, pd), per_output=True)
    live_px = mask.any(axis=1)                                 # [N, H, W]
    expect = np.where(live_px, per[:, 0], 0).reshape(-1)       # pixel order (n, h, w)
    assert np.array_equal(counts, expect)
    assert total == int(expect.sum())


@pytest.mark.parametrize("kind,d", [("channel_shared", 0.1), ("clustered", 0.2)])
def test_elementwise_structured_masks(kind, d):
    """Structured footprints (whole dead pixels are skipped) against the
    matrix-core masked path and the oracle."""
    spec = _spec(2, 256, 14, 14, 256, 3, 3, 1, 1, d, d, kind=kind)
    print("\n[case] elementwise structured %s %.2f" % (kind, d), flush=True)
    t = wl.draw(spec)
    dx, counts, _ = _run(spec, t)
    mfma = gpu_backward(spec, t, masked=True)
    x64, w64, dy64 = oracle_inputs(t)
    mask = oracle.relu_mask(x64)
    ref, ab, nt = oracle.conv_bwd_data(dy64, w64, (14, 14), (1, 1), (1, 1), mask=mask, with_bound=True)
    check_values(dx_as_nchw(dx), ref, ab, nt, tol_for("bf16"), True, "elementwise dX")
    check_values(dx_as_nchw(mfma["dx"]), ref, ab, nt, tol_for("bf16"), True, "matrix-core dX")
    dead_px = ~mask.any(axis=1).reshape(-1)
    assert np.all(counts[dead_px] == 0)
    if kind == "channel_shared":        # whole pixels die only when the footprint is shared over channels
        assert dead_px.sum() > 0


def test_elementwise_deterministic_and_full_size():
    """Configuration 2's layer in full: two runs give the same bits; the zero
    pattern matches the footprint; sampled outputs match the oracle."""
    spec = wl.config2()[0]
    print("\n[case] elementwise full size", flush=True)
    t = wl.draw(spec)
    a, ca, _ = _run(spec, t)
    b, cb_, _ = _run(spec, t)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16)) and np.array_equal(ca, cb_)
    dead = (t["x"] <= 0).cuda()
    assert not (a.view(torch.int16)[dead] != 0).any().item()
    rng = np.random.default_rng(11)
    m = 3000
    co = np.stack([rng.integers(0, spec.N, m), rng.integers(0, spec.C, m), rng.integers(0, spec.H, m),
                   rng.integers(0, spec.W, m)], 1).astype(np.int32)
    x64, w64, dy64 = oracle_inputs(t)
    o, ab, nt = oracle.conv_bwd_data_at(dy64, w64, (spec.H, spec.W), co, (1, 1), (1, 1))
    live = oracle.relu_mask(x64)[co[:, 0], co[:, 1], co[:, 2], co[:, 3]]
    o, ab, nt = np.where(live, o, 0.0), np.where(live, ab, 0.0), np.where(live, nt, 0)
    g = a.float().cpu().numpy()[co[:, 0], co[:, 2], co[:, 3], co[:, 1]].astype(np.float64)
    check_values(g, o, ab, nt, tol_for("bf16"), True, "elementwise full size (sampled)")
