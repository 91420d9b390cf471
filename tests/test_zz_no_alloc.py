"""The masked data gradient on the library's built-in scratch
(conv_bwd_data_masked_noalloc), through the C-ABI, against the workspace
entry point conv_bwd_data_masked and the oracle: two calls in a row, the
second with a smaller input, so the second call also runs on scratch that
still holds the first call's lists and filters."""
import numpy as np
import pytest
import torch

import paper_2109_07710_amd as cb
import workloads as wl
from parity import check_values, check_zero_pattern, dx_as_nchw, dx_bits_nchw, oracle_backward, tol_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


def _both(spec, t):
    dev = "cuda"
    desc = cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad,
                            dtype=spec.dtype)
    x, w, dy = (t[k].to(dev) for k in ("x", "w", "dy"))
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device=dev)
    cb.cbw_relu_mask_pack(desc, x, xm)
    dx_ws = torch.empty_like(x)
    ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED, dev)
    cb.conv_bwd_data_masked(desc, dy, w, xm, dx_ws, ws, 0)
    dx_na = torch.full_like(x, float("nan"))      # every output must be written
    cb.conv_bwd_data_masked_noalloc(desc, dy, w, xm, dx_na, 0)
    torch.cuda.synchronize()
    stats = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_DATA_MASKED, ws)
    return desc, dx_ws, dx_na, stats


def test_noalloc_two_calls_second_smaller():
    # 1: the benchmark layer at full size; its tiles are too many for the
    # workspace call to split the reduction, so both calls run the same
    # kernels in the same order: identical bits
    spec = wl.config2()[0]
    print("\n[case] noalloc call 1: %s N=%d %dx%d" % (spec.name, spec.N, spec.H, spec.W), flush=True)
    t = wl.draw(spec)
    _, dx_ws, dx_na, stats = _both(spec, t)
    assert stats.rows_live == stats.rows_total
    assert torch.equal(dx_ws.view(torch.int16), dx_na.view(torch.int16)), "noalloc differs from the workspace call"
    del dx_ws, dx_na, t
    # 2: a smaller layer right after (two images of 12 x 12): the workspace
    # call splits its few tiles' reductions, the scratch call does not, so
    # both are checked against the oracle and against each other
    spec = wl.config2(N=2, H=12)[0]
    print("[case] noalloc call 2: %s N=%d %dx%d" % (spec.name, spec.N, spec.H, spec.W), flush=True)
    t = wl.draw(spec)
    _, dx_ws, dx_na, _ = _both(spec, t)
    ref = oracle_backward(spec, t)
    tol = tol_for(spec.dtype)
    check_zero_pattern(dx_bits_nchw(dx_na), ref["mask"], "noalloc dX")
    check_values(dx_as_nchw(dx_na), ref["dx"], ref["dx_abs"], ref["dx_n"], tol, True, "noalloc dX")
    check_values(dx_as_nchw(dx_ws), ref["dx"], ref["dx_abs"], ref["dx_n"], tol, True, "workspace dX")
    a, b = dx_as_nchw(dx_na), dx_as_nchw(dx_ws)
    assert np.max(np.abs(a - b)) <= 2.0 ** -7 * max(np.max(np.abs(b)), 1e-30)


def test_noalloc_fp32_and_strided_small():
    """fp32 and a strided layer, each called twice with the second smaller."""
    for spec in (wl.config1()[0],
                 wl.LayerSpec("strided_3x3_c64", 9, 1, N=2, C=64, H=15, W=13, K=32, R=3, S=3, stride=2, pad=1,
                              x_kind="shifted_gauss", x_param=0.3, dy_kind="bernoulli", dy_param=0.5)):
        for n in (spec.N, 1):
            spec.N = n
            print("[case] noalloc %s N=%d" % (spec.name, n), flush=True)
            t = wl.draw(spec)
            _, _, dx_na, _ = _both(spec, t)
            ref = oracle_backward(spec, t)
            check_zero_pattern(dx_bits_nchw(dx_na), ref["mask"], "noalloc dX")
            check_values(dx_as_nchw(dx_na), ref["dx"], ref["dx_abs"], ref["dx_n"], tol_for(spec.dtype),
                         spec.dtype == "bf16", "noalloc dX")
