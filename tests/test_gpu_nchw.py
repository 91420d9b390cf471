"""GPU checks of the NCHW boundary: the three backward operations (and the
X-skipping weight gradient) called with NCHW activations and footprints in
NCHW element order.

The library serves NCHW by transposing into NHWC copies and running the NHWC
path, so its results must equal the NHWC call on the same data bit for bit
(dX after the transpose back, dW, the +0.0 pattern and the skip statistics).
One case per dtype is also compared with the fp64 oracle, whose native layout
is NCHW.  Cases cover channel counts that are and are not multiples of 32
(the two footprint reorder paths), pixel counts that are not multiples of the
16-byte vector (the element-wise transpose path), stride 2 and both filter
layouts.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2109_07710_amd as cb
import workloads as wl
from parity import check_values, oracle_inputs, tol_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


CASES = [
    # N, C, H, W, K, R, S, stride, pad, dtype, w_layout
    (2, 64, 10, 12, 96, 3, 3, 1, 1, "bf16", "krsc"),    # HW = 120: vector transposes
    (3, 40, 9, 9, 24, 3, 3, 1, 1, "bf16", "kcrs"),      # C % 32 != 0, HW = 81: element transposes
    (2, 256, 17, 17, 264, 3, 3, 2, 1, "bf16", "krsc"),  # stride 2 (9 x 9 outputs), K past a tile
    (2, 32, 8, 5, 20, 1, 1, 1, 0, "f32", "krsc"),       # fp32, 1x1
    (2, 12, 8, 8, 36, 3, 3, 1, 1, "f32", "kcrs"),       # fp32, C % 32 != 0
]
IDS = ["c64", "c40_hw81_kcrs", "c256_s2", "f32_1x1", "f32_c12_kcrs"]


def _draw(case):
    N, C, H, W, K, R, S, st, pd, dt, wl_ = case
    spec = wl.LayerSpec("nchw", 0, 3, N=N, C=C, H=H, W=W, K=K, R=R, S=S, stride=st, pad=pd, dtype=dt,
                        x_kind="shifted_gauss", x_param=0.25, dy_kind="bernoulli", dy_param=0.5)
    t = wl.draw(spec)
    # a zero dY image (each case's first image holds a whole weight-gradient
    # chunk of output pixels) and a zero X image, so that both skips act
    t["dy"][0] = 0
    t["x"][-1] = 0
    return spec, t


def _desc(spec, layout, w_layout):
    return cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad,
                            dtype=spec.dtype, w_layout=w_layout, act_layout=layout)


def _run_all(desc, x, w, dy):
    """Every backward call on one layout; footprints packed in that layout's order."""
    xm = torch.zeros(cb.cbw_mask_words(desc), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, x, xm)
    dym = torch.zeros(cb.cbw_dy_mask_words(desc), dtype=torch.int32, device="cuda")
    cb.cbw_nonzero_mask_pack(desc.dtype, dy.numel(), dy, dym)
    out = {}
    ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED)
    out["dx_masked"] = torch.full_like(x, float("nan"))
    cb.conv_bwd_data_masked(desc, dy, w, xm, out["dx_masked"], ws)
    out["rows"] = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_DATA_MASKED, ws).rows_live
    wsd = cb.workspace(desc, cb.CBW_OP_BWD_DATA)
    out["dx_dense"] = torch.full_like(x, float("nan"))
    cb.conv_bwd_data(desc, dy, w, out["dx_dense"], wsd)
    wsw = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT)
    kshape = (desc.K, desc.R, desc.S, desc.C) if desc.w_layout == cb.CBW_KRSC else (desc.K, desc.C, desc.R, desc.S)
    for name, call in (("dw_bits", lambda o: cb.conv_bwd_weight_sparse(desc, x, dy, dym, o, wsw)),
                       ("dw_nobits", lambda o: cb.conv_bwd_weight_sparse(desc, x, dy, None, o, wsw)),
                       ("dw_x_bits", lambda o: cb.conv_bwd_weight_sparse_x(desc, x, dy, xm, dym, o, wsw)),
                       ("dw_x_nobits", lambda o: cb.conv_bwd_weight_sparse_x(desc, x, dy, None, None, o, wsw))):
        o = torch.full(kshape, float("nan"), dtype=torch.float32, device="cuda")
        call(o)
        out[name] = o
        out[name + "_skipped"] = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, wsw).blocks_skipped
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_nchw_equals_nhwc_bitwise(case):
    spec, t = _draw(case)
    w_layout = case[-1]
    print("\n[case] nchw %s" % (case,), flush=True)
    x, w, dy = (t[k].cuda() for k in ("x", "w", "dy"))       # NHWC, KRSC
    if w_layout == "kcrs":
        w = w.permute(0, 3, 1, 2).contiguous()
    ref = _run_all(_desc(spec, "nhwc", w_layout), x, w, dy)
    got = _run_all(_desc(spec, "nchw", w_layout), x.permute(0, 3, 1, 2).contiguous(), w,
                   dy.permute(0, 3, 1, 2).contiguous())
    bits = torch.int16 if spec.dtype == "bf16" else torch.int32
    for k in ("dx_masked", "dx_dense"):
        back = got[k].permute(0, 2, 3, 1)
        assert torch.equal(back.contiguous().view(bits), ref[k].view(bits)), k
    assert got["rows"] == ref["rows"]
    for k in ("dw_bits", "dw_nobits", "dw_x_bits", "dw_x_nobits"):
        assert torch.equal(got[k].view(torch.int32), ref[k].view(torch.int32)), k
        assert got[k + "_skipped"] == ref[k + "_skipped"], k
    assert ref["dw_bits_skipped"] > 0 and ref["dw_x_bits_skipped"] >= ref["dw_bits_skipped"]


@pytest.mark.parametrize("case", [CASES[1], CASES[4]], ids=["bf16", "f32"])
def test_nchw_against_oracle(case):
    spec, t = _draw(case)
    print("\n[case] nchw oracle %s" % (case,), flush=True)
    desc = _desc(spec, "nchw", "kcrs")
    x = t["x"].permute(0, 3, 1, 2).contiguous().cuda()
    dy = t["dy"].permute(0, 3, 1, 2).contiguous().cuda()
    w = t["w"].permute(0, 3, 1, 2).contiguous().cuda()         # KCRS
    xm = torch.zeros(cb.cbw_mask_words(desc), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, x, xm)
    dx = torch.full_like(x, float("nan"))
    cb.conv_bwd_data_masked(desc, dy, w, xm, dx, cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED))
    dw = torch.empty((spec.K, spec.C, spec.R, spec.S), dtype=torch.float32, device="cuda")
    cb.conv_bwd_weight_sparse(desc, x, dy, None, dw, cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT))
    torch.cuda.synchronize()
    x64, w64, dy64 = oracle_inputs(t)
    mask = oracle.relu_mask(x64)
    st, pd = (spec.stride, spec.stride), (spec.pad, spec.pad)
    ref, ab, nt = oracle.conv_bwd_data(dy64, w64, (spec.H, spec.W), st, pd, mask=mask, with_bound=True)
    tol = tol_for(spec.dtype)
    check_values(dx.double().cpu().numpy(), ref, ab, nt, tol, spec.dtype == "bf16", "NCHW masked dX")
    bits = dx.view(torch.int16 if spec.dtype == "bf16" else torch.int32).cpu().numpy()
    assert not (~mask & (bits != 0)).any(), "dead outputs must be +0.0"
    rw, aw, nw = oracle.conv_bwd_weight(x64, dy64, (spec.R, spec.S), st, pd, with_bound=True)
    check_values(dw.double().cpu().numpy(), rw, aw, nw, tol, False, "NCHW dW")
