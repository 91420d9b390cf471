"""Seeded random layer shapes through every backward entry point, against the
fp64 oracle.

Each case draws its own batch, image size, channel counts (multiples of the
16-byte vector), filter size, stride and padding (each independently per
axis), element type, filter layout and activation layout, so combinations
the hand-picked tests do not name (unequal strides, R != S with unequal
pads, odd widths just past a tile, NCHW with KCRS) are exercised.  dY is
zero over the first image (its upper half for a batch of one) so that the
weight gradient skips blocks where a whole chunk of pixels falls inside.
Checks: masked and dense dX (values, and the +0.0 pattern of killed
outputs), dW with dY skipping, with X skipping and without skipping (values;
the skipping runs agree with the unskipped one to fp32 reassociation), and
that a second call of the masked dX and of both skipping dW calls gives the
same bits.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2109_07710_amd as cb
from parity import check_dw_regrouped, check_values, tol_for

pytestmark = pytest.mark.gpu

NCASES = 48


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cb.lib()


def _case(i):
    rng = np.random.default_rng([210907710, 77, i])
    dt = "bf16" if rng.random() < 0.7 else "f32"
    v = 8 if dt == "bf16" else 4
    while True:
        N = int(rng.integers(1, 4))
        H, W = (int(a) for a in rng.integers(1, 30, 2))
        R, S = (int(a) for a in rng.integers(1, 6, 2))
        sh, sw = (int(a) for a in rng.integers(1, 4, 2))
        ph, pw = int(rng.integers(0, R)), int(rng.integers(0, S))
        P, Q = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
        if P >= 1 and Q >= 1 and H + 2 * ph >= R and W + 2 * pw >= S:
            break
    C = v * int(rng.integers(1, 200 // v + 1))
    K = v * int(rng.integers(1, 200 // v + 1))
    return dict(N=N, C=C, H=H, W=W, K=K, R=R, S=S, stride=(sh, sw), pad=(ph, pw), P=P, Q=Q, dtype=dt,
                w_layout="kcrs" if rng.random() < 0.4 else "krsc", act="nchw" if rng.random() < 0.3 else "nhwc",
                seed=i)


CASES = [_case(i) for i in range(NCASES)]


def _ids(c):
    return "%s_%s_%s_N%dC%dK%d_%dx%d_f%dx%d_s%dx%d_p%dx%d" % (
        c["dtype"], c["act"], c["w_layout"], c["N"], c["C"], c["K"], c["H"], c["W"], c["R"], c["S"],
        c["stride"][0], c["stride"][1], c["pad"][0], c["pad"][1])


def _inputs(c):
    rng = np.random.default_rng([210907710, 78, c["seed"]])
    td = torch.bfloat16 if c["dtype"] == "bf16" else torch.float32
    x = np.maximum(rng.standard_normal((c["N"], c["H"], c["W"], c["C"]), dtype=np.float32) - 0.1, 0.0)
    w = rng.standard_normal((c["K"], c["R"], c["S"], c["C"]), dtype=np.float32) * np.sqrt(
        2.0 / (c["C"] * c["R"] * c["S"]))
    dy = rng.standard_normal((c["N"], c["P"], c["Q"], c["K"]), dtype=np.float32)
    dy *= rng.random(dy.shape) < 0.5
    if c["N"] > 1:
        dy[0] = 0.0
    else:
        dy[0, : max(1, c["P"] // 2)] = 0.0
    return {k: torch.from_numpy(np.ascontiguousarray(a)).to(td) for k, a in (("x", x), ("w", w), ("dy", dy))}


@pytest.mark.parametrize("c", CASES, ids=[_ids(c) for c in CASES])
def test_random_shape(c):
    print("\n[case] random shape %s" % _ids(c), flush=True)
    t = _inputs(c)
    nchw = c["act"] == "nchw"
    desc = cb.ConvDesc.make(c["N"], c["C"], c["H"], c["W"], c["K"], c["R"], c["S"], c["stride"], c["pad"],
                            dtype=c["dtype"], w_layout=c["w_layout"], act_layout=c["act"])
    assert cb.cbw_validate_desc(desc) == cb.CBW_OK
    act = (lambda a: a.permute(0, 3, 1, 2).contiguous()) if nchw else (lambda a: a)
    x, dy = act(t["x"]).cuda(), act(t["dy"]).cuda()
    w = t["w"].cuda() if c["w_layout"] == "krsc" else t["w"].permute(0, 3, 1, 2).contiguous().cuda()
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.cbw_relu_mask_pack(desc, x, xm)
    dym = torch.zeros(max(cb.cbw_dy_mask_words(desc), 1), dtype=torch.int32, device="cuda")
    cb.cbw_nonzero_mask_pack(desc.dtype, dy.numel(), dy, dym)
    dxm = torch.full_like(x, float("nan"))
    cb.conv_bwd_data_masked(desc, dy, w, xm, dxm, cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED))
    dxd = torch.full_like(x, float("nan"))
    cb.conv_bwd_data(desc, dy, w, dxd, cb.workspace(desc, cb.CBW_OP_BWD_DATA))
    wsw = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT)
    dws = {}
    for name, call in (("dy_skip", lambda o: cb.conv_bwd_weight_sparse(desc, x, dy, dym, o, wsw)),
                       ("x_skip", lambda o: cb.conv_bwd_weight_sparse_x(desc, x, dy, xm, dym, o, wsw)),
                       ("no_skip", lambda o: cb.conv_bwd_weight_sparse(desc, x, dy, None, o, wsw,
                                                                       cb.CBW_FLAG_NO_SKIP))):
        o = torch.full(w.shape, float("nan"), dtype=torch.float32, device="cuda")
        call(o)
        torch.cuda.synchronize()
        dws[name] = (o, cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, wsw).blocks_skipped)
    torch.cuda.synchronize()
    # a second run of every call gives the same bits (fixed reduction orders)
    again = torch.full_like(x, float("nan"))
    cb.conv_bwd_data_masked(desc, dy, w, xm, again, cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED))
    assert torch.equal(again.view(torch.int16 if c["dtype"] == "bf16" else torch.int32),
                       dxm.view(torch.int16 if c["dtype"] == "bf16" else torch.int32)), "masked dX not reproducible"
    for name, fn in (("dy_skip", lambda o: cb.conv_bwd_weight_sparse(desc, x, dy, dym, o, wsw)),
                     ("x_skip", lambda o: cb.conv_bwd_weight_sparse_x(desc, x, dy, xm, dym, o, wsw))):
        o = torch.full(w.shape, float("nan"), dtype=torch.float32, device="cuda")
        fn(o)
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int32), dws[name][0].view(torch.int32)), "dW %s not reproducible" % name

    x64 = oracle.nhwc_to_nchw(t["x"].double().numpy())
    w64 = oracle.krsc_to_kcrs(t["w"].double().numpy())
    dy64 = oracle.nhwc_to_nchw(t["dy"].double().numpy())
    mask = oracle.relu_mask(x64)
    st, pd, tol, bf = c["stride"], c["pad"], tol_for(c["dtype"]), c["dtype"] == "bf16"
    nchw_of = (lambda g: g.double().cpu().numpy()) if nchw else \
        (lambda g: oracle.nhwc_to_nchw(g.double().cpu().numpy()))
    ref, ab, nt = oracle.conv_bwd_data(dy64, w64, (c["H"], c["W"]), st, pd, mask=mask, with_bound=True)
    check_values(nchw_of(dxm), ref, ab, nt, tol, bf, "masked dX")
    bits = dxm.view(torch.int16 if bf else torch.int32).cpu().numpy()
    if not nchw:
        bits = oracle.nhwc_to_nchw(bits)
    assert not (~mask & (bits != 0)).any(), "killed outputs must be +0.0"
    refd, abd, ntd = oracle.conv_bwd_data(dy64, w64, (c["H"], c["W"]), st, pd, with_bound=True)
    check_values(nchw_of(dxd), refd, abd, ntd, tol, bf, "dense dX")
    rw, aw, nw = oracle.conv_bwd_weight(x64, dy64, (c["R"], c["S"]), st, pd, with_bound=True)
    kcrs = (lambda g: g.cpu().double().numpy()) if c["w_layout"] == "kcrs" else \
        (lambda g: oracle.krsc_to_kcrs(g.cpu().double().numpy()))
    for name, (o, skipped) in dws.items():
        check_values(kcrs(o), rw, aw, nw, tol, False, "dW " + name)
        check_dw_regrouped(o, dws["no_skip"][0], skipped, "dW %s against no skipping" % name)
    # the zero region covers output pixels [0, zero_px) of the first image;
    # it empties a block when it holds a whole chunk of output pixels
    chunk = 64 if bf else 32
    zero_px = c["P"] * c["Q"] if c["N"] > 1 else max(1, c["P"] // 2) * c["Q"]
    if zero_px >= chunk:
        assert dws["dy_skip"][1] > 0, "the zero dY band must empty a block"
    assert dws["x_skip"][1] >= dws["dy_skip"][1]
