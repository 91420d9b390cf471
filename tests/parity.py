"""Helpers shared by the GPU parity tests: run a layer through the C-ABI and
compare with the fp64 oracle.

Tolerance reading (stated once here, used by every parity test):
  * zero pattern: where the ReLU footprint of X is 0, dX must be the +0.0 bit
    pattern (exact);
  * normwise: max_i |g_i - o_i| / max_i |o_i| <= tol, per output tensor, with
    tol = 2e-2 for bf16 inputs and 1e-5 for fp32 inputs;
  * per element: |g_i - o_i| <= tol |o_i| + 2 L_i 2^-24 sum_j |a_j b_j|
    (+ 2^-8 |o_i| when the output is rounded to bf16), where L_i is the
    number of terms of output i and sum_j |a_j b_j| its conditioning, both
    from the oracle.  The second term is the standard bound of an fp32 sum of
    L_i exact products; it catches a wrong element that the normwise check
    alone could hide.
"""
import numpy as np
import torch

import oracle
import paper_2109_07710_amd as cb

U_ACC = 2.0 ** -24


def tol_for(dtype):
    return 2e-2 if dtype == "bf16" else 1e-5


def desc_of(spec, w_layout="krsc"):
    return cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad,
                            dtype=spec.dtype, w_layout=w_layout)


def to_dev(t, dev="cuda"):
    return {k: v.to(dev) for k, v in t.items()}


def gpu_backward(spec, t, flags=0, masked=None, dy_mask=False, w_layout="krsc", dev="cuda"):
    """Run the layer's data and weight gradients on the GPU.  t holds CPU
    tensors x [N,H,W,C], w [K,R,S,C], dy [N,P,Q,K].  Returns a dict with dx
    (NHWC, input dtype), dw (float32 in w_layout), the X footprint words and
    the workspaces."""
    masked = spec.masked if masked is None else masked
    desc = desc_of(spec, w_layout)
    d = to_dev(t, dev)
    w = d["w"]
    if w_layout == "kcrs":
        w = w.permute(0, 3, 1, 2).contiguous()
    out = {"desc": desc}
    xm = torch.zeros(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device=dev)
    cb.cbw_relu_mask_pack(desc, d["x"], xm)
    out["xmask"] = xm
    if spec.need_dx:
        dx = torch.empty_like(d["x"])
        if masked:
            ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED, dev)
            cb.conv_bwd_data_masked(desc, d["dy"], w, xm, dx, ws, flags)
        else:
            ws = cb.workspace(desc, cb.CBW_OP_BWD_DATA, dev)
            cb.conv_bwd_data(desc, d["dy"], w, dx, ws)
        out["dx"], out["ws_dx"] = dx, ws
    dym = None
    if dy_mask:
        dym = torch.zeros(max(cb.cbw_dy_mask_words(desc), 1), dtype=torch.int32, device=dev)
        cb.cbw_nonzero_mask_pack(desc.dtype, d["dy"].numel(), d["dy"], dym)
    shape = (spec.K, spec.R, spec.S, spec.C) if w_layout == "krsc" else (spec.K, spec.C, spec.R, spec.S)
    dw = torch.empty(shape, dtype=torch.float32, device=dev)
    ws2 = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT, dev)
    cb.conv_bwd_weight_sparse(desc, d["x"], d["dy"], dym, dw, ws2, flags)
    out["dw"], out["ws_dw"] = dw, ws2
    torch.cuda.synchronize()
    return out


def oracle_inputs(t):
    x64 = oracle.nhwc_to_nchw(t["x"].double().numpy())
    w64 = oracle.krsc_to_kcrs(t["w"].double().numpy())
    dy64 = oracle.nhwc_to_nchw(t["dy"].double().numpy())
    return x64, w64, dy64


def oracle_backward(spec, t, masked=None):
    masked = spec.masked if masked is None else masked
    x64, w64, dy64 = oracle_inputs(t)
    st, pd = (spec.stride, spec.stride), (spec.pad, spec.pad)
    mask = oracle.relu_mask(x64)
    res = {"mask": mask}
    if spec.need_dx:
        res["dx"], res["dx_abs"], res["dx_n"] = oracle.conv_bwd_data(
            dy64, w64, (spec.H, spec.W), st, pd, mask=mask if masked else None, with_bound=True)
    res["dw"], res["dw_abs"], res["dw_n"] = oracle.conv_bwd_weight(x64, dy64, (spec.R, spec.S), st, pd,
                                                                  with_bound=True)
    return res


def check_dw_regrouped(a, b, skipped, what):
    """Two weight gradients of the same inputs: bitwise equal when no block was
    skipped (same split ranges, same summation order); otherwise the skipping
    run's splits cover the live blocks in balanced ranges, so its fp32 sums are
    grouped differently and agree to fp32 reassociation (normwise 1e-5)."""
    if skipped == 0:
        assert torch.equal(a, b), what + ": differs without any skipped block"
        return 0.0
    err = (a.double() - b.double()).abs().max().item() / max(b.double().abs().max().item(), 1e-30)
    assert err <= 1e-5, "%s: normwise %.3e" % (what, err)
    return err


def dx_as_nchw(dx):
    return oracle.nhwc_to_nchw(dx.float().cpu().double().numpy())


def dx_bits_nchw(dx):
    if dx.dtype == torch.bfloat16:
        b = dx.cpu().view(torch.int16).numpy().astype(np.int64) & 0xFFFF
    else:
        b = dx.cpu().view(torch.int32).numpy().astype(np.int64) & 0xFFFFFFFF
    return oracle.nhwc_to_nchw(b)


def dw_as_kcrs(dw, w_layout="krsc"):
    a = dw.cpu().double().numpy()
    return oracle.krsc_to_kcrs(a) if w_layout == "krsc" else a


def check_values(g, o, absb, nterms, tol, out_bf16, what):
    """Normwise and per-element checks (see module docstring)."""
    err = np.abs(g - o)
    scale = np.abs(o).max()
    normwise = err.max() / scale if scale > 0 else err.max()
    bound = tol * np.abs(o) + 2.0 * nterms * U_ACC * absb
    if out_bf16:
        bound = bound + 2.0 ** -8 * np.abs(o)
    bad = err > bound
    assert normwise <= tol, "%s: normwise error %.3e > %.1e" % (what, normwise, tol)
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError("%s: %d elements outside the per-element bound; worst at %s: gpu %r oracle %r "
                             "bound %r" % (what, bad.sum(), i, g[i], o[i], bound[i]))
    return normwise


def check_zero_pattern(dx_bits, mask, what):
    """Every killed output must be the +0.0 bit pattern."""
    dead = ~mask
    nz = dx_bits[dead] != 0
    assert not nz.any(), "%s: %d killed outputs are not +0.0" % (what, int(nz.sum()))


def check_layer(spec, t, gpu, ref, masked=None, w_layout="krsc"):
    masked = spec.masked if masked is None else masked
    tol = tol_for(spec.dtype)
    errs = {}
    if spec.need_dx:
        g = dx_as_nchw(gpu["dx"])
        if masked:
            check_zero_pattern(dx_bits_nchw(gpu["dx"]), ref["mask"], spec.name + " dX")
        errs["dx"] = check_values(g, ref["dx"], ref["dx_abs"], ref["dx_n"], tol, spec.dtype == "bf16",
                                  spec.name + " dX")
    errs["dw"] = check_values(dw_as_kcrs(gpu["dw"], w_layout), ref["dw"], ref["dw_abs"], ref["dw_n"], tol, False,
                              spec.name + " dW")
    return errs
