"""Definition-level nested-loop convolution for tiny shapes.

TEST INFRASTRUCTURE ONLY (part of the oracle): pure-Python loops, used to pin
the C oracle on inputs small enough for Python to finish in well under a
second.  It shares no code with the C oracle and none with the HIP library.

Notation follows the paper (Sec. II-A, Sec. IV-B): input [C,H,W], filters
[M,C,R,S], output [M,U,V]; here M is K and [U,V] is [P,Q].  Arrays are nested
Python lists or numpy arrays indexed [n][c][h][w], [k][c][r][s], [n][k][p][q].
Cross-correlation with zero padding.
"""


def out_size(h, r, stride, pad):
    """Number of output rows of a padded, strided window sweep."""
    return (h + 2 * pad - r) // stride + 1


def conv_fwd(x, w, stride=(1, 1), pad=(0, 0)):
    """Y[n][k][p][q] = sum over c, r, s of X[n][c][p*sh-ph+r][q*sw-pw+s] * W[k][c][r][s]."""
    n_, c_, h_, w_ = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    k_, r_, s_ = len(w), len(w[0][0]), len(w[0][0][0])
    p_ = out_size(h_, r_, stride[0], pad[0])
    q_ = out_size(w_, s_, stride[1], pad[1])
    y = [[[[0.0] * q_ for _ in range(p_)] for _ in range(k_)] for _ in range(n_)]
    for n in range(n_):
        for k in range(k_):
            for p in range(p_):
                for q in range(q_):
                    acc = 0.0
                    for c in range(c_):
                        for r in range(r_):
                            for s in range(s_):
                                h = p * stride[0] - pad[0] + r
                                ww = q * stride[1] - pad[1] + s
                                if 0 <= h < h_ and 0 <= ww < w_:
                                    acc += float(x[n][c][h][ww]) * float(w[k][c][r][s])
                    y[n][k][p][q] = acc
    return y


def conv_bwd_data(dy, w, hw, stride=(1, 1), pad=(0, 0)):
    """dX as the transpose of conv_fwd, written by scattering.

    Every forward term X[n][c][h][w] * W[k][c][r][s] -> Y[n][k][p][q]
    contributes dY[n][k][p][q] * W[k][c][r][s] to dX[n][c][h][w].  Scattering
    from each (p, q) is a different loop order from the C oracle's gather over
    (k, r, s), so the two do not share an indexing mistake.
    """
    h_, w_ = hw
    n_, k_, p_, q_ = len(dy), len(dy[0]), len(dy[0][0]), len(dy[0][0][0])
    c_, r_, s_ = len(w[0]), len(w[0][0]), len(w[0][0][0])
    dx = [[[[0.0] * w_ for _ in range(h_)] for _ in range(c_)] for _ in range(n_)]
    for n in range(n_):
        for k in range(k_):
            for p in range(p_):
                for q in range(q_):
                    g = float(dy[n][k][p][q])
                    for c in range(c_):
                        for r in range(r_):
                            for s in range(s_):
                                h = p * stride[0] - pad[0] + r
                                ww = q * stride[1] - pad[1] + s
                                if 0 <= h < h_ and 0 <= ww < w_:
                                    dx[n][c][h][ww] += g * float(w[k][c][r][s])
    return dx


def conv_bwd_weight(x, dy, rs, stride=(1, 1), pad=(0, 0)):
    """dW by scattering every forward term's dY * X into its filter tap."""
    r_, s_ = rs
    n_, c_, h_, w_ = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    k_, p_, q_ = len(dy[0]), len(dy[0][0]), len(dy[0][0][0])
    dw = [[[[0.0] * s_ for _ in range(r_)] for _ in range(c_)] for _ in range(k_)]
    for n in range(n_):
        for k in range(k_):
            for p in range(p_):
                for q in range(q_):
                    g = float(dy[n][k][p][q])
                    for c in range(c_):
                        for r in range(r_):
                            for s in range(s_):
                                h = p * stride[0] - pad[0] + r
                                ww = q * stride[1] - pad[1] + s
                                if 0 <= h < h_ and 0 <= ww < w_:
                                    dw[k][c][r][s] += g * float(x[n][c][h][ww])
    return dw
