"""Tolerances for the bf16-weight parity tests, derived from how the GPU
path rounds.

Both sides use the same bf16 weights; the GPU path also rounds every
activation operand of its MFMA products to bf16 (nearest even: relative
error at most 2^-8, about uniform within the rounding interval, so rms
u = 2^-8 / sqrt(3)), while the oracle keeps them in fp64.  A pre-activation
y = sum_k a_k w_k then carries an error of standard deviation about
u * sigma_w * ||a|| (independent roundings), with ||a|| the norm of the row's
operand vector, taken from the oracle's own values (largest over the rows).
Standard deviations propagate layer by layer:
  - the GRU cell passes pre-activation errors on with gain at most about 1/2
    (tanh' <= 1 times 1 - z ~ 1/2; sigma' <= 1/4 times |h - n| <= 2), and its
    input state's error with gain <= 1 (through z);
  - the readout's tanh has gain <= 1, and a product with N(0, sigma_w)
    weights over K inputs carries an input error e as sigma_w sqrt(K) e;
  - the annotations come from the bf16 encoder, a recurrence of such steps
    that contracts (z ~ 1/2), so its error is at most twice a step's; the
    context is a convex combination of annotations;
  - a score's error is ||v||_2 times the key and query errors (tanh' <= 1),
    and softmax moves alpha_i by at most 2 alpha_i times it.
A bar is 6.5 standard deviations: the largest of up to 10^8 Gaussian
errors stays below it.  The context and the readout are also stored in bf16
between kernels (the only form their consumers read), so their bars add that
rounding itself: at most 2^-8 of the largest value.
"""
import numpy as np

U_RMS = 2.0 ** -8 / np.sqrt(3.0)
NSIG = 6.5


def bf16_bars(cfg, wl, ref, ctx, rows=None):
    """Per-output bars for a bf16-weight workload ``wl``: ``ref`` holds the
    oracle's outputs with intermediates for ``rows`` of the batch (all rows
    if None), ``ctx`` the oracle's annotations [S, Tpad, 2H]."""
    sel = slice(None) if rows is None else rows
    sw, u, H = cfg.sigma_w, U_RMS, cfg.H
    norm = lambda *a: np.sqrt(sum((np.asarray(x, np.float64) ** 2).sum(-1) for x in a)).max()
    emb = wl.params["emb_tgt"].astype(np.float64)
    yp = wl.y_prev[sel]
    x = np.where((yp >= 0)[:, None], emb[np.maximum(yp, 0)], 0.0)
    s1 = 0.5 * u * sw * norm(x, wl.s_prev[sel])
    s_new = np.hypot(s1, 0.5 * u * sw * norm(ref["s1"], ref["c"]))
    t = np.hypot(u * sw * norm(ref["s_new"], x, ref["c"]), sw * np.sqrt(H) * s_new)
    hmax = max(norm(ctx[..., :H]), norm(ctx[..., H:]))
    enc = 2.0 * 0.5 * u * sw * np.sqrt(cfg.E * cfg.sigma_emb ** 2 + hmax ** 2)
    c = enc
    dq = np.hypot(u * sw * norm(ref["s1"]), sw * np.sqrt(H) * s1)
    dk = np.hypot(u * sw * norm(ctx), sw * np.sqrt(2 * H) * enc)
    de = np.linalg.norm(wl.params["att_v"].astype(np.float64)) * np.hypot(dq, dk)
    alpha = 2.0 * float(ref["alpha"].max()) * de
    bars = {k: NSIG * v for k, v in dict(s1=s1, s_new=s_new, t=t, c=c, alpha=alpha).items()}
    bars["c"] += 2.0 ** -8 * float(np.abs(ref["c"]).max())
    bars["t"] += 2.0 ** -8 * float(np.abs(ref["t"]).max())
    return bars
