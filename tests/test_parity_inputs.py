"""CPU checks that the GPU parity tests' inputs can show the mistakes they
are meant to catch: with the oracle alone, a deliberately broken variant of
the computation must move the compared outputs by far more than the test's
tolerance.  (At sigma = 0.01 attention is nearly uniform and a wrong
attention moves log p by about 1e-8, so such inputs would hide it.)"""
import numpy as np
import pytest

import oracle
from paper_1605_04809_amd.workloads import random_annotations, unit_gain
from tests.parity_cases import ATT, ATT_CASES, CLAMP_SCALES, PAPER_SIGNAL

TOL_HS = 1e-4      # intermediates and log p in the high-signal GPU tests
TOL_ALPHA = 1e-5   # attention weights there


def _run(wl, ctx, params=None):
    c = wl.cfg
    m = oracle.Model(params or wl.params, c.V_src, c.V, c.E, c.H, c.A)
    cx, pc = oracle.keys_from_annotations(m, ctx, wl.src_len)
    return oracle.score_batch(m, cx, pc, wl.src_len, wl.s_prev, wl.y_prev, wl.sent_id, wl.req), pc


def _zero_v(p):
    p["att_v"] = np.zeros_like(p["att_v"])


def _zero_upper_query(p):  # what a bug in the lanes past the first 256 attention columns would do
    q = p["att_Wq"].copy()
    q[:, 256:] = 0
    p["att_Wq"] = q


@pytest.mark.parametrize("cfg,seed", [(ATT.replace(**ATT_CASES["g1_16w"]), 72), (PAPER_SIGNAL, 74)],
                         ids=["A1024_small", "paper_dims"])
@pytest.mark.parametrize("broken", [_zero_v, _zero_upper_query], ids=["uniform_attention", "upper_query_lanes"])
def test_attention_mistakes_move_outputs_far_beyond_the_bar(cfg, seed, broken):
    wl = unit_gain(cfg)
    if cfg is PAPER_SIGNAL:  # the oracle's vocabulary pass dominates; 48 rows suffice here
        for k in ("sent_id", "s_prev", "y_prev", "req"):
            setattr(wl, k, getattr(wl, k)[:48])
    ctx = random_annotations(cfg, seed=seed)
    ref, _ = _run(wl, ctx)
    p = dict(wl.params)
    broken(p)
    bad, _ = _run(wl, ctx, p)
    d_alpha = np.abs(bad["alpha"] - ref["alpha"]).max()
    d_logp = np.abs(bad["logp"] - ref["logp"]).max()
    print(f"max |d alpha| {d_alpha:.3g}, max |d logp| {d_logp:.3g}")
    assert d_alpha >= 100 * TOL_ALPHA and d_alpha >= 100 * TOL_HS
    assert d_logp >= 100 * TOL_HS


def _clamped_factor_alpha(pctx, q, v, sent_id, src_len):
    """Attention weights scored from factors 2^{2 log2(e) x} whose exponents
    are clamped to [-126, 126] (the shortcut the GPU kernels take for
    moderate keys and queries), in fp64."""
    c = 2.0 / np.log(2.0)
    out = np.zeros((len(sent_id), pctx.shape[1]))
    for b, s in enumerate(sent_id):
        L = src_len[s]
        K = np.exp2(np.clip(pctx[s, :L] * c, -126, 126))
        Q = np.exp2(np.clip(q[b] * c, -126, 126))
        e = ((-2.0 * v)[None, :] / (K * Q[None, :] + 1.0)).sum(axis=1)
        e = np.exp(e - e.max())
        out[b, :L] = e / e.sum()
    return out


@pytest.mark.parametrize("case", ["g4_16w", "per_row"])
def test_large_keys_defeat_clamped_factors(case):
    """On the inputs of test_keys_beyond_the_factor_range_every_row, scoring
    every term from clamped factors would miss the oracle's attention weights
    by more than 100 times the bar, so that test tells exact scoring from the
    clamped shortcut."""
    cfg = ATT.replace(**ATT_CASES[case])
    wl = unit_gain(cfg, **CLAMP_SCALES)
    ctx = random_annotations(cfg, seed=72)
    ref, pctx = _run(wl, ctx)
    q = ref["s1"] @ wl.params["att_Wq"].astype(np.float64)
    with np.errstate(over="ignore"):
        a = _clamped_factor_alpha(pctx, q, wl.params["att_v"].astype(np.float64), wl.sent_id, wl.src_len)
    d = np.abs(a - ref["alpha"]).max()
    print(f"max |pctx| {np.abs(pctx).max():.1f}, max |q| {np.abs(q).max():.1f}, clamped-factor |d alpha| {d:.3g}")
    assert d >= 100 * TOL_ALPHA


def _drop_bias(p):  # what skipping the k group that holds the bias row would do
    p["out_b"] = np.zeros_like(p["out_b"])


def _drop_last_readout_rows(p):  # what skipping the last real k rows (E - 4 .. E - 1) would do
    w = p["out_W"].copy()
    w[-4:, :] = 0
    p["out_W"] = w


@pytest.mark.parametrize("E", [244, 500])
@pytest.mark.parametrize("broken", [_drop_bias, _drop_last_readout_rows], ids=["bias", "last_rows"])
def test_vocabulary_padding_mistakes_move_log_p(E, broken):
    """The inputs of the GPU test at the vocabulary kernel's skipped padding:
    dropping the bias row or the readout's last four rows from the output
    projection moves log p far beyond the 1e-4 bar."""
    from paper_1605_04809_amd.workloads import CONFIGS
    wl = unit_gain(CONFIGS["tiny"].replace(E=E, V=3001, B=70, S=2, len_lo=3, len_hi=9, Tpad=9, seed=31 + E))
    c = wl.cfg
    m = oracle.Model(wl.params, c.V_src, c.V, c.E, c.H, c.A)
    ctx, pctx, _ = oracle.encode(m, wl.src_ids, wl.src_len)
    ref = oracle.score_batch(m, ctx, pctx, wl.src_len, wl.s_prev, wl.y_prev, wl.sent_id, wl.req, intermediates=False)
    p = dict(wl.params)
    broken(p)
    mb = oracle.Model(p, c.V_src, c.V, c.E, c.H, c.A)
    bad = oracle.score_batch(mb, ctx, pctx, wl.src_len, wl.s_prev, wl.y_prev, wl.sent_id, wl.req, intermediates=False)
    d = np.abs(bad["logp"] - ref["logp"]).max()
    print(f"E={E}: max |d logp| {d:.3g}")
    assert d >= 100 * TOL_HS
