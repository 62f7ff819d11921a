"""Pins for the fp64 oracle, checked against things other than itself.

Each pin ties one part of the oracle to a library routine (``torch.nn.GRUCell``,
``torch.softmax``, ``torch.logsumexp`` in float64), a closed form, an
invariant, or brute force on tiny inputs.  The model equations are the
DL4MT conditional GRU the paper names (Sections 1 and 3); the step is the
forward step of Section 5.1.  ``test_planted_mistakes`` rebuilds the oracle
with one deliberate mistake at a time and checks that these pins fail.
"""
import math
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_1605_04809_amd.workloads import param_shapes, PARAM_ORDER

DIMS = dict(V_src=41, V=53, E=6, H=5, A=7)


def rand_params(seed, V_src, V, E, H, A, sigma=0.5):
    rng = np.random.default_rng(seed)
    shapes = param_shapes(V_src, V, E, H, A)
    return {n: (rng.standard_normal(shapes[n]) * sigma).astype(np.float32) for n in PARAM_ORDER}


def make_model(seed=0, **kw):
    d = dict(DIMS)
    d.update(kw)
    p = rand_params(seed, **d)
    return p, oracle.Model(p, **d)


def torch_cell(W, U, b_in, b_st):
    nin, G = W.shape
    H = G // 3
    cell = torch.nn.GRUCell(nin, H).double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(W.astype(np.float64).T))
        cell.weight_hh.copy_(torch.from_numpy(U.astype(np.float64).T))
        cell.bias_ih.copy_(torch.from_numpy(np.zeros(G) if b_in is None else b_in.astype(np.float64)))
        cell.bias_hh.copy_(torch.from_numpy(np.zeros(G) if b_st is None else b_st.astype(np.float64)))
    return cell


# --------------------------------------------------------------------- GRU


@pytest.mark.parametrize("bias_side", ["input", "state", "both"])
def test_gru_matches_torch_grucell(bias_side):
    rng = np.random.default_rng(1)
    n, nin, H = 9, 7, 6
    u = rng.standard_normal((n, nin))
    h = np.tanh(rng.standard_normal((n, H)))
    W = rng.standard_normal((nin, 3 * H)).astype(np.float32)
    U = rng.standard_normal((H, 3 * H)).astype(np.float32)
    b = rng.standard_normal(3 * H).astype(np.float32)
    b2 = rng.standard_normal(3 * H).astype(np.float32)
    b_in = b if bias_side in ("input", "both") else None
    b_st = (b2 if bias_side == "both" else b) if bias_side in ("state", "both") else None
    got = oracle.gru(u, h, W, U, b_in, b_st)
    with torch.no_grad():
        want = torch_cell(W, U, b_in, b_st)(torch.from_numpy(u), torch.from_numpy(h)).numpy()
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-13)


def test_gru_bias_placement_matters():
    """The same bias on the input side and on the state side differ through r."""
    rng = np.random.default_rng(2)
    u, h = rng.standard_normal((4, 3)), rng.standard_normal((4, 5))
    W = rng.standard_normal((3, 15)).astype(np.float32)
    U = rng.standard_normal((5, 15)).astype(np.float32)
    b = (3 * rng.standard_normal(15)).astype(np.float32)
    assert np.abs(oracle.gru(u, h, W, U, b, None) - oracle.gru(u, h, W, U, None, b)).max() > 1e-3


def test_gru_convex_bound_and_saturated_update_gate():
    rng = np.random.default_rng(3)
    n, nin, H = 50, 4, 8
    u = 3 * rng.standard_normal((n, nin))
    h = 2 * rng.standard_normal((n, H))
    W = rng.standard_normal((nin, 3 * H)).astype(np.float32)
    U = rng.standard_normal((H, 3 * H)).astype(np.float32)
    out = oracle.gru(u, h, W, U, None, None)
    assert np.all(np.abs(out) <= np.maximum(np.abs(h), 1.0) + 1e-15)
    b = np.zeros(3 * H, np.float32)
    b[H:2 * H] = 60.0          # z -> 1: the state passes through unchanged
    np.testing.assert_allclose(oracle.gru(u, h, W, U, b, None), h, rtol=0, atol=1e-20 + 1e-12)
    b[H:2 * H] = -60.0         # z -> 0: the state is the candidate; with zero U_n and W_n, n = 0
    W0, U0 = W.copy(), U.copy()
    W0[:, 2 * H:] = 0
    U0[:, 2 * H:] = 0
    np.testing.assert_allclose(oracle.gru(u, h, W0, U0, b, None), 0.0, atol=1e-12)


# ----------------------------------------------------------------- encoder


def torch_encode(p, src_ids, src_len, H):
    fwd = torch_cell(p["enc_f_W"], p["enc_f_U"], p["enc_f_b"], None)
    bwd = torch_cell(p["enc_b_W"], p["enc_b_U"], p["enc_b_b"], None)
    S, T = src_ids.shape
    ctx = np.zeros((S, T, 2 * H))
    with torch.no_grad():
        for s in range(S):
            L = int(src_len[s])
            x = torch.from_numpy(p["emb_src"][src_ids[s, :L]].astype(np.float64))
            h = torch.zeros(1, H, dtype=torch.float64)
            for i in range(L):
                h = fwd(x[i:i + 1], h)
                ctx[s, i, :H] = h[0].numpy()
            h = torch.zeros(1, H, dtype=torch.float64)
            for i in reversed(range(L)):
                h = bwd(x[i:i + 1], h)
                ctx[s, i, H:] = h[0].numpy()
    return ctx


def test_encoder_matches_torch_grucell_scan():
    p, m = make_model(4)
    rng = np.random.default_rng(5)
    S, T = 3, 9
    src_len = np.array([9, 4, 1], np.int32)
    src_ids = rng.integers(0, DIMS["V_src"], (S, T)).astype(np.int32)
    ctx, pctx, s0 = oracle.encode(m, src_ids, src_len)
    want = torch_encode(p, src_ids, src_len, DIMS["H"])
    np.testing.assert_allclose(ctx, want, rtol=0, atol=1e-13)
    for s in range(S):
        assert np.all(ctx[s, src_len[s]:] == 0) and np.all(pctx[s, src_len[s]:] == 0)
    # keys: pctx = ctx Wc + b (torch.nn.functional.linear), s0 = tanh(mean ctx . Winit + b)
    with torch.no_grad():
        for s in range(S):
            L = src_len[s]
            c = torch.from_numpy(ctx[s, :L])
            kw = torch.nn.functional.linear(c, torch.from_numpy(p["att_Wc"].T.astype(np.float64)),
                                            torch.from_numpy(p["att_b"].astype(np.float64)))
            np.testing.assert_allclose(pctx[s, :L], kw.numpy(), rtol=0, atol=1e-12)
            mean = c.mean(0, keepdim=True)
            s0w = torch.tanh(torch.nn.functional.linear(
                mean, torch.from_numpy(p["init_W"].T.astype(np.float64)),
                torch.from_numpy(p["init_b"].astype(np.float64))))
            np.testing.assert_allclose(s0[s], s0w[0].numpy(), rtol=0, atol=1e-12)


def test_encoder_backward_is_forward_on_reversed_ids_and_padding_is_ignored():
    p, m = make_model(6)
    rng = np.random.default_rng(7)
    T, L, H = 8, 6, DIMS["H"]
    ids = rng.integers(0, DIMS["V_src"], (1, T)).astype(np.int32)
    ctx, pctx, s0 = oracle.encode(m, ids, np.array([L], np.int32))
    # backward direction == a forward pass with the backward weights on the reversed sentence
    p2 = dict(p)
    p2["enc_f_W"], p2["enc_f_U"], p2["enc_f_b"] = p["enc_b_W"], p["enc_b_U"], p["enc_b_b"]
    m2 = oracle.Model(p2, **DIMS)
    rev = ids.copy()
    rev[0, :L] = ids[0, :L][::-1]
    ctx2, _, _ = oracle.encode(m2, rev, np.array([L], np.int32))
    np.testing.assert_allclose(ctx[0, :L, H:], ctx2[0, :L, :H][::-1], rtol=0, atol=1e-14)
    # padding ids and extra padded positions change nothing
    ids_b = np.concatenate([ids, rng.integers(0, DIMS["V_src"], (1, 5)).astype(np.int32)], 1)
    ids_b[0, L:] = rng.integers(0, DIMS["V_src"], T + 5 - L)
    ctx_b, pctx_b, s0_b = oracle.encode(m, ids_b, np.array([L], np.int32))
    np.testing.assert_array_equal(ctx_b[:, :T], ctx)
    np.testing.assert_array_equal(s0_b, s0)
    np.testing.assert_array_equal(pctx_b[:, :T], pctx)


def test_initial_state_closed_form():
    p, _ = make_model(8)
    p["init_W"][:] = 0
    m = oracle.Model(p, **DIMS)
    ids = np.zeros((2, 4), np.int32)
    _, _, s0 = oracle.encode(m, ids, np.array([4, 2], np.int32))
    np.testing.assert_allclose(s0, np.tanh(p["init_b"].astype(np.float64))[None].repeat(2, 0),
                               rtol=0, atol=1e-15)


def test_keys_from_annotations_closed_forms_and_encoder_agreement():
    """Keys from given annotations: zero key weights give the bias; a single
    non-zero annotation entry gives that entry times its weight row plus the
    bias (one rounding); padding contents are ignored; and fed the encoder's
    own annotations (rounded to fp32, the entry point's input type) it gives
    the encoder's keys up to that rounding."""
    p, m = make_model(31)
    H, A, C = DIMS["H"], DIMS["A"], 2 * DIMS["H"]
    S, T = 3, 6
    src_len = np.array([6, 2, 1], np.int32)
    rng = np.random.default_rng(32)
    ann = rng.standard_normal((S, T, C)).astype(np.float32)
    # zero key weights: pctx = att_b below the length, 0 past it; ctx is the input widened, 0 past the length
    p0 = dict(p)
    p0["att_Wc"] = np.zeros_like(p["att_Wc"])
    ctx, pctx = oracle.keys_from_annotations(oracle.Model(p0, **DIMS), ann, src_len)
    for s in range(S):
        L = src_len[s]
        np.testing.assert_array_equal(pctx[s, :L], np.broadcast_to(p["att_b"].astype(np.float64), (L, A)))
        np.testing.assert_array_equal(ctx[s, :L], ann[s, :L].astype(np.float64))
        assert np.all(pctx[s, L:] == 0) and np.all(ctx[s, L:] == 0)
    # one non-zero entry x at (s, i, k): pctx[s, i] = b + x * Wc[k] exactly, other positions b
    one = np.zeros_like(ann)
    one[0, 3, 4] = np.float32(1.75)
    _, pctx = oracle.keys_from_annotations(m, one, src_len)
    want = p["att_b"].astype(np.float64) + 1.75 * p["att_Wc"][4].astype(np.float64)
    np.testing.assert_array_equal(pctx[0, 3], want)
    np.testing.assert_array_equal(pctx[0, 2], p["att_b"].astype(np.float64))
    # padding contents are ignored
    junk = ann.copy()
    for s in range(S):
        junk[s, src_len[s]:] = 1e6
    np.testing.assert_array_equal(oracle.keys_from_annotations(m, junk, src_len)[1],
                                  oracle.keys_from_annotations(m, ann, src_len)[1])
    # the encoder's annotations give the encoder's keys, within the fp32 rounding of the annotations
    ids = rng.integers(0, DIMS["V_src"], (S, T)).astype(np.int32)
    ectx, epctx, _ = oracle.encode(m, ids, src_len)
    c32 = ectx.astype(np.float32)
    _, kpctx = oracle.keys_from_annotations(m, c32, src_len)
    bound = (np.abs(ectx - c32.astype(np.float64)) @ np.abs(p["att_Wc"].astype(np.float64))) + 1e-15
    assert np.all(np.abs(kpctx - epctx) <= bound)
    assert np.abs(kpctx - epctx).max() > 0  # the rounding is visible, so the bound is doing the work


def test_fp64_states_equal_the_fp32_path_on_fp32_values():
    """The step with fp64 input states (used for stepwise phrase scoring)
    equals the step with fp32 states when the states are fp32 values: the
    two entry points differ only in how the state is widened."""
    p, m = make_model(33)
    src_ids, src_len, s_prev, y_prev, sent_id, req = step_inputs(34)
    ctx, pctx, _ = oracle.encode(m, src_ids, src_len)
    a = oracle.score_batch(m, ctx, pctx, src_len, s_prev, y_prev, sent_id, req)
    b = oracle.score_batch(m, ctx, pctx, src_len, s_prev.astype(np.float64), y_prev, sent_id, req)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    # and an fp64 state that is not an fp32 value is used as such (not rounded to fp32)
    s64 = s_prev.astype(np.float64) + 1e-12
    c = oracle.score_batch(m, ctx, pctx, src_len, s64, y_prev, sent_id, req)
    assert np.abs(c["s_new"] - a["s_new"]).max() > 0


# ------------------------------------------------------------ whole step


def torch_step(p, ctx, pctx, src_len, s_prev, y_prev, sent_id, req):
    """The decoder step composed from torch library routines (float64)."""
    E = p["emb_tgt"].shape[1]
    d = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    with torch.no_grad():
        emb = d(p["emb_tgt"])
        x = torch.where(torch.from_numpy(y_prev >= 0)[:, None],
                        emb[torch.from_numpy(np.maximum(y_prev, 0)).long()],
                        torch.zeros(1, E, dtype=torch.float64))
        s1 = torch_cell(p["g1_W"], p["g1_U"], p["g1_b"], None)(x, d(s_prev))
        q = s1 @ d(p["att_Wq"])
        sid = torch.from_numpy(sent_id).long()
        P, Cx = d(pctx)[sid], d(ctx)[sid]
        e = torch.tanh(P + q[:, None, :]) @ d(p["att_v"])
        T = P.shape[1]
        mask = torch.arange(T)[None, :] < torch.from_numpy(src_len)[sid][:, None]
        alpha = torch.softmax(e.masked_fill(~mask, -math.inf), dim=1)
        c = (alpha[:, :, None] * Cx).sum(1)
        s2 = torch_cell(p["g2_Wc"], p["g2_U"], None, p["g2_b"])(c, s1)
        t = torch.tanh(s2 @ d(p["ro_Ws"]) + x @ d(p["ro_Wy"]) + c @ d(p["ro_Wc"]) + d(p["ro_b"]))
        z = t @ d(p["out_W"]) + d(p["out_b"])
        logZ = torch.logsumexp(z, dim=1)
        logp = z[torch.arange(len(req)), torch.from_numpy(req).long()] - logZ
    return dict(logp=logp.numpy(), logZ=logZ.numpy(), s_new=s2.numpy(), s1=s1.numpy(),
                alpha=alpha.numpy(), c=c.numpy(), t=t.numpy())


def step_inputs(seed, S=3, T=7, B=11, lens=(7, 3, 1), V=None, H=None, bos=True):
    rng = np.random.default_rng(seed)
    V = V or DIMS["V"]
    H = H or DIMS["H"]
    src_len = np.array(lens, np.int32)
    src_ids = rng.integers(0, DIMS["V_src"], (S, T)).astype(np.int32)
    s_prev = np.tanh(2 * rng.standard_normal((B, H))).astype(np.float32)
    y_prev = rng.integers(0, V, B).astype(np.int32)
    if bos:
        y_prev[0] = -1
    sent_id = rng.integers(0, S, B).astype(np.int32)
    req = rng.integers(0, V, B).astype(np.int32)
    return src_ids, src_len, s_prev, y_prev, sent_id, req


def test_step_matches_torch_composition():
    p, m = make_model(9)
    src_ids, src_len, s_prev, y_prev, sent_id, req = step_inputs(10)
    ctx, pctx, _ = oracle.encode(m, src_ids, src_len)
    got = oracle.score_batch(m, ctx, pctx, src_len, s_prev, y_prev, sent_id, req)
    want = torch_step(p, ctx, pctx, src_len, s_prev, y_prev, sent_id, req)
    for k in want:
        np.testing.assert_allclose(got[k], want[k], rtol=0, atol=1e-12, err_msg=k)


def test_step_row_independence_and_permutation():
    p, m = make_model(11)
    src_ids, src_len, s_prev, y_prev, sent_id, req = step_inputs(12, B=9)
    ctx, pctx, _ = oracle.encode(m, src_ids, src_len)
    full = oracle.score_batch(m, ctx, pctx, src_len, s_prev, y_prev, sent_id, req)
    for b in (0, 4, 8):
        one = oracle.score_batch(m, ctx, pctx, src_len, s_prev[b:b + 1], y_prev[b:b + 1],
                                 sent_id[b:b + 1], req[b:b + 1])
        for k in ("logp", "s_new", "logZ", "alpha", "c", "t"):
            np.testing.assert_array_equal(one[k][0], full[k][b])
    perm = np.random.default_rng(0).permutation(9)
    pm = oracle.score_batch(m, ctx, pctx, src_len, s_prev[perm], y_prev[perm], sent_id[perm], req[perm])
    for k in ("logp", "s_new", "logZ"):
        np.testing.assert_array_equal(pm[k], full[k][perm])


def test_attention_invariants_and_closed_forms():
    p, m = make_model(13)
    src_ids, src_len, s_prev, y_prev, sent_id, req = step_inputs(14, B=12)
    ctx, pctx, _ = oracle.encode(m, src_ids, src_len)
    out = oracle.score_batch(m, ctx, pctx, src_len, s_prev, y_prev, sent_id, req)
    a = out["alpha"]
    L = src_len[sent_id]
    T = a.shape[1]
    assert np.all(a >= 0)
    np.testing.assert_allclose(a.sum(1), 1.0, rtol=0, atol=1e-14)
    assert np.all(a[np.arange(T)[None, :] >= L[:, None]] == 0)
    for b in np.nonzero(L == 1)[0]:     # one source position: all weight on it, c = ctx_0
        assert a[b, 0] == 1.0
        np.testing.assert_allclose(out["c"][b], ctx[sent_id[b], 0], rtol=0, atol=1e-15)
    # zero scoring vector: uniform weights over the unmasked positions, c = mean annotation
    p0 = dict(p)
    p0["att_v"] = np.zeros_like(p["att_v"])
    out0 = oracle.score_batch(oracle.Model(p0, **DIMS), ctx, pctx, src_len, s_prev, y_prev,
                              sent_id, req)
    for b in range(len(L)):
        np.testing.assert_allclose(out0["alpha"][b, :L[b]], 1.0 / L[b], rtol=0, atol=1e-15)
        np.testing.assert_allclose(out0["c"][b], ctx[sent_id[b], :L[b]].mean(0), rtol=0, atol=1e-14)
    # garbage in padded positions of ctx / pctx changes nothing
    ctx_g, pctx_g = ctx.copy(), pctx.copy()
    for s in range(len(src_len)):
        ctx_g[s, src_len[s]:] = 1e3
        pctx_g[s, src_len[s]:] = -1e3
    outg = oracle.score_batch(m, ctx_g, pctx_g, src_len, s_prev, y_prev, sent_id, req)
    for k in ("logp", "s_new", "alpha", "c"):
        np.testing.assert_array_equal(outg[k], out[k])


def test_readout_closed_form():
    p, _ = make_model(15)
    for k in ("ro_Ws", "ro_Wy", "ro_Wc"):
        p[k] = np.zeros_like(p[k])
    m = oracle.Model(p, **DIMS)
    src_ids, src_len, s_prev, y_prev, sent_id, req = step_inputs(16)
    ctx, pctx, _ = oracle.encode(m, src_ids, src_len)
    out = oracle.score_batch(m, ctx, pctx, src_len, s_prev, y_prev, sent_id, req)
    np.testing.assert_allclose(out["t"], np.tanh(p["ro_b"].astype(np.float64))[None].repeat(len(req), 0),
                               rtol=0, atol=1e-15)


def test_bos_row_uses_zero_embedding():
    p, m = make_model(17)
    src_ids, src_len, s_prev, y_prev, sent_id, req = step_inputs(18, bos=False)
    ctx, pctx, _ = oracle.encode(m, src_ids, src_len)
    y_bos = y_prev.copy()
    y_bos[:] = -1
    a = oracle.score_batch(m, ctx, pctx, src_len, s_prev, y_bos, sent_id, req)
    p2 = dict(p)
    p2["emb_tgt"] = p["emb_tgt"].copy()
    p2["emb_tgt"][5] = 0
    b = oracle.score_batch(oracle.Model(p2, **DIMS), ctx, pctx, src_len, s_prev,
                           np.full_like(y_prev, 5), sent_id, req)
    for k in ("logp", "s_new", "t"):
        np.testing.assert_array_equal(a[k], b[k])


# ------------------------------------------------------------- log-softmax


def test_vocab_logsoftmax_brute_force_and_library():
    rng = np.random.default_rng(19)
    B, E, V = 5, 4, 37
    t = np.tanh(rng.standard_normal((B, E)))
    W = (3 * rng.standard_normal((E, V))).astype(np.float32)
    b = rng.standard_normal(V).astype(np.float32)
    req = rng.integers(0, V, B).astype(np.int32)
    logp, logZ, la = oracle.vocab_logsoftmax(t, W, b, req, full=True)
    for r in range(B):
        z = [math.fsum(float(t[r, k]) * float(W[k, v]) for k in range(E)) + float(b[v]) for v in range(V)]
        lz = math.log(math.fsum(math.exp(zv) for zv in z))
        assert abs(logZ[r] - lz) < 1e-12
        assert abs(logp[r] - (z[req[r]] - lz)) < 1e-12
    zt = torch.from_numpy(t) @ torch.from_numpy(W.astype(np.float64)) + torch.from_numpy(b.astype(np.float64))
    np.testing.assert_allclose(logZ, torch.logsumexp(zt, 1).numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(la, torch.log_softmax(zt, 1).numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(np.exp(la).sum(1), 1.0, rtol=0, atol=1e-13)
    assert np.all(la <= 0)


def test_vocab_logsoftmax_uniform_closed_form():
    for V in (1, 7, 100000):
        t = np.ones((2, 3))
        logp, logZ, _ = oracle.vocab_logsoftmax(t, np.zeros((3, V), np.float32), np.zeros(V, np.float32),
                                                np.array([0, V - 1], np.int32))
        np.testing.assert_allclose(logp, -math.log(V), rtol=0, atol=1e-12)
        np.testing.assert_allclose(logZ, math.log(V), rtol=0, atol=1e-12)


def test_vocab_logsoftmax_large_logits_are_stable():
    t = np.ones((1, 1))
    W = np.array([[1000.0, 999.0, -1000.0]], np.float32)
    logp, logZ, _ = oracle.vocab_logsoftmax(t, W, np.zeros(3, np.float32), np.array([1], np.int32))
    want = 1000.0 + math.log(1 + math.exp(-1) + math.exp(-2000))
    assert abs(logZ[0] - want) < 1e-12 and abs(logp[0] - (999.0 - want)) < 1e-12


def test_full_vocab_sums_to_one_through_the_step():
    """Requesting every word of a row: the probabilities over V sum to 1."""
    p, m = make_model(20)
    src_ids, src_len, s_prev, y_prev, sent_id, req = step_inputs(21, B=3)
    ctx, pctx, _ = oracle.encode(m, src_ids, src_len)
    V = DIMS["V"]
    rows = np.repeat(np.arange(3), V)
    out = oracle.score_batch(m, ctx, pctx, src_len, s_prev[rows], y_prev[rows], sent_id[rows],
                             np.tile(np.arange(V, dtype=np.int32), 3), intermediates=False)
    np.testing.assert_allclose(np.exp(out["logp"]).reshape(3, V).sum(1), 1.0, rtol=0, atol=1e-13)


# ------------------------------------------------------------ error codes


def test_out_of_range_ids_are_rejected():
    p, m = make_model(22)
    src_ids, src_len, s_prev, y_prev, sent_id, req = step_inputs(23)
    ctx, pctx, _ = oracle.encode(m, src_ids, src_len)
    for field, bad in (("y", -2), ("y", DIMS["V"]), ("r", DIMS["V"]), ("r", -1), ("s", 3)):
        y, r, s = y_prev.copy(), req.copy(), sent_id.copy()
        {"y": y, "r": r, "s": s}[field][2] = bad
        with pytest.raises(oracle.OracleError):
            oracle.score_batch(m, ctx, pctx, src_len, s_prev, y, s, r)


# ------------------------------------------------------- planted mistakes

PLANTS = {
    "reset": "test_gru_matches_torch_grucell",
    "zswap": "test_gru_matches_torch_grucell",
    "bwdorder": "test_encoder_matches_torch_grucell_scan",
    "nomask": "test_attention_invariants_and_closed_forms",
    "g2bias": "test_step_matches_torch_composition",
    "readout_s1": "test_step_matches_torch_composition",
    "lsedrop": "test_vocab_logsoftmax_brute_force_and_library",
    "wqt": "test_step_matches_torch_composition_square",
}


def test_step_matches_torch_composition_square():
    """Same as the composition pin with H == A, where a transposed query matrix still fits."""
    p, m = make_model(24, H=7, A=7)
    src_ids, src_len, s_prev, y_prev, sent_id, req = step_inputs(25, H=7)
    ctx, pctx, _ = oracle.encode(m, src_ids, src_len)
    got = oracle.score_batch(m, ctx, pctx, src_len, s_prev, y_prev, sent_id, req)
    want = torch_step(p, ctx, pctx, src_len, s_prev, y_prev, sent_id, req)
    for k in want:
        np.testing.assert_allclose(got[k], want[k], rtol=0, atol=1e-12, err_msg=k)


@pytest.mark.parametrize("plant", sorted(PLANTS))
def test_planted_mistakes_are_caught(plant):
    """Each planted oracle mistake makes its pin fail (run in a fresh process)."""
    oracle.build(plant, force=False)
    env = dict(os.environ, ORACLE_PLANT=plant)
    here = os.path.abspath(__file__)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        f"{here}::{PLANTS[plant]}"], env=env, capture_output=True, text=True,
                       cwd=os.path.dirname(os.path.dirname(here)))
    assert r.returncode != 0, f"planted mistake {plant!r} went unnoticed:\n{r.stdout[-2000:]}"
    assert "failed" in r.stdout
