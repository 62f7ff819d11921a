"""Pins of the oracle's stack rescoring (Section 5.3, Figure 4) and of the
synthetic stack generator, on the CPU.

The rescoring oracle splits each hypothesis' target sequence at stack
boundaries; by the chain rule of the decoder's factorisation the scores
along a hypothesis' ancestry must add up to the log-probability of its whole
target sequence scored word by word from the sentence start, and its state
must be the state reached there.  That pins the bookkeeping (parents, last
words, states, the predecessor set) independently of how stacks cut the
sequence."""
import numpy as np
import pytest

import oracle
from paper_1605_04809_amd.workloads import CONFIGS, make_workload, make_stacks


@pytest.fixture(scope="module")
def tiny():
    cfg = CONFIGS["tiny"].replace(S=2, len_lo=6, len_hi=9, Tpad=9)
    wl = make_workload(cfg)
    m = oracle.Model.from_workload(wl)
    ctx, pctx, s0 = oracle.encode(m, wl.src_ids, wl.src_len)
    return cfg, wl, m, ctx, pctx, s0


def _ancestry(sw, stacks):
    """parent and phrase of every hypothesis id (roots: None)."""
    par, phr = {}, {}
    nid = sw.n_roots
    for parents, phrases in stacks:
        for p, ph in zip(parents, phrases):
            par[nid], phr[nid] = int(p), list(ph)
            nid += 1
    return par, phr


def test_generator_shape(tiny):
    cfg = tiny[0]
    sw = make_stacks(cfg, src_len=6, stack_size=40, seed=3, sent=1)
    assert len(sw.stacks) == 6 and sw.n_roots == cfg.S
    first = sw.n_roots
    for c, (parents, phrases) in enumerate(sw.stacks, start=1):
        assert 0 < len(parents) <= 40 and len(parents) == len(phrases)
        assert np.all(parents < first) and all(1 <= len(p) <= 4 for p in phrases)
        first += len(parents)
    assert np.all(sw.stacks[0][0] == 1)  # the first stack extends sentence 1's empty hypothesis


def test_chain_rule_over_stacks(tiny):
    cfg, wl, m, ctx, pctx, s0 = tiny
    sw = make_stacks(cfg, src_len=5, stack_size=12, seed=4, sent=1)
    scores, states = oracle.rescore_stacks(m, ctx, pctx, wl.src_len, s0, sw.stacks)
    par, phr = _ancestry(sw, sw.stacks)
    score_of = {}
    nid = sw.n_roots
    for sc in scores:
        for x in sc:
            score_of[nid] = x
            nid += 1
    last = list(range(sw.n_roots + sum(len(s[0]) for s in sw.stacks) - 8, nid))  # last few hypotheses
    for h in last:
        seq, total, k = [], 0.0, h
        while k >= sw.n_roots:
            seq = phr[k] + seq
            total += score_of[k]
            k = par[k]
        # the whole sequence, one word per step from the sentence start
        st, y, lp = s0[k:k + 1].astype(np.float64), -1, 0.0
        for w in seq:
            r = oracle.score_batch(m, ctx, pctx, wl.src_len, st, np.array([y], np.int32), np.array([k], np.int32),
                                   np.array([w], np.int32), intermediates=False)
            lp += r["logp"][0]
            st, y = r["s_new"], w
        assert abs(lp - total) < 1e-12 * max(1.0, abs(lp)), (h, lp, total)
        np.testing.assert_allclose(states[h], st[0], rtol=0, atol=1e-14)


def test_duplicates_and_empty_phrases(tiny):
    cfg, wl, m, ctx, pctx, s0 = tiny
    stacks = [(np.array([0, 0, 1, 0], np.int32), [[5, 6], [5, 6], [7], []]),
              (np.array([2, 3, 5, 5], np.int32), [[8], [8], [], [9, 10, 11]])]
    scores, states = oracle.rescore_stacks(m, ctx, pctx, wl.src_len, s0, stacks)
    assert scores[0][0] == scores[0][1]
    np.testing.assert_array_equal(states[2], states[3])
    assert scores[0][3] == 0.0 and scores[1][2] == 0.0
    np.testing.assert_array_equal(states[5], s0[0])        # empty phrase keeps the parent's (root 0) state
    np.testing.assert_array_equal(states[8], states[5])    # and again one stack later
    assert np.all(scores[0][:3] < 0) and scores[1][3] < 0
