"""Stack rescoring on the GPU (Section 5.3, Figure 4) through the C-ABI
(nmt_rescorer_*), against the plain fp64 oracle of the same procedure on
the same synthetic stacks.

Scores are phrase log-probabilities, sums of up to four word scores, so the
bar is four times the per-word bar: 4e-4 with fp32 weights, 8e-2 with bf16
weights.  Hypothesis states are carried from stack to stack in fp32 on the
GPU and in fp64 in the oracle; after the last stack they must still agree
within 1e-4 (fp32) and 1e-2 (bf16).
"""
import numpy as np
import pytest

import oracle
from paper_1605_04809_amd.workloads import CONFIGS, make_workload, make_stacks

pytestmark = pytest.mark.gpu


def _torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.fixture(scope="module")
def env():
    torch = _torch()
    from paper_1605_04809_amd import binding as nb
    from tests import gpu_cases
    return torch, nb, gpu_cases


def _members(cfgs):
    """Workloads of K models sharing the source sentences of the first."""
    wls = [make_workload(c) for c in cfgs]
    for w in wls[1:]:
        w.src_ids, w.src_len = wls[0].src_ids, wls[0].src_len
    return wls


def _rescore_both(env, wls, sw, capacity=None):
    torch, nb, gc = env
    runs = [gc.GpuRun(w) for w in wls]
    n_total = sw.n_roots + sum(len(p) for p, _ in sw.stacks)
    r = nb.Rescorer([g.model for g in runs], [g.src for g in runs], [g.s0 for g in runs],
                    capacity or n_total)
    gpu_scores, info = [], []
    for parents, phrases in sw.stacks:
        lp, ids = r.rescore(parents, phrases)
        gpu_scores.append(lp)
        info.append(r.info())
    gpu_states = [r.states(k, wls[k].cfg.H) for k in range(len(wls))]
    orc = []
    for w in wls:
        m = oracle.Model.from_workload(w)
        ctx, pctx, s0 = oracle.encode(m, w.src_ids, w.src_len)
        orc.append(oracle.rescore_stacks(m, ctx, pctx, w.src_len, s0, sw.stacks))
    r.close()
    for g in runs:
        g.close()
    return gpu_scores, gpu_states, orc, info


def _check(gpu_scores, gpu_states, orc, tol_score, tol_state):
    from tests.gpu_cases import max_abs
    for k, (o_scores, o_states) in enumerate(orc):
        e_sc = max(max_abs(g[k], o) for g, o in zip(gpu_scores, o_scores))
        e_st = max_abs(gpu_states[k], o_states)
        print(f"model {k}: max |gpu - oracle| score {e_sc:.2e} state {e_st:.2e}", flush=True)
        assert e_sc <= tol_score and e_st <= tol_state, (k, e_sc, e_st)


@pytest.mark.parametrize("wtype,tol_score,tol_state", [("f32", 4e-4, 1e-4), ("bf16", 8e-2, 1e-2)])
def test_rescorer_matches_oracle(env, wtype, tol_score, tol_state):
    cfg = CONFIGS["tiny"].replace(S=3, len_lo=5, len_hi=10, Tpad=10, wtype=wtype, seed=61)
    wls = _members([cfg])
    sw = make_stacks(cfg, src_len=6, stack_size=60, seed=5, sent=2)
    gpu_scores, gpu_states, orc, info = _rescore_both(env, wls, sw)
    _check(gpu_scores, gpu_states, orc, tol_score, tol_state)
    # predecessors are deduplicated: a stack's forest holds each distinct pair once
    for (parents, phrases), inf in zip(sw.stacks, info):
        assert inf["last_pairs"] == len({(int(p), tuple(ph)) for p, ph in zip(parents, phrases)})


def test_rescorer_with_two_models_of_different_widths(env):
    base = CONFIGS["tiny"].replace(S=2, len_lo=4, len_hi=8, Tpad=8)
    wls = _members([base.replace(seed=71), base.replace(seed=72, E=16, H=32, A=48)])
    sw = make_stacks(base, src_len=5, stack_size=40, seed=6, sent=0)
    gpu_scores, gpu_states, orc, _ = _rescore_both(env, wls, sw)
    _check(gpu_scores, gpu_states, orc, 4e-4, 1e-4)


def test_rescorer_at_paper_dimensions(env):
    cfg = CONFIGS["enru_b2000"].replace(S=2, len_lo=12, len_hi=20, Tpad=20)
    wls = _members([cfg])
    sw = make_stacks(cfg, src_len=3, stack_size=12, seed=7, sent=1)
    gpu_scores, gpu_states, orc, _ = _rescore_both(env, wls, sw)
    _check(gpu_scores, gpu_states, orc, 4e-4, 1e-4)


def test_rescorer_duplicates_empty_phrases_and_errors(env):
    torch, nb, gc = env
    cfg = CONFIGS["tiny"].replace(S=2, len_lo=5, len_hi=5, Tpad=5, seed=91)
    w = make_workload(cfg)
    g = gc.GpuRun(w)
    r = nb.Rescorer([g.model], [g.src], [g.s0], capacity=12)
    lp, ids = r.rescore([0, 0, 1, 0], [[5, 6], [5, 6], [7], []])
    assert list(ids) == [2, 3, 4, 5]
    assert lp[0, 0] == lp[0, 1] and lp[0, 3] == 0.0 and np.all(lp[0, :3] < 0)
    st = r.states(0, cfg.H)
    np.testing.assert_array_equal(st[2], st[3])
    np.testing.assert_array_equal(st[5], g.s0[0].cpu().numpy())
    assert r.info()["last_pairs"] == 3
    with pytest.raises(nb.NmtError, match="ERANGE"):   # parent that does not exist yet
        r.rescore([6], [[1]])
    with pytest.raises(nb.NmtError, match="ERANGE"):   # word outside the vocabulary
        r.rescore([2], [[cfg.V]])
    with pytest.raises(nb.NmtError, match="ERANGE"):   # 6 + 7 > capacity 12
        r.rescore([2] * 7, [[1]] * 7)
    assert r.info()["n_hyp"] == 6                     # failed calls add nothing
    lp2, ids2 = r.rescore([5, 2], [[3], [4, 4]])
    assert list(ids2) == [6, 7] and np.all(lp2 < 0)
    r.close()
    g.close()
