"""Host-side forest builder of the ScoreBatch procedure (Section 5.1,
Figures 1 and 2), checked without a GPU: the paper's worked example and a
replay of random forests against their phrases."""
import json
import os

import numpy as np
import pytest

from paper_1605_04809_amd import binding as nb
from paper_1605_04809_amd.workloads import CONFIGS, make_forest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "figure1_forest.json")


def build(hyp_word, hyp_sent, pair_hyp, phrases):
    return nb.Forest(hyp_word, hyp_sent, pair_hyp, phrases)


def test_figure1_forest():
    g = json.load(open(GOLDEN))
    pairs = [(g["hypotheses"][h], words) for h, words in g["pairs"]]
    f = build([100, 101], [0, 0], [p[0] for p in pairs], [p[1] for p in pairs])
    sh = f.shape()
    assert sh["depth"] == g["steps"]
    assert [f.level(d)["req"].size for d in range(1, sh["depth"] + 1)] == g["edges_per_step"]
    assert sh["n_req"] == sum(g["edges_per_step"])
    lv1 = f.level(1)
    # E_1: the edge words of the first step; H_0: the hypothesis behind each edge
    assert lv1["req"].tolist() == g["E_1_words"]
    per_req_hyp = np.repeat(lv1["state_row"], np.diff(lv1["req_off"]))
    assert per_req_hyp.tolist() == g["H_0_hypotheses"]
    # one row per tree node with children: both roots, then 3, 3 and 1 nodes
    assert [f.level(d)["y_prev"].size for d in range(1, 5)] == [2, 3, 3, 1]
    assert lv1["y_prev"].tolist() == [100, 101]
    f.close()


def replay(f, hyp_word, hyp_sent, pair_hyp, phrases):
    """Every pair's path must walk its phrase through rows with the right inputs."""
    sh = f.shape()
    levels = [f.level(d) for d in range(1, sh["depth"] + 1)]
    row_base = np.cumsum([0] + [lv["y_prev"].size for lv in levels])
    req_base = np.cumsum([0] + [lv["req"].size for lv in levels])
    req_row = []  # global row of each global request
    for d, lv in enumerate(levels):
        req_row += (row_base[d] + np.repeat(np.arange(lv["y_prev"].size), np.diff(lv["req_off"]))).tolist()
    req_word = np.concatenate([lv["req"] for lv in levels]) if levels else np.zeros(0, np.int32)
    row_y = np.concatenate([lv["y_prev"] for lv in levels]) if levels else np.zeros(0, np.int32)
    row_state = np.concatenate([lv["state_row"] for lv in levels]) if levels else np.zeros(0, np.int32)
    row_sent = np.concatenate([lv["sent_id"] for lv in levels]) if levels else np.zeros(0, np.int32)
    paths = f.pair_paths()
    for p, (h, words) in enumerate(zip(pair_hyp, phrases)):
        assert np.all(paths[p, len(words):] == -1)
        prev_row = None
        for k, w in enumerate(words):
            j = paths[p, k]
            assert req_base[k] <= j < req_base[k + 1]      # the request sits in level k+1
            assert req_word[j] == w
            r = req_row[j]
            assert row_sent[r] == hyp_sent[h]
            if k == 0:
                assert row_y[r] == hyp_word[h] and row_state[r] == h
            else:
                assert row_y[r] == words[k - 1] and row_state[r] == prev_row
            prev_row = r
    return levels


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_forests_replay_and_count(seed):
    cfg = CONFIGS["tiny"].replace(V=7, S=3)
    fw = make_forest(cfg, n_hyp=25, seed=seed, max_phrases=6, max_len=5, branch=2)
    f = build(fw.hyp_word, fw.hyp_sent, fw.pair_hyp, fw.phrases)
    levels = replay(f, fw.hyp_word, fw.hyp_sent, fw.pair_hyp, fw.phrases)
    # requests at depth d = distinct phrase prefixes of length d per hypothesis
    for d, lv in enumerate(levels, start=1):
        prefixes = {(h, tuple(w[:d])) for h, w in zip(fw.pair_hyp, fw.phrases) if len(w) >= d}
        assert lv["req"].size == len(prefixes)
        extended = {(h, tuple(w[:d - 1])) for h, w in zip(fw.pair_hyp, fw.phrases) if len(w) >= d}
        assert lv["y_prev"].size == len(extended)
    assert f.shape()["depth"] == max(len(w) for w in fw.phrases)
    f.close()


def test_degenerate_forests():
    # no pairs, empty phrases, identical pairs, hypotheses without pairs
    f = build([1, 2, 3], [0, 0, 0], [], [])
    assert f.shape() == {"depth": 0, "n_rows": 0, "n_req": 0, "max_rows": 0}
    f.close()
    f = build([1, 2, 3], [0, 1, 0], [2, 2, 0], [[], [5, 6], [5, 6]])
    sh = f.shape()
    assert sh["depth"] == 2 and sh["n_req"] == 4 and sh["n_rows"] == 4
    paths = f.pair_paths()
    assert paths[0].tolist() == [-1, -1]
    replay(f, [1, 2, 3], [0, 1, 0], [2, 2, 0], [[], [5, 6], [5, 6]])
    f.close()
    f = build([1], [0], [0, 0], [[4, 4, 4], [4, 4, 4]])  # the same pair twice shares one path
    assert (f.pair_paths()[0] == f.pair_paths()[1]).all() and f.shape()["n_req"] == 3
    f.close()


def test_bad_pairs_are_rejected():
    with pytest.raises(nb.NmtError) as ei:
        build([1], [0], [1], [[3]])
    assert ei.value.status == nb.NMT_ERANGE


def test_phrases_flatten_for_the_rescorer():
    """The rescorer binding's flat form of a stack's phrases: phrase j is
    words[off[j]:off[j+1]], in order, empty phrases included."""
    off, words = nb.phrases_csr([[5, 6], [], (7,), np.array([8, 9, 10]), []])
    assert off.dtype == np.int32 and words.dtype == np.int32
    assert off.tolist() == [0, 2, 2, 3, 6, 6]
    assert words.tolist() == [5, 6, 7, 8, 9, 10]
    off, words = nb.phrases_csr([])
    assert off.tolist() == [0] and words.size == 0
    rng = np.random.default_rng(3)
    phrases = [rng.integers(0, 1000, size=rng.integers(0, 5)).tolist() for _ in range(200)]
    off, words = nb.phrases_csr(phrases)
    assert [words[off[j]:off[j + 1]].tolist() for j in range(len(phrases))] == phrases
