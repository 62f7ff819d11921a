"""Seeded synthetic workloads for the batched cGRU-attention scoring step.

This module only draws inputs: model parameters, source sentences and the
batch of hypothesis rows to score.  It holds none of the method's arithmetic,
so both the fp64 oracle and the HIP path consume exactly the same arrays.

Shapes follow the paper's systems (Section 2: BPE vocabularies of 50,000
English and 100,000 Russian units; Section 3: embeddings of 500, hidden
layers of 1024, training sentences of at most 50 tokens; Section 6: stacks of
1,000 and pop limits of 2,000-5,000, which set hypothesis batches in the
thousands, and development sentences shorter than 40 words).  No trained
model or WMT data is used: weights are N(0, sigma) with sigma the standard
deviation, drawn with ``numpy.random.default_rng(seed)`` in the fixed order
below.

Draw order (one generator per workload):
  1. parameters, in ``PARAM_ORDER``;
  2. source lengths, then source ids (all ``Tpad`` positions are drawn, so
     padding holds random ids that the method must ignore);
  3. ``sent_id``, ``s_prev`` (tanh of a standard normal), ``y_prev``;
  4. ``req`` -- or, for the phrase workload, phrase lengths then phrase
     tokens (the first token of each phrase is the first request).
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Dict, Optional

import numpy as np

# Parameter names, shapes (as functions of the dims) and the draw order.
# Matrices use the x.W convention: [input dim x output dim], row-major.
# The 3H-wide GRU blocks hold the gates in the column order [r | z | n].
PARAM_ORDER = (
    "emb_src", "enc_f_W", "enc_f_b", "enc_f_U", "enc_b_W", "enc_b_b", "enc_b_U",
    "att_Wc", "att_b", "init_W", "init_b",
    "emb_tgt", "g1_W", "g1_b", "g1_U", "att_Wq", "att_v",
    "g2_U", "g2_b", "g2_Wc", "ro_Ws", "ro_Wy", "ro_Wc", "ro_b", "out_W", "out_b",
)

EMBEDDINGS = ("emb_src", "emb_tgt")


def param_shapes(V_src: int, V: int, E: int, H: int, A: int) -> Dict[str, tuple]:
    C = 2 * H
    return {
        "emb_src": (V_src, E),
        "enc_f_W": (E, 3 * H), "enc_f_b": (3 * H,), "enc_f_U": (H, 3 * H),
        "enc_b_W": (E, 3 * H), "enc_b_b": (3 * H,), "enc_b_U": (H, 3 * H),
        "att_Wc": (C, A), "att_b": (A,),
        "init_W": (C, H), "init_b": (H,),
        "emb_tgt": (V, E),
        "g1_W": (E, 3 * H), "g1_b": (3 * H,), "g1_U": (H, 3 * H),
        "att_Wq": (H, A), "att_v": (A,),
        "g2_U": (H, 3 * H), "g2_b": (3 * H,), "g2_Wc": (C, 3 * H),
        "ro_Ws": (H, E), "ro_Wy": (E, E), "ro_Wc": (C, E), "ro_b": (E,),
        "out_W": (E, V), "out_b": (V,),
    }


@dataclass(frozen=True)
class Config:
    """One synthetic workload: model dims, weight recipe and the row batch."""
    name: str
    V: int
    V_src: int
    E: int
    H: int
    A: int
    B: int                 # rows scored per step (hypotheses for the phrase workload)
    S: int                 # source sentences
    len_lo: int            # source length drawn uniform in [len_lo, len_hi]
    len_hi: int
    Tpad: int              # padded source length
    sigma_w: float
    sigma_emb: float
    seed: int
    wtype: str = "f32"     # "f32" or "bf16" storage of weights and embeddings
    phrase_max: int = 0    # >0: phrase workload, each row extended by 1..phrase_max tokens

    @property
    def C(self) -> int:
        return 2 * self.H

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# The five workloads.  "tiny" is the small case the oracle finishes at once;
# "enru_b2000" is the headline shape (en->ru, 100k target vocabulary).
CONFIGS = {
    "tiny": Config("tiny", V=1000, V_src=1000, E=32, H=64, A=64, B=8, S=1,
                   len_lo=10, len_hi=10, Tpad=10, sigma_w=0.05, sigma_emb=0.1, seed=0),
    "ruen_b1000": Config("ruen_b1000", V=50000, V_src=100000, E=500, H=1024, A=1024,
                         B=1000, S=1, len_lo=30, len_hi=30, Tpad=30,
                         sigma_w=0.01, sigma_emb=0.01, seed=1),
    "enru_b2000": Config("enru_b2000", V=100000, V_src=50000, E=500, H=1024, A=1024,
                         B=2000, S=20, len_lo=10, len_hi=50, Tpad=50,
                         sigma_w=0.01, sigma_emb=0.01, seed=2),
    "phrase_h500": Config("phrase_h500", V=100000, V_src=50000, E=500, H=1024, A=1024,
                          B=500, S=10, len_lo=5, len_hi=80, Tpad=80,
                          sigma_w=0.01, sigma_emb=0.01, seed=3, phrase_max=4),
    "bf16_b4096": Config("bf16_b4096", V=100000, V_src=50000, E=500, H=1024, A=1024,
                         B=4096, S=32, len_lo=20, len_hi=80, Tpad=80,
                         sigma_w=0.01, sigma_emb=0.01, seed=4, wtype="bf16"),
}
CONFIG_ORDER = ("tiny", "ruen_b1000", "enru_b2000", "phrase_h500", "bf16_b4096")


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even), kept as fp32.

    Both sides of a bf16 comparison consume these identical values; the
    oracle widens them exactly.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


@dataclass
class Workload:
    cfg: Config
    params: Dict[str, np.ndarray]
    src_len: np.ndarray          # [S] int32
    src_ids: np.ndarray          # [S, Tpad] int32
    sent_id: np.ndarray          # [B] int32
    s_prev: np.ndarray           # [B, H] float32
    y_prev: np.ndarray           # [B] int32, -1 = sentence start
    req: np.ndarray              # [B] int32 (phrase workload: first phrase token)
    phrase_len: Optional[np.ndarray] = None    # [B] int32
    phrase_tok: Optional[np.ndarray] = None    # [B, phrase_max] int32, -1 past the end
    extra: dict = field(default_factory=dict)


def draw_params(cfg: Config, rng: np.random.Generator) -> Dict[str, np.ndarray]:
    shapes = param_shapes(cfg.V_src, cfg.V, cfg.E, cfg.H, cfg.A)
    out = {}
    for name in PARAM_ORDER:
        sigma = cfg.sigma_emb if name in EMBEDDINGS else cfg.sigma_w
        a = rng.standard_normal(shapes[name], dtype=np.float32)
        a *= np.float32(sigma)
        if cfg.wtype == "bf16":
            a = round_to_bf16(a)
        out[name] = a
    return out


def make_workload(cfg: Config, B: Optional[int] = None) -> Workload:
    """Draw the whole workload for ``cfg`` (``B`` overrides the row count)."""
    rng = np.random.default_rng(cfg.seed)
    params = draw_params(cfg, rng)
    B = cfg.B if B is None else B
    S, T = cfg.S, cfg.Tpad
    src_len = rng.integers(cfg.len_lo, cfg.len_hi + 1, size=S, dtype=np.int64).astype(np.int32)
    src_ids = rng.integers(0, cfg.V_src, size=(S, T), dtype=np.int64).astype(np.int32)
    sent_id = rng.integers(0, S, size=B, dtype=np.int64).astype(np.int32)
    s_prev = np.tanh(rng.standard_normal((B, cfg.H), dtype=np.float32)).astype(np.float32)
    y_prev = rng.integers(0, cfg.V, size=B, dtype=np.int64).astype(np.int32)
    wl = Workload(cfg, params, src_len, src_ids, sent_id, s_prev, y_prev,
                  req=np.zeros(B, np.int32))
    if cfg.phrase_max > 0:
        plen = rng.integers(1, cfg.phrase_max + 1, size=B, dtype=np.int64).astype(np.int32)
        tok = rng.integers(0, cfg.V, size=(B, cfg.phrase_max), dtype=np.int64).astype(np.int32)
        tok[np.arange(cfg.phrase_max)[None, :] >= plen[:, None]] = -1
        wl.phrase_len, wl.phrase_tok = plen, tok
        wl.req = tok[:, 0].copy()
    else:
        wl.req = rng.integers(0, cfg.V, size=B, dtype=np.int64).astype(np.int32)
    return wl


def phrase_schedule(phrase_len: np.ndarray):
    """Row order and per-step row counts for stepwise phrase scoring.

    Rows are sorted by phrase length, longest first, so step j (1-based)
    scores the prefix of rows whose phrase has at least j tokens.  Returns
    ``(order, counts)``; ``counts[j-1]`` is the number of rows at step j.
    """
    order = np.argsort(-phrase_len.astype(np.int64), kind="stable").astype(np.int32)
    kmax = int(phrase_len.max()) if phrase_len.size else 0
    counts = [int((phrase_len >= j).sum()) for j in range(1, kmax + 1)]
    return order, counts


def high_signal(cfg: Config, seed: int = 100) -> Config:
    """A variant of ``cfg`` with large weights so every term moves log p."""
    return cfg.replace(sigma_w=0.5, sigma_emb=0.5, seed=seed)


def unit_gain(cfg: Config, v_spread: float = 1.5, key_scale: float = 1.0, query_scale: float = 1.0) -> Workload:
    """The workload of ``cfg`` with every layer passing signal at unit scale,
    so that a mistake anywhere in the step moves its outputs (at sigma = 0.01
    attention is nearly uniform and hides attention bugs).

    Weight matrices are N(0, 1/fan-in) (fan-in: rows of the x.W matrix),
    embeddings N(0, 1), biases N(0, 0.1^2).  For N(0, 1) annotations the keys
    are then about N(0, key_scale^2) and the queries about query_scale times
    the first GRU's state scale (|s1| < 1); the attention vector is scaled so
    that a row's scores vary by about ``v_spread`` over source positions
    (tanh(k + q) varies by about 0.3 in variance per term).  bf16 workloads
    are rounded to bf16 again after scaling.
    """
    wl = make_workload(cfg.replace(sigma_w=1.0, sigma_emb=1.0))
    p = wl.params
    for name, a in p.items():
        if name in EMBEDDINGS:
            continue
        a *= np.float32(1.0 / np.sqrt(a.shape[0]) if a.ndim == 2 else 0.1)
    p["att_Wc"] *= np.float32(key_scale)
    p["att_b"] *= np.float32(key_scale)
    p["att_Wq"] *= np.float32(query_scale)
    p["att_v"] *= np.float32(10.0 * v_spread / np.sqrt(0.3 * cfg.A))
    if cfg.wtype == "bf16":
        for name in p:
            p[name] = round_to_bf16(p[name])
    return wl


def random_annotations(cfg: Config, seed: int, scale: float = 1.0) -> np.ndarray:
    """Source annotations [S, Tpad, 2H] drawn N(0, scale) for injected-context tests."""
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((cfg.S, cfg.Tpad, cfg.C), dtype=np.float32) * np.float32(scale))


@dataclass
class ForestWorkload:
    """(hypothesis, target phrase) pairs whose phrases share prefixes per hypothesis."""
    hyp_word: np.ndarray     # [n_hyp] int32, -1 = sentence start
    hyp_sent: np.ndarray     # [n_hyp] int32
    hyp_state: np.ndarray    # [n_hyp, H] float32
    pair_hyp: np.ndarray     # [n_pairs] int32
    phrases: list            # n_pairs lists of word ids


def make_forest(cfg: Config, n_hyp: int, seed: int, max_phrases: int = 6, max_len: int = 4,
                branch: int = 3) -> ForestWorkload:
    """Synthetic expansions in the shape of a phrase-based stack: each hypothesis
    gets 1..max_phrases target phrases of 1..max_len words, drawn position by
    position from `branch` candidate words per position, so phrases of one
    hypothesis share prefixes as phrase-table options do."""
    rng = np.random.default_rng(seed)
    hyp_word = rng.integers(-1, cfg.V, size=n_hyp, dtype=np.int64).astype(np.int32)
    hyp_sent = rng.integers(0, cfg.S, size=n_hyp, dtype=np.int64).astype(np.int32)
    hyp_state = np.tanh(rng.standard_normal((n_hyp, cfg.H), dtype=np.float32)).astype(np.float32)
    pair_hyp, phrases = [], []
    for h in range(n_hyp):
        cand = rng.integers(0, cfg.V, size=(max_len, branch), dtype=np.int64)
        for _ in range(int(rng.integers(1, max_phrases + 1))):
            n = int(rng.integers(1, max_len + 1))
            pick = rng.integers(0, branch, size=n)
            phrases.append([int(cand[i, pick[i]]) for i in range(n)])
            pair_hyp.append(h)
    return ForestWorkload(hyp_word, hyp_sent, hyp_state, np.asarray(pair_hyp, np.int32), phrases)


@dataclass
class StackWorkload:
    """Synthetic stacks of a phrase-based search over one source sentence.

    Hypotheses are numbered in creation order: 0..n_roots-1 are the empty
    hypotheses of the n_roots source sentences; stack c (c = 1..src_len
    covered words) numbers its hypotheses next.  stacks[c-1] = (parents
    [n_c] int32, phrases: n_c lists of target word ids)."""
    n_roots: int
    sent: int
    stacks: list


def make_stacks(cfg: Config, src_len: int, stack_size: int, seed: int, sent: int = 0, max_src_phrase: int = 3,
                max_len: int = 4, options: int = 6, branch: int = 3, dup_rate: float = 0.05) -> StackWorkload:
    """Stacks shaped like a phrase-based decoder's: every source span of up
    to max_src_phrase words has `options` target phrases of 1..max_len words,
    drawn position by position from `branch` candidate words (so options
    share prefixes as phrase-table entries do); a hypothesis in stack c
    extends a hypothesis of stack c-m by an option of a length-m span.  Stack
    sizes grow with the number of expansions until the stack limit; a
    fraction dup_rate of each stack repeats an earlier (parent, phrase) pair
    of the same stack, as different coverages with the same target do."""
    rng = np.random.default_rng(seed)
    table = {}
    for i in range(src_len):
        for m in range(1, max_src_phrase + 1):
            if i + m > src_len:
                break
            cand = rng.integers(0, cfg.V, size=(max_len, branch), dtype=np.int64)
            opts = []
            for _ in range(options):
                n = int(rng.integers(1, max_len + 1))
                pick = rng.integers(0, branch, size=n)
                opts.append([int(cand[t, pick[t]]) for t in range(n)])
            table[(i, m)] = opts
    ids = [[sent]]            # hypothesis ids per stack; stack 0 is the empty hypothesis
    next_id = cfg.S
    stacks = []
    for c in range(1, src_len + 1):
        ms = [m for m in range(1, min(max_src_phrase, c) + 1)]
        w = np.array([len(ids[c - m]) for m in ms], np.float64)
        n_c = int(min(stack_size, 4 * options * w.sum()))
        parents, phrases = [], []
        for j in range(n_c):
            if j > 0 and rng.random() < dup_rate:
                k = int(rng.integers(0, j))
                parents.append(parents[k])
                phrases.append(list(phrases[k]))
                continue
            m = ms[int(rng.choice(len(ms), p=w / w.sum()))]
            par = ids[c - m][int(rng.integers(0, len(ids[c - m])))]
            start = int(rng.integers(0, src_len - m + 1))
            opt = table[(start, m)][int(rng.integers(0, options))]
            parents.append(par)
            phrases.append(list(opt))
        stacks.append((np.asarray(parents, np.int32), phrases))
        ids.append(list(range(next_id, next_id + n_c)))
        next_id += n_c
    return StackWorkload(cfg.S, sent, stacks)
