"""fp64 CPU oracle for the batched cGRU-attention decoder step.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It is a thin ctypes
wrapper around ``oracle.c`` (plain C, OpenMP over rows, fp64 arithmetic) and
shares no code with the HIP library; both sides consume the same seeded
inputs from ``paper_1605_04809_amd.workloads``.

Set ``ORACLE_PLANT=<name>`` before the first import to load a copy of the
oracle built with one deliberate mistake (see ``oracle.c``); the pin tests
use this to show that each pin catches the mistake it guards against.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")

PARAM_FIELDS = (
    "emb_src", "enc_f_W", "enc_f_b", "enc_f_U", "enc_b_W", "enc_b_b", "enc_b_U",
    "att_Wc", "att_b", "init_W", "init_b",
    "emb_tgt", "g1_W", "g1_b", "g1_U", "att_Wq", "att_v",
    "g2_U", "g2_b", "g2_Wc", "ro_Ws", "ro_Wy", "ro_Wc", "ro_b", "out_W", "out_b",
)

_F = ctypes.POINTER(ctypes.c_float)
_D = ctypes.POINTER(ctypes.c_double)
_I = ctypes.POINTER(ctypes.c_int32)


class Dims(ctypes.Structure):
    _fields_ = [("V_src", ctypes.c_int32), ("V", ctypes.c_int32), ("E", ctypes.c_int32),
                ("H", ctypes.c_int32), ("A", ctypes.c_int32)]


class Weights(ctypes.Structure):
    _fields_ = [(n, _F) for n in PARAM_FIELDS]


def lib_path(plant: Optional[str] = None) -> str:
    name = "liboracle.so" if not plant else f"liboracle_plant_{plant}.so"
    return os.path.join(_HERE, name)


def build(plant: Optional[str] = None, force: bool = True) -> str:
    """Compile oracle.c with gcc (-O2, no fast-math, OpenMP) into the package dir."""
    out = lib_path(plant)
    if not force and os.path.exists(out) and os.path.getmtime(out) >= os.path.getmtime(_SRC):
        return out
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall",
           "-Wno-unused-variable", _SRC, "-o", out + ".tmp", "-lm"]
    if plant:
        cmd.insert(1, f"-DORACLE_PLANT_{plant.upper()}=1")
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    plant = os.environ.get("ORACLE_PLANT") or None
    path = build(plant, force=False)
    lib = ctypes.CDLL(path)
    i32, p = ctypes.c_int32, ctypes.POINTER
    lib.oracle_gru.argtypes = [i32, i32, i32, _D, _D, _F, _F, _F, _F, _D]
    lib.oracle_encode.argtypes = [p(Dims), p(Weights), i32, i32, _I, _I, _D, _D, _D]
    lib.oracle_keys_from_annotations.argtypes = [p(Dims), p(Weights), i32, i32, _F, _I, _D, _D]
    score_args = [p(Dims), p(Weights), i32, i32, _D, _D, _I, i32, None, _I, _I, _I,
                  _D, _D, _D, _D, _D, _D, _D]
    a = list(score_args)
    a[8] = _F
    lib.oracle_score_batch.argtypes = a
    a = list(score_args)
    a[8] = _D
    lib.oracle_score_batch_f64state.argtypes = a
    lib.oracle_vocab_logsoftmax.argtypes = [i32, i32, i32, _D, _F, _F, _I, _D, _D, _D]
    lib.oracle_num_threads.argtypes = []
    for f in ("oracle_gru", "oracle_encode", "oracle_keys_from_annotations", "oracle_score_batch",
              "oracle_score_batch_f64state", "oracle_vocab_logsoftmax", "oracle_num_threads"):
        getattr(lib, f).restype = ctypes.c_int
    _lib = lib
    return lib


class OracleError(RuntimeError):
    pass


def _chk(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"{what} failed with status {rc}")


def _f32(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a, a.ctypes.data_as(_F)


def _f64(a):
    a = np.ascontiguousarray(a, dtype=np.float64)
    return a, a.ctypes.data_as(_D)


def _i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(_I)


def _out(shape):
    a = np.zeros(shape, dtype=np.float64)
    return a, a.ctypes.data_as(_D)


class Model:
    """Holds the fp32 parameter arrays (kept alive) and their C views."""

    def __init__(self, params: Dict[str, np.ndarray], V_src: int, V: int, E: int, H: int, A: int):
        self.dims = Dims(V_src, V, E, H, A)
        self._keep = {}
        w = Weights()
        for n in PARAM_FIELDS:
            arr, ptr = _f32(params[n])
            self._keep[n] = arr
            setattr(w, n, ptr)
        self.w = w
        self.V_src, self.V, self.E, self.H, self.A = V_src, V, E, H, A
        self.C = 2 * H

    @classmethod
    def from_workload(cls, wl) -> "Model":
        c = wl.cfg
        return cls(wl.params, c.V_src, c.V, c.E, c.H, c.A)


def num_threads() -> int:
    return _load().oracle_num_threads()


def gru(u: Optional[np.ndarray], h: np.ndarray, W, U, b_in=None, b_st=None) -> np.ndarray:
    """DL4MT GRU cell on rows: u [n x nin] (or None), h [n x H] -> [n x H] fp64."""
    lib = _load()
    h, hp = _f64(h)
    n, H = h.shape
    if u is None:
        nin, up, Wp = 0, None, None
    else:
        u, up = _f64(u)
        nin = u.shape[1]
        W, Wp = _f32(W)
    U, Up = _f32(U)
    bi, bip = _f32(b_in) if b_in is not None else (None, None)
    bs, bsp = _f32(b_st) if b_st is not None else (None, None)
    out, op = _out((n, H))
    _chk(lib.oracle_gru(n, nin, H, up, hp, Wp, Up, bip, bsp, op), "oracle_gru")
    return out


def encode(m: Model, src_ids: np.ndarray, src_len: np.ndarray):
    """-> (ctx [S,Tpad,2H], pctx [S,Tpad,A], s0 [S,H]) in fp64."""
    lib = _load()
    src_ids, ip = _i32(src_ids)
    src_len, lp = _i32(src_len)
    S, T = src_ids.shape
    ctx, cp = _out((S, T, m.C))
    pctx, pp = _out((S, T, m.A))
    s0, sp = _out((S, m.H))
    _chk(lib.oracle_encode(ctypes.byref(m.dims), ctypes.byref(m.w), S, T, ip, lp, cp, pp, sp),
         "oracle_encode")
    return ctx, pctx, s0


def keys_from_annotations(m: Model, ctx_f32: np.ndarray, src_len: np.ndarray):
    """Given fp32 annotations [S,Tpad,2H] -> (ctx fp64 masked, pctx fp64)."""
    lib = _load()
    ctx_f32, cfp = _f32(ctx_f32)
    src_len, lp = _i32(src_len)
    S, T, _ = ctx_f32.shape
    ctx, cp = _out((S, T, m.C))
    pctx, pp = _out((S, T, m.A))
    _chk(lib.oracle_keys_from_annotations(ctypes.byref(m.dims), ctypes.byref(m.w), S, T, cfp, lp,
                                          cp, pp), "oracle_keys_from_annotations")
    return ctx, pctx


def score_batch(m: Model, ctx: np.ndarray, pctx: np.ndarray, src_len: np.ndarray,
                s_prev: np.ndarray, y_prev: np.ndarray, sent_id: np.ndarray, req: np.ndarray,
                intermediates: bool = True) -> Dict[str, np.ndarray]:
    """One decoder step for B rows.  s_prev may be fp32 or fp64."""
    lib = _load()
    ctx, cp = _f64(ctx)
    pctx, pp = _f64(pctx)
    src_len, lp = _i32(src_len)
    y_prev, yp = _i32(y_prev)
    sent_id, sip = _i32(sent_id)
    req, rp = _i32(req)
    S, T, _ = ctx.shape
    B = y_prev.shape[0]
    out = {}
    logp, lpp = _out((B,))
    s_new, snp = _out((B, m.H))
    logZ, lzp = _out((B,))
    out.update(logp=logp, s_new=s_new, logZ=logZ)
    ptrs = [lpp, snp, lzp]
    if intermediates:
        alpha, ap = _out((B, T))
        c, ccp = _out((B, m.C))
        s1, s1p = _out((B, m.H))
        t, tp = _out((B, m.E))
        out.update(alpha=alpha, c=c, s1=s1, t=t)
        ptrs += [ap, ccp, s1p, tp]
    else:
        ptrs += [None] * 4
    if s_prev.dtype == np.float64:
        s_prev, spp = _f64(s_prev)
        fn = lib.oracle_score_batch_f64state
    else:
        s_prev, spp = _f32(s_prev)
        fn = lib.oracle_score_batch
    _chk(fn(ctypes.byref(m.dims), ctypes.byref(m.w), S, T, cp, pp, lp, B, spp, yp, sip, rp, *ptrs),
         "oracle_score_batch")
    return out


def vocab_logsoftmax(t: np.ndarray, out_W: np.ndarray, out_b: np.ndarray,
                     req: Optional[np.ndarray] = None, full: bool = False):
    """-> (logp [B] or None, logZ [B], logp_all [B,V] or None) for readouts t [B,E]."""
    lib = _load()
    t, tp = _f64(t)
    out_W, wp = _f32(out_W)
    out_b, bp = _f32(out_b)
    B, E = t.shape
    V = out_W.shape[1]
    logZ, lzp = _out((B,))
    logp, lpp = (_out((B,)) if req is not None else (None, None))
    rp = None
    if req is not None:
        req, rp = _i32(req)
    la, lap = (_out((B, V)) if full else (None, None))
    _chk(lib.oracle_vocab_logsoftmax(B, E, V, tp, wp, bp, rp, lpp, lzp, lap),
         "oracle_vocab_logsoftmax")
    return logp, logZ, la


# --------------------------------------------------------------- several models

def _nearest_bf16(x32: np.ndarray) -> np.ndarray:
    """fp32 values rounded to the nearest bf16 value, ties to even (kept as fp32)."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def average_params(params_list, coef=None, bf16: bool = False) -> Dict[str, np.ndarray]:
    """Section 6.3: a model whose parameters are the element-wise (weighted)
    average of K models' parameters.

    Each parameter is sum_k coef[k] * p_k in fp64, then stored the way the
    models store parameters: rounded to fp32, and for bf16 models further to
    the nearest bf16 value (ties to even).  ``coef`` defaults to 1/K taken as
    an fp32 number, the value the library uses.
    """
    K = len(params_list)
    if coef is None:
        coef = [float(np.float32(1.0 / K))] * K
    out = {}
    for name in PARAM_FIELDS:
        acc = np.zeros(np.shape(params_list[0][name]), dtype=np.float64)
        for k in range(K):
            acc += np.float64(coef[k]) * np.asarray(params_list[k][name], dtype=np.float64)
        a32 = acc.astype(np.float32)
        out[name] = _nearest_bf16(a32) if bf16 else a32
    return out


def log_linear(logp: np.ndarray, weights=None) -> np.ndarray:
    """Section 5: K models as separate features of the log-linear model; their
    share of a hypothesis score is sum_k weight_k * logp_k (fp64).  logp: [K, B]."""
    logp = np.asarray(logp, dtype=np.float64)
    w = np.ones(logp.shape[0]) if weights is None else np.asarray(weights, dtype=np.float64)
    return (w[:, None] * logp).sum(axis=0)


# ------------------------------------------------------------- stack rescoring

def rescore_stacks(m: Model, ctx, pctx, src_len, s0, stacks):
    """Section 5.3 (Figure 4) in plain form, one predecessor at a time.

    Hypotheses are numbered 0..S-1 (the empty hypothesis of each sentence:
    state s0, sentence start) and then in stack order.  For each stack, the
    set L of distinct predecessors (parent, phrase) is scored word by word:
    log p(phrase | parent) = sum_t log p(w_t | parent, w_<t), each word one
    decoder step from the state and last word reached so far (no prefix
    sharing, no batching beyond rows being independent).  Each hypothesis
    gets its predecessor's score; its state is the one reached after the
    phrase's last word (the parent's for an empty phrase), kept in fp64.

    Returns (per-stack lists of fp64 scores, fp64 states [n_hyp, H]).
    """
    S = s0.shape[0]
    states = [np.asarray(s0[s], np.float64) for s in range(S)]
    last = [-1] * S
    sent = list(range(S))
    scores = []
    for parents, phrases in stacks:
        index = {}
        for p, ph in zip(parents, phrases):
            index.setdefault((int(p), tuple(int(w) for w in ph)), len(index))
        pairs = list(index.keys())
        cur = np.stack([states[p] for p, _ in pairs]) if pairs else np.zeros((0, m.H))
        word = np.array([last[p] for p, _ in pairs], np.int32)
        sid = np.array([sent[p] for p, _ in pairs], np.int32)
        logp = np.zeros(len(pairs))
        for t in range(max((len(ph) for _, ph in pairs), default=0)):
            live = np.array([i for i, (_, ph) in enumerate(pairs) if len(ph) > t], np.int64)
            req = np.array([pairs[i][1][t] for i in live], np.int32)
            r = score_batch(m, ctx, pctx, src_len, cur[live], word[live], sid[live], req, intermediates=False)
            logp[live] += r["logp"]
            cur[live] = r["s_new"]
            word[live] = req
        out = np.empty(len(parents))
        for j, (p, ph) in enumerate(zip(parents, phrases)):
            i = index[(int(p), tuple(int(w) for w in ph))]
            out[j] = logp[i]
            states.append(cur[i].copy())
            last.append(int(ph[-1]) if len(ph) else last[int(p)])
            sent.append(sent[int(p)])
        scores.append(out)
    return scores, np.stack(states)
