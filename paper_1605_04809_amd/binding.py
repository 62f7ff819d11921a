"""ctypes binding of libnmt (include/nmt.h) with the same call names.

Argument marshalling only: every arithmetic step runs in the HIP kernels of
libnmt.so.  torch tensors provide device memory (``data_ptr()``) and the
stream (``torch.cuda.current_stream()``).  There is no CPU fallback: if the
library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import itertools
import os
from typing import Dict, Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# NMT_LIBRARY may point at another build of the same library (tuning sweeps).
LIB_PATH = os.environ.get("NMT_LIBRARY") or os.path.join(HERE, "libnmt.so")

NMT_OK, NMT_EINVAL, NMT_ENOMEM, NMT_EDEVICE, NMT_ERANGE, NMT_EWORKSPACE = 0, -1, -2, -3, -4, -5
NMT_F32, NMT_BF16 = 0, 1
STATUS_NAMES = {0: "NMT_OK", -1: "NMT_EINVAL", -2: "NMT_ENOMEM", -3: "NMT_EDEVICE", -4: "NMT_ERANGE",
                -5: "NMT_EWORKSPACE"}

WEIGHT_FIELDS = (
    "emb_src", "enc_f_W", "enc_f_b", "enc_f_U", "enc_b_W", "enc_b_b", "enc_b_U",
    "att_Wc", "att_b", "init_W", "init_b",
    "emb_tgt", "g1_W", "g1_b", "g1_U", "att_Wq", "att_v",
    "g2_U", "g2_b", "g2_Wc", "ro_Ws", "ro_Wy", "ro_Wc", "ro_b", "out_W", "out_b",
)

# Every function the header declares (checked against include/nmt.h by the tests).
EXPORTS = ("nmt_model_create", "nmt_model_destroy", "nmt_encode", "nmt_source_from_annotations",
           "nmt_source_info", "nmt_source_destroy", "nmt_score_workspace_bytes", "nmt_score_batch",
           "nmt_score_batch_debug", "nmt_score_batch_noalloc", "nmt_stream_status", "nmt_last_error", "nmt_profile_begin",
           "nmt_profile_end", "nmt_score_forest_step", "nmt_forest_build", "nmt_forest_shape",
           "nmt_forest_level", "nmt_forest_pair_paths", "nmt_forest_workspace_bytes", "nmt_score_forest",
           "nmt_forest_destroy", "nmt_model_average", "nmt_ensemble_workspace_bytes", "nmt_score_ensemble",
           "nmt_rescorer_create", "nmt_rescore_stack", "nmt_rescorer_info", "nmt_rescorer_destroy",
           "nmt_debug_alloc_hook", "nmt_debug_gemm_form", "nmt_debug_gemm_streamed", "nmt_debug_precompute")

PHASES = ("gru1", "query", "attention", "gru2", "readout", "vocab", "combine")

_VP = ctypes.c_void_p
_I32 = ctypes.c_int32


class Dims(ctypes.Structure):
    _fields_ = [("V_src", _I32), ("V", _I32), ("E", _I32), ("H", _I32), ("A", _I32), ("wtype", _I32)]


class Weights(ctypes.Structure):
    _fields_ = [(n, ctypes.POINTER(ctypes.c_float)) for n in WEIGHT_FIELDS]


class Timing(ctypes.Structure):
    _fields_ = [("steps", _I32), ("ms", ctypes.c_double * len(PHASES))]


class NmtError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libnmt.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_1605_04809_amd.build`")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    lib.nmt_model_create.argtypes = [P(Dims), P(Weights), P(_VP)]
    lib.nmt_model_destroy.argtypes = [_VP]
    lib.nmt_model_destroy.restype = None
    lib.nmt_encode.argtypes = [_VP, _I32, _I32, _VP, P(_I32), _VP, _VP, P(_VP)]
    lib.nmt_source_from_annotations.argtypes = [_VP, _I32, _I32, _VP, P(_I32), _VP, P(_VP)]
    lib.nmt_source_info.argtypes = [_VP, P(_I32), P(_I32), P(_VP), P(_VP)]
    lib.nmt_source_destroy.argtypes = [_VP]
    lib.nmt_source_destroy.restype = None
    lib.nmt_score_workspace_bytes.argtypes = [_VP, _I32]
    lib.nmt_score_workspace_bytes.restype = ctypes.c_size_t
    score = [_VP, _VP, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP]
    lib.nmt_score_batch.argtypes = score
    lib.nmt_score_batch_debug.argtypes = score + [_VP, _VP, _VP, _VP]
    lib.nmt_score_batch_noalloc.argtypes = [_VP, _VP, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP]
    lib.nmt_stream_status.argtypes = [_VP, _VP]
    lib.nmt_profile_begin.argtypes = [_VP, _I32]
    lib.nmt_profile_end.argtypes = [_VP, _VP, P(Timing)]
    lib.nmt_score_forest_step.argtypes = [_VP, _VP, _I32, _VP, _I32, _VP, _VP, _VP, _VP, _VP, _I32, _VP, _VP, _VP,
                                          _VP, ctypes.c_size_t, _VP]
    IP = P(_I32)
    lib.nmt_forest_build.argtypes = [_I32, IP, IP, _I32, IP, IP, IP, P(_VP)]
    lib.nmt_forest_shape.argtypes = [_VP, IP, IP, IP, IP]
    lib.nmt_forest_level.argtypes = [_VP, _I32, IP, IP, IP, IP, IP, IP, IP]
    lib.nmt_forest_pair_paths.argtypes = [_VP, IP]
    lib.nmt_forest_workspace_bytes.argtypes = [_VP, _VP]
    lib.nmt_forest_workspace_bytes.restype = ctypes.c_size_t
    lib.nmt_score_forest.argtypes = [_VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP]
    lib.nmt_forest_destroy.argtypes = [_VP]
    lib.nmt_forest_destroy.restype = None
    lib.nmt_model_average.argtypes = [_I32, P(_VP), P(ctypes.c_float), _VP, P(_VP)]
    lib.nmt_ensemble_workspace_bytes.argtypes = [_I32, P(_VP), _I32]
    lib.nmt_ensemble_workspace_bytes.restype = ctypes.c_size_t
    lib.nmt_score_ensemble.argtypes = [_I32, P(_VP), P(_VP), _I32, P(_VP), _VP, _VP, _VP, _VP, P(_VP), _VP,
                                       P(ctypes.c_float), _VP, _VP, ctypes.c_size_t, _VP]
    lib.nmt_rescorer_create.argtypes = [_I32, P(_VP), P(_VP), P(_VP), _I32, _VP, P(_VP)]
    lib.nmt_rescore_stack.argtypes = [_VP, _I32, IP, IP, IP, P(ctypes.c_float), IP, _VP]
    lib.nmt_rescorer_info.argtypes = [_VP, _I32, P(_VP), IP, IP, IP, IP, IP]
    lib.nmt_rescorer_destroy.argtypes = [_VP]
    lib.nmt_rescorer_destroy.restype = None
    lib.nmt_debug_alloc_hook.argtypes = [_I32]
    lib.nmt_debug_alloc_hook.restype = ctypes.c_int64
    lib.nmt_debug_gemm_form.argtypes = [_I32]
    lib.nmt_debug_gemm_form.restype = _I32
    lib.nmt_debug_gemm_streamed.argtypes = []
    lib.nmt_debug_gemm_streamed.restype = ctypes.c_int64
    lib.nmt_debug_precompute.argtypes = [_I32]
    lib.nmt_debug_precompute.restype = _I32
    lib.nmt_last_error.argtypes = []
    lib.nmt_last_error.restype = ctypes.c_char_p
    for f in ("nmt_model_create", "nmt_encode", "nmt_source_from_annotations", "nmt_source_info",
              "nmt_score_batch", "nmt_score_batch_debug", "nmt_score_batch_noalloc", "nmt_stream_status", "nmt_profile_begin",
              "nmt_profile_end", "nmt_score_forest_step", "nmt_forest_build", "nmt_forest_shape",
              "nmt_forest_level", "nmt_forest_pair_paths", "nmt_score_forest", "nmt_model_average",
              "nmt_score_ensemble", "nmt_rescorer_create", "nmt_rescore_stack", "nmt_rescorer_info"):
        getattr(lib, f).restype = ctypes.c_int
    _lib = lib
    return lib


def debug_alloc_hook(fail_after: int) -> int:
    """Test hook (nmt_debug.h): make device allocations fail after
    ``fail_after`` more (negative: never); returns the library's live
    device allocations."""
    return int(load_library().nmt_debug_alloc_hook(fail_after))


def debug_gemm_form(form: int) -> int:
    """Test hook (nmt_debug.h): kernel form of the bf16 products: 0
    automatic, 1 weight-streaming wherever the shapes allow, 2 LDS-staged
    only, 3 / 4 as 1 with the plain products' in-block K split off / on;
    returns the previous form."""
    return int(load_library().nmt_debug_gemm_form(form))


def debug_gemm_streamed() -> int:
    """Test hook (nmt_debug.h): launches so far that streamed weights."""
    return int(load_library().nmt_debug_gemm_streamed())


def debug_precompute(on: int) -> int:
    """Test hook (nmt_debug.h): whether fp32 models created from now on
    take the previous word's and the context's products from precomputed
    tables and projections (1, the default) or compute them per step (0);
    returns the previous setting."""
    return int(load_library().nmt_debug_precompute(on))


def last_error() -> str:
    return load_library().nmt_last_error().decode()


def _check(rc: int):
    if rc != NMT_OK:
        raise NmtError(rc, last_error())


def _ptr(t) -> Optional[int]:
    """Device address of a torch tensor (None stays NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


class Model:
    """nmt_model_create / nmt_model_destroy around host fp32 parameters."""

    def __init__(self, params: Dict[str, np.ndarray], V_src: int, V: int, E: int, H: int, A: int,
                 wtype: str = "f32"):
        lib = load_library()
        self.V_src, self.V, self.E, self.H, self.A = V_src, V, E, H, A
        self.C = 2 * H
        self.wtype = wtype
        dims = Dims(V_src, V, E, H, A, NMT_BF16 if wtype == "bf16" else NMT_F32)
        keep = [np.ascontiguousarray(params[n], dtype=np.float32) for n in WEIGHT_FIELDS]
        w = Weights(*[a.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) for a in keep])
        h = _VP()
        _check(lib.nmt_model_create(ctypes.byref(dims), ctypes.byref(w), ctypes.byref(h)))
        self.handle = h

    @classmethod
    def from_workload(cls, wl) -> "Model":
        c = wl.cfg
        return cls(wl.params, c.V_src, c.V, c.E, c.H, c.A, c.wtype)

    @classmethod
    def _wrap(cls, handle, like: "Model") -> "Model":
        m = cls.__new__(cls)
        m.V_src, m.V, m.E, m.H, m.A, m.C, m.wtype = like.V_src, like.V, like.E, like.H, like.A, like.C, like.wtype
        m.handle = handle
        return m

    def close(self):
        if getattr(self, "handle", None):
            load_library().nmt_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Source:
    """An nmt_source (annotations, attention keys, lengths of S sentences)."""

    def __init__(self, handle, S: int, Tpad: int, src_len: np.ndarray, model: Model):
        self.handle, self.S, self.Tpad, self.src_len, self.model = handle, S, Tpad, src_len, model

    def device_views(self):
        """(ctx_ptr, pctx_ptr) device addresses of the source's buffers."""
        c, p = _VP(), _VP()
        _check(load_library().nmt_source_info(self.handle, None, None, ctypes.byref(c), ctypes.byref(p)))
        return c.value, p.value

    def copy_out(self):
        """Copies of (ctx [S,Tpad,2H], pctx [S,Tpad,A]) as device tensors (test helper)."""
        import torch
        cptr, pptr = self.device_views()
        m = self.model
        ctx = torch.empty((self.S, self.Tpad, m.C), dtype=torch.float32, device="cuda")
        pctx = torch.empty((self.S, self.Tpad, m.A), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        _hip_memcpy_d2d(ctx.data_ptr(), cptr, ctx.numel() * 4)
        _hip_memcpy_d2d(pctx.data_ptr(), pptr, pctx.numel() * 4)
        return ctx, pctx

    def close(self):
        if getattr(self, "handle", None):
            load_library().nmt_source_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


_hip = None


def _hip_memcpy(dst: int, src: int, nbytes: int, kind: int):
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpy.argtypes = [_VP, _VP, ctypes.c_size_t, ctypes.c_int]
    rc = _hip.hipMemcpy(dst, src, nbytes, kind)
    if rc != 0:
        raise RuntimeError(f"hipMemcpy failed ({rc})")


def _hip_memcpy_d2d(dst: int, src: int, nbytes: int):
    _hip_memcpy(dst, src, nbytes, 3)  # hipMemcpyDeviceToDevice


def _hip_memcpy_d2h(out: np.ndarray, src: int):
    _hip_memcpy(out.ctypes.data, src, out.nbytes, 2)  # hipMemcpyDeviceToHost


def _len_array(src_len):
    a = np.ascontiguousarray(src_len, dtype=np.int32)
    return a, a.ctypes.data_as(ctypes.POINTER(_I32))


def nmt_encode(model: Model, src_ids, src_len, s0_out=None, stream=None) -> Source:
    """Source initialisation from device ids [S, Tpad] int32 and host lengths [S]."""
    lib = load_library()
    S, T = int(src_ids.shape[0]), int(src_ids.shape[1])
    lens, lp = _len_array(src_len)
    h = _VP()
    _check(lib.nmt_encode(model.handle, S, T, _ptr(src_ids), lp, _ptr(s0_out), _stream(stream), ctypes.byref(h)))
    return Source(h, S, T, lens.copy(), model)


def nmt_source_from_annotations(model: Model, ctx, src_len, stream=None) -> Source:
    lib = load_library()
    S, T = int(ctx.shape[0]), int(ctx.shape[1])
    lens, lp = _len_array(src_len)
    h = _VP()
    _check(lib.nmt_source_from_annotations(model.handle, S, T, _ptr(ctx), lp, _stream(stream), ctypes.byref(h)))
    return Source(h, S, T, lens.copy(), model)


def nmt_score_workspace_bytes(model: Model, B: int) -> int:
    return int(load_library().nmt_score_workspace_bytes(model.handle, B))


def nmt_score_batch(model: Model, src: Source, s_prev, y_prev, sent_id, req, logp, s_new, logZ=None,
                    workspace=None, stream=None, alpha=None, c=None, s1=None, t=None):
    """One batched decoder step; outputs are written into the given tensors.

    With any of ``alpha``, ``c``, ``s1``, ``t`` given, nmt_score_batch_debug is
    called and those intermediates are written too.
    """
    import torch
    lib = load_library()
    B = int(y_prev.shape[0])
    if workspace is None:
        workspace = torch.empty(max(nmt_score_workspace_bytes(model, B), 256), dtype=torch.uint8, device="cuda")
    args = [model.handle, src.handle, B, _ptr(s_prev), _ptr(y_prev), _ptr(sent_id), _ptr(req), _ptr(logp),
            _ptr(s_new), _ptr(logZ), _ptr(workspace), workspace.numel(), _stream(stream)]
    if any(x is not None for x in (alpha, c, s1, t)):
        _check(lib.nmt_score_batch_debug(*args, _ptr(alpha), _ptr(c), _ptr(s1), _ptr(t)))
    else:
        _check(lib.nmt_score_batch(*args))


# The scratch size of nmt_score_batch_noalloc (NMT_NOALLOC_SCRATCH_BYTES in nmt.h).
NOALLOC_SCRATCH_BYTES = 64 << 20


def nmt_score_batch_noalloc(model: Model, src: Source, s_prev, y_prev, sent_id, req, logp, s_new, logZ=None,
                            stream=None):
    """nmt_score_batch on the library's own per-device scratch: allocates nothing."""
    B = int(y_prev.shape[0])
    _check(load_library().nmt_score_batch_noalloc(model.handle, src.handle, B, _ptr(s_prev), _ptr(y_prev),
                                                  _ptr(sent_id), _ptr(req), _ptr(logp), _ptr(s_new), _ptr(logZ),
                                                  _stream(stream)))


def _handles(objs):
    return (_VP * len(objs))(*[o.handle for o in objs])


def nmt_model_average(models, coef=None, stream=None) -> Model:
    """Element-wise weighted average of K models with identical dimensions."""
    lib = load_library()
    K = len(models)
    c = None if coef is None else (ctypes.c_float * K)(*[float(x) for x in coef])
    h = _VP()
    _check(lib.nmt_model_average(K, _handles(models), c, _stream(stream), ctypes.byref(h)))
    return Model._wrap(h, models[0])


def nmt_ensemble_workspace_bytes(models, B: int) -> int:
    return int(load_library().nmt_ensemble_workspace_bytes(len(models), _handles(models), B))


def nmt_score_ensemble(models, srcs, s_prev, y_prev, sent_id, req, logp, s_new, logZ=None, weights=None,
                       score=None, workspace=None, stream=None):
    """One batched step of the same rows under K models; logp is [K, B]."""
    import torch
    lib = load_library()
    K, B = len(models), int(y_prev.shape[0])
    if workspace is None:
        workspace = torch.empty(max(nmt_ensemble_workspace_bytes(models, B), 256), dtype=torch.uint8, device="cuda")
    sp = (_VP * K)(*[_ptr(x) for x in s_prev])
    sn = (_VP * K)(*[_ptr(x) for x in s_new])
    w = None if weights is None else (ctypes.c_float * K)(*[float(x) for x in weights])
    _check(lib.nmt_score_ensemble(K, _handles(models), _handles(srcs), B, sp, _ptr(y_prev), _ptr(sent_id),
                                  _ptr(req), _ptr(logp), sn, _ptr(logZ), w, _ptr(score), _ptr(workspace),
                                  workspace.numel(), _stream(stream)))


def nmt_stream_status(model: Model, stream=None) -> int:
    """Status code (NMT_OK / NMT_ERANGE / ...) without raising."""
    return int(load_library().nmt_stream_status(model.handle, _stream(stream)))


def nmt_profile_begin(model: Model, max_steps: int):
    _check(load_library().nmt_profile_begin(model.handle, max_steps))


def nmt_profile_end(model: Model, stream=None) -> dict:
    """Summed milliseconds per phase over the timed steps, plus ``steps``."""
    t = Timing()
    _check(load_library().nmt_profile_end(model.handle, _stream(stream), ctypes.byref(t)))
    out = {name: float(t.ms[i]) for i, name in enumerate(PHASES)}
    out["steps"] = int(t.steps)
    return out


def nmt_score_forest_step(model: Model, src: Source, state_pool, state_row, y_prev, sent_id, req_off, req, logp,
                          s_new, logZ=None, workspace=None, stream=None):
    """One ScoreBatch level: gathered input states, CSR requests (see nmt.h)."""
    import torch
    lib = load_library()
    B = int(y_prev.shape[0])
    if workspace is None:
        workspace = torch.empty(max(nmt_score_workspace_bytes(model, B), 256), dtype=torch.uint8, device="cuda")
    _check(lib.nmt_score_forest_step(model.handle, src.handle, B, _ptr(state_pool), int(state_pool.shape[0]),
                                     _ptr(state_row), _ptr(y_prev), _ptr(sent_id), _ptr(req_off), _ptr(req),
                                     int(req.shape[0]), _ptr(logp), _ptr(s_new), _ptr(logZ), _ptr(workspace),
                                     workspace.numel(), _stream(stream)))


def _i32p(a):
    return a.ctypes.data_as(ctypes.POINTER(_I32))


class Forest:
    """nmt_forest_build over (hypothesis, phrase) pairs; host-only."""

    def __init__(self, hyp_word, hyp_sent, pair_hyp, phrases):
        lib = load_library()
        self.hyp_word = np.ascontiguousarray(hyp_word, dtype=np.int32)
        self.hyp_sent = np.ascontiguousarray(hyp_sent, dtype=np.int32)
        self.pair_hyp = np.ascontiguousarray(pair_hyp, dtype=np.int32)
        self.phrase_off = np.zeros(len(phrases) + 1, dtype=np.int32)
        self.phrase_off[1:] = np.cumsum([len(p) for p in phrases])
        words = [w for p in phrases for w in p]
        self.phrase_words = np.asarray(words if words else [0], dtype=np.int32)
        self.n_hyp, self.n_pairs = len(self.hyp_word), len(phrases)
        h = _VP()
        _check(lib.nmt_forest_build(self.n_hyp, _i32p(self.hyp_word), _i32p(self.hyp_sent), self.n_pairs,
                                    _i32p(self.pair_hyp), _i32p(self.phrase_off), _i32p(self.phrase_words),
                                    ctypes.byref(h)))
        self.handle = h

    def shape(self) -> dict:
        v = [_I32() for _ in range(4)]
        _check(load_library().nmt_forest_shape(self.handle, *[ctypes.byref(x) for x in v]))
        return dict(zip(("depth", "n_rows", "n_req", "max_rows"), (int(x.value) for x in v)))

    def level(self, d: int) -> dict:
        lib = load_library()
        rows, nreq = _I32(), _I32()
        _check(lib.nmt_forest_level(self.handle, d, ctypes.byref(rows), ctypes.byref(nreq), None, None, None,
                                    None, None))
        R, Q = rows.value, nreq.value
        out = {k: np.zeros(n, np.int32) for k, n in (("state_row", R), ("y_prev", R), ("sent_id", R),
                                                        ("req_off", R + 1), ("req", Q))}
        _check(lib.nmt_forest_level(self.handle, d, None, None, *[_i32p(out[k]) for k in
                                                                   ("state_row", "y_prev", "sent_id", "req_off",
                                                                    "req")]))
        return out

    def pair_paths(self) -> np.ndarray:
        sh = self.shape()
        out = np.zeros((self.n_pairs, sh["depth"]), np.int32)
        if out.size:
            _check(load_library().nmt_forest_pair_paths(self.handle, _i32p(out)))
        return out

    def close(self):
        if getattr(self, "handle", None):
            load_library().nmt_forest_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def nmt_forest_workspace_bytes(model: Model, forest: Forest) -> int:
    return int(load_library().nmt_forest_workspace_bytes(model.handle, forest.handle))


def nmt_score_forest(model: Model, src: Source, forest: Forest, hyp_states, pair_logp, req_logp=None,
                     node_states=None, workspace=None, stream=None):
    """ScoreBatch on the device: per-pair log p(phrase | hypothesis)."""
    import torch
    lib = load_library()
    if workspace is None:
        workspace = torch.empty(max(nmt_forest_workspace_bytes(model, forest), 256), dtype=torch.uint8,
                                device="cuda")
    _check(lib.nmt_score_forest(model.handle, src.handle, forest.handle, _ptr(hyp_states), _ptr(pair_logp),
                                _ptr(req_logp), _ptr(node_states), _ptr(workspace), workspace.numel(),
                                _stream(stream)))


def phrases_csr(phrases):
    """Flattens a list of phrases (sequences of word ids) into (off, words):
    phrase j is words[off[j]:off[j+1]]."""
    n = len(phrases)
    off = np.zeros(n + 1, np.int32)
    np.cumsum(np.fromiter(map(len, phrases), np.int32, n), out=off[1:])
    words = np.fromiter(itertools.chain.from_iterable(phrases), np.int32, int(off[-1]))
    return off, words


class Rescorer:
    """Stack rescoring state (nmt_rescorer): per-model hypothesis states on the device."""

    def __init__(self, models, srcs, s0, capacity: int, stream=None):
        lib = load_library()
        self.K = len(models)
        self._keep = (list(models), list(srcs), list(s0))
        s0p = (_VP * self.K)(*[_ptr(x) for x in s0])
        h = _VP()
        _check(lib.nmt_rescorer_create(self.K, _handles(models), _handles(srcs), s0p, capacity, _stream(stream),
                                       ctypes.byref(h)))
        self.handle = h

    def rescore(self, parents, phrases, stream=None):
        """-> (logp [K, n] float32, ids [n] int32) for hypotheses (parents[j], phrases[j])."""
        off, words = phrases_csr(phrases)
        return self.rescore_csr(parents, off, words, stream)

    def rescore_csr(self, parents, off, words, stream=None):
        """rescore() with the phrases already flattened: hypothesis j's phrase is
        words[off[j]:off[j+1]] (int32 arrays, off[0] = 0)."""
        lib = load_library()
        par = np.ascontiguousarray(parents, dtype=np.int32)
        off = np.ascontiguousarray(off, dtype=np.int32)
        words = np.ascontiguousarray(words, dtype=np.int32)
        n = len(par)
        if off.shape != (n + 1,):
            raise ValueError("off must hold one offset more than there are parents")
        logp = np.empty((self.K, n), np.float32)
        ids = np.empty(n, np.int32)
        _check(lib.nmt_rescore_stack(self.handle, n, _i32p(par), _i32p(off), _i32p(words) if words.size else None,
                                     logp.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), _i32p(ids),
                                     _stream(stream)))
        return logp, ids

    def info(self, k: int = 0) -> dict:
        lib = load_library()
        d = _VP()
        v = [_I32() for _ in range(5)]
        _check(lib.nmt_rescorer_info(self.handle, k, ctypes.byref(d), *[ctypes.byref(x) for x in v]))
        return {"d_states": d.value, "n_hyp": v[0].value, "last_pairs": v[1].value, "last_rows": v[2].value,
                "last_edges": v[3].value, "last_depth": v[4].value}

    def states(self, k: int = 0, H: int = None):
        """Host copy of model k's states of all hypotheses so far."""
        inf = self.info(k)
        H = H or self._keep[0][k].H
        out = np.empty((inf["n_hyp"], H), np.float32)
        if out.size:
            _hip_memcpy_d2h(out, inf["d_states"])
        return out

    def close(self):
        if getattr(self, "handle", None):
            load_library().nmt_rescorer_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
