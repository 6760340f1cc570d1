"""Python binding of librvqsd.so (argument marshalling only).

Every step of the decode runs in the HIP library; this module converts
arguments and raises on error.  It fails loudly when the library is missing:
there is no CPU fallback.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import weakref

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librvqsd.so")

RVQSD_ABI_VERSION = 1
OK, EINVAL, EBLOB, ENOMEM, EHIP, EUNSUPPORTED, ENUMERIC, ETIMEOUT = 0, -1, -2, -3, -4, -5, -6, -7
DTYPE_F32, DTYPE_BF16, DTYPE_I8 = 0, 1, 2
TRACE_ROUND_INTS = 32

# every symbol include/rvqsd.h declares
EXPORTS = ("rvqsd_create", "rvqsd_destroy", "rvqsd_model_info", "rvqsd_stream_create", "rvqsd_tree_stream_create",
           "rvqsd_stream_destroy",
           "rvqsd_decode_frame", "rvqsd_decode_frame_u", "rvqsd_decode_frame_async", "rvqsd_decode_frames_async",
           "rvqsd_decode_frame_noalloc", "rvqsd_stream_reset",
           "rvqsd_set_trace", "rvqsd_decode_frames_batched", "rvqsd_decode_frames_batched_async",
           "rvqsd_batch_totals", "rvqsd_set_batch_trace", "rvqsd_outer_create", "rvqsd_outer_destroy", "rvqsd_outer_reset",
           "rvqsd_pipeline_frames_async", "rvqsd_uniforms_from_seed", "rvqsd_status_str", "rvqsd_last_error")


class rvqsd_cfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "abi_version", "n_layers", "hidden", "n_q_heads", "n_kv_heads", "head_dim", "ffn", "n_codes", "vocab",
        "max_draft", "dtype", "qk_norm", "topk", "draft_len", "draft_greedy")] + [
        ("matrix_path", ctypes.c_int32), ("reserved", ctypes.c_int32 * 2), ("rms_eps", ctypes.c_double),
        ("rope_base", ctypes.c_double),
        ("temperature", ctypes.c_double)]


class rvqsd_weights(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("bytes", ctypes.c_uint64)]


class rvqsd_stats(ctypes.Structure):
    _fields_ = [("target_calls", ctypes.c_int32), ("rounds", ctypes.c_int32), ("drafted", ctypes.c_int32),
                ("accepted", ctypes.c_int32), ("accept_mask", ctypes.c_uint32), ("status", ctypes.c_int32),
                ("weight_bytes", ctypes.c_uint64), ("clk_start", ctypes.c_uint64), ("clk_end", ctypes.c_uint64)]

    def as_dict(self):
        return {k: int(getattr(self, k)) for k, _ in self._fields_}


STATS_DTYPE = np.dtype([("target_calls", np.int32), ("rounds", np.int32), ("drafted", np.int32),
                        ("accepted", np.int32), ("accept_mask", np.uint32), ("status", np.int32),
                        ("weight_bytes", np.uint64), ("clk_start", np.uint64), ("clk_end", np.uint64)])
assert STATS_DTYPE.itemsize == ctypes.sizeof(rvqsd_stats)


class rvqsd_trace(ctypes.Structure):
    _fields_ = [("logits", ctypes.c_void_p), ("rounds", ctypes.c_void_p), ("clock", ctypes.c_void_p),
                ("wg_clock", ctypes.c_void_p), ("max_rounds", ctypes.c_int32), ("wg_ready", ctypes.c_void_p)]


class rvqsd_info(ctypes.Structure):
    _fields_ = [("workgroups", ctypes.c_int32), ("threads", ctypes.c_int32), ("max_rows", ctypes.c_int32),
                ("trace_slots", ctypes.c_int32), ("lds_bytes", ctypes.c_uint64),
                ("layer_weight_bytes", ctypes.c_uint64), ("head_bytes", ctypes.c_uint64),
                ("emb_row_bytes", ctypes.c_uint64), ("device_weight_bytes", ctypes.c_uint64)]

    def as_dict(self):
        return {k: int(getattr(self, k)) for k, _ in self._fields_}


class RvqsdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


_lib = None


# live handles, closed in this order by the exit hook below
_live = {"outer": weakref.WeakSet(), "stream": weakref.WeakSet(), "model": weakref.WeakSet()}


def _shutdown():
    """Interpreter-exit hook: close every live handle, then unload the library.

    Unloading runs the library's code-object unregistration now, while the HIP
    runtime (and any profiler attached to it) is still up, instead of from the
    C exit handlers after the process has begun tearing the runtime down. Objects
    that outlive this hook see the library gone and release nothing."""
    global _lib
    if _lib is None:
        return
    for kind in ("outer", "stream", "model"):
        for obj in list(_live[kind]):
            try:
                obj.close()
            except Exception:
                pass
    L, _lib = _lib, None
    try:
        import _ctypes
        _ctypes.dlclose(L._handle)
    except Exception:
        pass


atexit.register(_shutdown)


def lib():
    """Load librvqsd.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_37007_amd.build_ext`")
        L = ctypes.CDLL(LIB_PATH)
        P, vp, i32 = ctypes.POINTER, ctypes.c_void_p, ctypes.c_int32
        L.rvqsd_create.argtypes = [P(rvqsd_weights), P(rvqsd_cfg), P(vp)]
        L.rvqsd_destroy.argtypes = [vp]
        L.rvqsd_destroy.restype = None
        L.rvqsd_model_info.argtypes = [vp, P(rvqsd_info)]
        L.rvqsd_stream_create.argtypes = [vp, vp, i32, P(vp)]
        L.rvqsd_tree_stream_create.argtypes = [vp, vp, i32, i32, vp, vp, P(vp)]
        L.rvqsd_stream_destroy.argtypes = [vp]
        L.rvqsd_stream_destroy.restype = None
        L.rvqsd_decode_frame.argtypes = [vp, vp, i32, ctypes.c_uint64, vp, P(rvqsd_stats)]
        L.rvqsd_decode_frame_u.argtypes = [vp, vp, i32, vp, vp, P(rvqsd_stats)]
        L.rvqsd_decode_frame_async.argtypes = [vp, vp, vp, vp, vp, vp]
        L.rvqsd_decode_frames_async.argtypes = [vp, i32, vp, vp, vp, vp, vp]
        L.rvqsd_decode_frame_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp]
        L.rvqsd_set_trace.argtypes = [vp, P(rvqsd_trace)]
        L.rvqsd_decode_frames_batched.argtypes = [vp, i32, vp, vp, vp, vp, vp]
        L.rvqsd_decode_frames_batched_async.argtypes = [vp, i32, vp, vp, vp, vp, vp]
        L.rvqsd_batch_totals.argtypes = [vp, P(ctypes.c_uint64), P(ctypes.c_uint64)]
        L.rvqsd_set_batch_trace.argtypes = [vp, vp, vp, i32, i32]
        L.rvqsd_outer_create.argtypes = [vp, vp, i32, i32, i32, ctypes.c_double, i32, P(vp)]
        L.rvqsd_outer_destroy.argtypes = [vp]
        L.rvqsd_outer_destroy.restype = None
        L.rvqsd_outer_reset.argtypes = [vp]
        L.rvqsd_pipeline_frames_async.argtypes = [vp, vp, i32, vp, vp, vp, vp, vp, vp]
        L.rvqsd_stream_reset.argtypes = [vp]
        L.rvqsd_uniforms_from_seed.argtypes = [ctypes.c_uint64, i32, vp]
        L.rvqsd_status_str.argtypes = [i32]
        L.rvqsd_status_str.restype = ctypes.c_char_p
        L.rvqsd_last_error.argtypes = []
        L.rvqsd_last_error.restype = ctypes.c_char_p
        for n in ("rvqsd_create", "rvqsd_model_info", "rvqsd_stream_create", "rvqsd_tree_stream_create",
                  "rvqsd_decode_frame",
                  "rvqsd_decode_frame_u", "rvqsd_decode_frame_async", "rvqsd_decode_frames_async",
                  "rvqsd_decode_frame_noalloc",
                  "rvqsd_stream_reset", "rvqsd_set_trace",
                  "rvqsd_decode_frames_batched", "rvqsd_decode_frames_batched_async", "rvqsd_batch_totals",
                  "rvqsd_set_batch_trace",
                  "rvqsd_outer_create", "rvqsd_outer_reset", "rvqsd_pipeline_frames_async",
                  "rvqsd_uniforms_from_seed"):
            getattr(L, n).restype = i32
        _lib = L
    return _lib


def _check(st: int, what: str):
    if st != OK:
        raise RvqsdError(st, f"{what}: {lib().rvqsd_last_error().decode()}")


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def make_cfg(*, n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, n_codes, vocab, max_draft, dtype, topk,
             temperature, draft_len, draft_greedy=0, qk_norm=1, rms_eps=1e-6, rope_base=1e6,
             matrix_path=0) -> rvqsd_cfg:
    c = rvqsd_cfg()
    c.abi_version = RVQSD_ABI_VERSION
    for k, v in dict(n_layers=n_layers, hidden=hidden, n_q_heads=n_q_heads, n_kv_heads=n_kv_heads,
                     head_dim=head_dim, ffn=ffn, n_codes=n_codes, vocab=vocab, max_draft=max_draft, dtype=dtype,
                     qk_norm=qk_norm, topk=topk, draft_len=draft_len, draft_greedy=draft_greedy,
                     matrix_path=matrix_path).items():
        setattr(c, k, int(v))
    c.rms_eps, c.rope_base, c.temperature = float(rms_eps), float(rope_base), float(temperature)
    return c


def uniforms_from_seed(seed: int, n_codes: int = 15) -> np.ndarray:
    out = np.zeros((n_codes, 3), dtype=np.float32)
    _check(lib().rvqsd_uniforms_from_seed(ctypes.c_uint64(seed), n_codes, _ptr(out)), "rvqsd_uniforms_from_seed")
    return out


class Model:
    """rvqsd_create / rvqsd_destroy / rvqsd_model_info."""

    def __init__(self, blob: bytes, cfg: rvqsd_cfg):
        self.cfg = cfg
        self._blob = bytes(blob)
        w = rvqsd_weights(ctypes.cast(ctypes.c_char_p(self._blob), ctypes.c_void_p), len(self._blob))
        h = ctypes.c_void_p()
        _check(lib().rvqsd_create(ctypes.byref(w), ctypes.byref(cfg), ctypes.byref(h)), "rvqsd_create")
        self._h = h
        _live["model"].add(self)
        self._blob = None  # the library copied the weights

    def info(self) -> dict:
        i = rvqsd_info()
        _check(lib().rvqsd_model_info(self._h, ctypes.byref(i)), "rvqsd_model_info")
        return i.as_dict()

    def decode_frame_noalloc(self, hip_stream, d_frame_hidden: int, d_c0: int, d_uniforms: int, d_out_codes: int,
                             d_stats: int):
        """The allocation-free decode (device pointers, ints); enqueues only."""
        _check(lib().rvqsd_decode_frame_noalloc(self._h, ctypes.c_void_p(hip_stream or 0),
                                                ctypes.c_void_p(d_frame_hidden), ctypes.c_void_p(d_c0),
                                                ctypes.c_void_p(d_uniforms), ctypes.c_void_p(d_out_codes),
                                                ctypes.c_void_p(d_stats)), "rvqsd_decode_frame_noalloc")

    def close(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.rvqsd_destroy(self._h)
        self._h = None

    __del__ = close


class Stream:
    """rvqsd_stream_create and the decode calls; ``hip_stream`` is a raw hipStream_t (int) or None."""

    def __init__(self, model: Model, hip_stream=None, max_streams: int = 1, tree=None):
        """tree: (parents, ranks) of packed rows 1..N for sparse-tree verification."""
        self.model = model
        self.n = model.cfg.n_codes
        h = ctypes.c_void_p()
        if tree is None:
            _check(lib().rvqsd_stream_create(model._h, ctypes.c_void_p(hip_stream or 0), max_streams,
                                             ctypes.byref(h)), "rvqsd_stream_create")
        else:
            par = np.ascontiguousarray(tree[0], dtype=np.int32)
            rk = np.ascontiguousarray(tree[1], dtype=np.int32)
            _check(lib().rvqsd_tree_stream_create(model._h, ctypes.c_void_p(hip_stream or 0), max_streams, par.size,
                                                  _ptr(par), _ptr(rk), ctypes.byref(h)), "rvqsd_tree_stream_create")
        self.tree = tree
        self._h = h
        _live["stream"].add(self)
        self._trace = None

    def close(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.rvqsd_stream_destroy(self._h)
        self._h = None

    __del__ = close

    def decode_frame(self, frame_hidden, c0: int, rng_seed: int):
        f = np.ascontiguousarray(frame_hidden, dtype=np.float32)
        out = np.zeros(self.n, dtype=np.int32)
        st = rvqsd_stats()
        _check(lib().rvqsd_decode_frame(self._h, _ptr(f), int(c0), ctypes.c_uint64(rng_seed), _ptr(out),
                                        ctypes.byref(st)), "rvqsd_decode_frame")
        return out, st.as_dict()

    def decode_frame_u(self, frame_hidden, c0: int, uniforms):
        f = np.ascontiguousarray(frame_hidden, dtype=np.float32)
        u = np.ascontiguousarray(uniforms, dtype=np.float32)
        out = np.zeros(self.n, dtype=np.int32)
        st = rvqsd_stats()
        _check(lib().rvqsd_decode_frame_u(self._h, _ptr(f), int(c0), _ptr(u), _ptr(out), ctypes.byref(st)),
               "rvqsd_decode_frame_u")
        return out, st.as_dict()

    def decode_frame_async(self, d_frame_hidden: int, d_c0: int, d_uniforms: int, d_out_codes: int, d_stats: int):
        """Device pointers (ints, e.g. torch tensor data_ptr()); enqueues only."""
        _check(lib().rvqsd_decode_frame_async(self._h, ctypes.c_void_p(d_frame_hidden), ctypes.c_void_p(d_c0),
                                              ctypes.c_void_p(d_uniforms), ctypes.c_void_p(d_out_codes),
                                              ctypes.c_void_p(d_stats)), "rvqsd_decode_frame_async")

    def decode_frames_async(self, n: int, d_frame_hidden: int, d_c0: int, d_uniforms: int, d_out_codes: int,
                            d_stats: int):
        """n frames in order (device pointers to [n][H], [n], [n][n_codes][3], [n][n_codes], [n] stats);
        enqueues only, up to 1024 frames per launch."""
        _check(lib().rvqsd_decode_frames_async(self._h, int(n), ctypes.c_void_p(d_frame_hidden), ctypes.c_void_p(d_c0),
                                               ctypes.c_void_p(d_uniforms), ctypes.c_void_p(d_out_codes),
                                               ctypes.c_void_p(d_stats)), "rvqsd_decode_frames_async")

    def decode_frames_batched(self, frame_hidden, c0, uniforms):
        """Host arrays [n][H], [n], [n][n_codes][3] -> (codes [n][n_codes], stats structured array [n])."""
        f = np.ascontiguousarray(frame_hidden, dtype=np.float32)
        c = np.ascontiguousarray(c0, dtype=np.int32)
        u = np.ascontiguousarray(uniforms, dtype=np.float32)
        nfr = int(c.shape[0])
        out = np.full((nfr, self.n), -1, dtype=np.int32)
        st = np.zeros(nfr, dtype=STATS_DTYPE)
        _check(lib().rvqsd_decode_frames_batched(self._h, nfr, _ptr(f), _ptr(c), _ptr(u), _ptr(out), _ptr(st)),
               "rvqsd_decode_frames_batched")
        return out, st

    def decode_frames_batched_async(self, n: int, d_frame_hidden: int, d_c0: int, d_uniforms: int,
                                    d_out_codes: int, d_stats: int):
        """Device pointers (ints); enqueues only."""
        _check(lib().rvqsd_decode_frames_batched_async(self._h, int(n), ctypes.c_void_p(d_frame_hidden),
                                                       ctypes.c_void_p(d_c0), ctypes.c_void_p(d_uniforms),
                                                       ctypes.c_void_p(d_out_codes), ctypes.c_void_p(d_stats)),
               "rvqsd_decode_frames_batched_async")

    def batch_totals(self):
        """(passes, algorithmic bytes) of the last batched call; synchronises the stream."""
        a, b = ctypes.c_uint64(), ctypes.c_uint64()
        _check(lib().rvqsd_batch_totals(self._h, ctypes.byref(a), ctypes.byref(b)), "rvqsd_batch_totals")
        return int(a.value), int(b.value)

    def set_batch_trace(self, logits_ptr: int = 0, rounds_ptr: int = 0, max_rounds: int = 0, max_frames: int = 0):
        """Per-frame trace of later batched calls (device pointers); no pointers = off."""
        _check(lib().rvqsd_set_batch_trace(self._h, ctypes.c_void_p(logits_ptr or None),
                                           ctypes.c_void_p(rounds_ptr or None), int(max_rounds), int(max_frames)),
               "rvqsd_set_batch_trace")

    def reset(self):
        _check(lib().rvqsd_stream_reset(self._h), "rvqsd_stream_reset")

    def set_trace(self, logits_ptr: int = 0, rounds_ptr: int = 0, clock_ptr: int = 0, max_rounds: int = 0,
                  wg_clock_ptr: int = 0, wg_ready_ptr: int = 0):
        if not (logits_ptr or rounds_ptr or clock_ptr or wg_clock_ptr or wg_ready_ptr):
            _check(lib().rvqsd_set_trace(self._h, None), "rvqsd_set_trace")
            self._trace = None
            return
        t = rvqsd_trace(logits_ptr or None, rounds_ptr or None, clock_ptr or None, wg_clock_ptr or None, max_rounds,
                        wg_ready_ptr or None)
        _check(lib().rvqsd_set_trace(self._h, ctypes.byref(t)), "rvqsd_set_trace")
        self._trace = t


class Outer:
    """rvqsd_outer_create / rvqsd_outer_reset / rvqsd_pipeline_frames_async."""

    def __init__(self, model: Model, code_tables: bytes, n_tables: int, table_vocab: int, topk: int,
                 temperature: float, max_frames: int):
        self.model = model
        tab = bytes(code_tables)
        h = ctypes.c_void_p()
        _check(lib().rvqsd_outer_create(model._h, ctypes.c_char_p(tab), n_tables, table_vocab, topk,
                                        float(temperature), max_frames, ctypes.byref(h)), "rvqsd_outer_create")
        self._h = h
        _live["outer"].add(self)

    def reset(self):
        _check(lib().rvqsd_outer_reset(self._h), "rvqsd_outer_reset")

    def pipeline_async(self, stream: "Stream", n: int, d_t: int, d_u_c0: int, d_uniforms: int, d_codes: int,
                       d_stats: int, d_hidden: int = 0):
        """Device pointers (ints); enqueues n frames on the inner stream."""
        _check(lib().rvqsd_pipeline_frames_async(stream._h, self._h, int(n), ctypes.c_void_p(d_t),
                                                 ctypes.c_void_p(d_u_c0), ctypes.c_void_p(d_uniforms),
                                                 ctypes.c_void_p(d_codes), ctypes.c_void_p(d_stats),
                                                 ctypes.c_void_p(d_hidden or None)), "rvqsd_pipeline_frames_async")

    def close(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.rvqsd_outer_destroy(self._h)
        self._h = None

    __del__ = close
