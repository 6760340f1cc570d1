"""ctypes wrapper of the CPU oracle (liboracle_rvqsd.so).

TEST INFRASTRUCTURE: only the tests, the smoke check and the benchmark's
CPU-baseline leg use this module.  It imports nothing from the GPU package.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle_rvqsd.so")
SRC_PATH = os.path.join(HERE, "rvqsd_oracle.c")

DRAFT_SAMPLED, DRAFT_GREEDY, DRAFT_SELF = 0, 1, 2
MAX_ROUNDS = 16
TRACE_ROWS = 16


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc (fp64, no FMA contraction, OpenMP over output rows)."""
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-ffp-contract=off", "-fopenmp", "-shared", "-fPIC",
           "-o", LIB_PATH + ".tmp", SRC_PATH, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


class OrcCfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "hidden", "n_q_heads", "n_kv_heads", "head_dim", "ffn", "n_codes", "vocab", "max_draft",
        "dtype", "qk_norm", "topk", "draft_len", "draft_mode")] + [
        ("rms_eps", ctypes.c_double), ("rope_base", ctypes.c_double), ("temperature", ctypes.c_double)]


class OrcStats(ctypes.Structure):
    _fields_ = [("target_calls", ctypes.c_int32), ("rounds", ctypes.c_int32), ("drafted", ctypes.c_int32),
                ("accepted", ctypes.c_int32), ("accept_mask", ctypes.c_uint32)]

    def as_dict(self):
        return {k: int(getattr(self, k)) for k, _ in self._fields_}


class OrcRound(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int32), ("kp", ctypes.c_int32), ("n_rows", ctypes.c_int32), ("m_new", ctypes.c_int32),
                ("drafts", ctypes.c_int32 * 16), ("accepted", ctypes.c_int32), ("token", ctypes.c_int32),
                ("margin", ctypes.c_double), ("topk_gap", ctypes.c_double)]


class OrcTrace(ctypes.Structure):
    _fields_ = [("rounds", ctypes.POINTER(OrcRound)), ("verify_logits", ctypes.POINTER(ctypes.c_double)),
                ("draft_logits", ctypes.POINTER(ctypes.c_double)), ("max_rounds", ctypes.c_int32),
                ("n_rounds", ctypes.c_int32)]


MAX_TREE = 80


class OrcTree(ctypes.Structure):
    _fields_ = [("n_nodes", ctypes.c_int32), ("parent", ctypes.c_int32 * (MAX_TREE + 1)),
                ("rank", ctypes.c_int32 * (MAX_TREE + 1))]


class OrcTreeRound(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int32), ("depth", ctypes.c_int32), ("n_rows", ctypes.c_int32),
                ("m_new", ctypes.c_int32), ("n_cand", ctypes.c_int32), ("accepted", ctypes.c_int32),
                ("token", ctypes.c_int32),
                ("tokens", ctypes.c_int32 * (MAX_TREE + 1)), ("path", ctypes.c_int32 * 16),
                ("margin", ctypes.c_double), ("topk_gap", ctypes.c_double)]


class OrcTreeTrace(ctypes.Structure):
    _fields_ = [("rounds", ctypes.POINTER(OrcTreeRound)), ("verify_logits", ctypes.POINTER(ctypes.c_double)),
                ("draft_logits", ctypes.POINTER(ctypes.c_double)), ("max_rounds", ctypes.c_int32),
                ("n_rounds", ctypes.c_int32)]


def make_tree(parents, ranks) -> OrcTree:
    """parents[i], ranks[i] of packed rows 1..N (row 0 is the root)."""
    t = OrcTree()
    t.n_nodes = len(parents)
    for i, (p, r) in enumerate(zip(parents, ranks), start=1):
        t.parent[i] = int(p)
        t.rank[i] = int(r)
    return t


PROBE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_double), ctypes.c_int32)

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        i32, f64, vp = ctypes.c_int32, ctypes.c_double, ctypes.c_void_p
        L.orc_create.restype = vp
        L.orc_create.argtypes = [P(OrcCfg), vp, ctypes.c_size_t, P(i32)]
        L.orc_destroy.argtypes = [vp]
        L.orc_set_threads.argtypes = [i32]
        L.orc_get_threads.restype = i32
        L.orc_forward.argtypes = [vp, vp, vp, i32, vp]
        L.orc_forward_vectors.argtypes = [vp, vp, i32, vp]
        L.orc_logits.argtypes = [vp, vp, i32, i32, vp]
        L.orc_topk_softmax.argtypes = [vp, i32, i32, f64, vp, vp]
        L.orc_sample.argtypes = [vp, vp, i32, f64]
        L.orc_accept_or_resample.argtypes = [vp, vp, i32, vp, vp, i32, i32, f64, f64, P(i32)]
        L.orc_ar_frame.argtypes = [vp, vp, i32, vp, vp]
        L.orc_spec_frame.argtypes = [vp, vp, i32, vp, vp, P(OrcStats), P(OrcTrace), PROBE_FN, vp]
        L.orc_uniforms_from_seed.argtypes = [ctypes.c_uint64, i32, vp]
        L.orc_tree_mask.argtypes = [P(OrcTree), vp]
        L.orc_tree_hidden.argtypes = [vp, P(OrcTree), vp, vp, i32, vp, i32, vp]
        L.orc_tree_frame.argtypes = [vp, P(OrcTree), vp, i32, vp, vp, P(OrcStats), P(OrcTreeTrace), PROBE_FN, vp]
        L.orc_splitmix64_at.restype = ctypes.c_uint64
        L.orc_splitmix64_at.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        for name in ("orc_forward", "orc_forward_vectors", "orc_logits", "orc_topk_softmax", "orc_sample", "orc_accept_or_resample",
                     "orc_ar_frame", "orc_spec_frame", "orc_abi_version", "orc_tree_mask", "orc_tree_hidden",
                     "orc_tree_frame"):
            getattr(L, name).restype = i32
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class OracleError(RuntimeError):
    pass


def _check(st: int, what: str):
    if st < 0:
        raise OracleError(f"{what} failed with status {st}")
    return st


class Oracle:
    """One oracle model.  Shape fields follow the weight blob's header."""

    def __init__(self, blob: bytes, *, n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, n_codes, vocab,
                 max_draft, dtype, topk, temperature, draft_len, draft_mode=DRAFT_SAMPLED, qk_norm=1,
                 rms_eps=1e-6, rope_base=1e6):
        self.cfg = OrcCfg(n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, n_codes, vocab, max_draft, dtype,
                          qk_norm, topk, draft_len, draft_mode, rms_eps, rope_base, temperature)
        self._blob = bytes(blob)
        st = ctypes.c_int32(0)
        self._h = lib().orc_create(ctypes.byref(self.cfg), ctypes.c_char_p(self._blob), len(self._blob),
                                   ctypes.byref(st))
        if not self._h:
            raise OracleError(f"orc_create failed with status {st.value}")

    def close(self):
        if getattr(self, "_h", None):
            lib().orc_destroy(self._h)
            self._h = None

    __del__ = close

    @property
    def H(self):
        return self.cfg.hidden

    @property
    def V(self):
        return self.cfg.vocab

    @property
    def n(self):
        return self.cfg.n_codes

    def forward(self, f: np.ndarray, in_codes) -> np.ndarray:
        """Final-normed hidden states of positions 0..len(in_codes) (fp64)."""
        f = np.ascontiguousarray(f, dtype=np.float32)
        ic = np.ascontiguousarray(np.asarray(in_codes, dtype=np.int32).reshape(-1))
        n_pos = ic.size + 1
        out = np.zeros((n_pos, self.H), dtype=np.float64)
        _check(lib().orc_forward(self._h, _ptr(f), _ptr(ic) if ic.size else None, n_pos, _ptr(out)), "orc_forward")
        return out

    def forward_vectors(self, rows: np.ndarray) -> np.ndarray:
        """Final-normed hidden states of positions 0..n-1 for input rows [n][H] (fp64)."""
        x = np.ascontiguousarray(rows, dtype=np.float64)
        out = np.zeros_like(x)
        _check(lib().orc_forward_vectors(self._h, _ptr(x), x.shape[0], _ptr(out)), "orc_forward_vectors")
        return out

    def logits(self, h: np.ndarray, head: int, offset: int = 0) -> np.ndarray:
        h = np.ascontiguousarray(h, dtype=np.float64)
        out = np.zeros(self.V, dtype=np.float64)
        _check(lib().orc_logits(self._h, _ptr(h), head, offset, _ptr(out)), "orc_logits")
        return out

    def ar_frame(self, f, c0: int, uni) -> np.ndarray:
        f = np.ascontiguousarray(f, dtype=np.float32)
        u = np.ascontiguousarray(uni, dtype=np.float32)
        out = np.zeros(self.n, dtype=np.int32)
        _check(lib().orc_ar_frame(self._h, _ptr(f), int(c0), _ptr(u), _ptr(out)), "orc_ar_frame")
        return out

    def spec_frame(self, f, c0: int, uni, trace: bool = False, probe=None, logits: bool = False):
        """Returns (codes, stats dict, trace dict or None)."""
        f = np.ascontiguousarray(f, dtype=np.float32)
        u = np.ascontiguousarray(uni, dtype=np.float32)
        out = np.zeros(self.n, dtype=np.int32)
        st = OrcStats()
        tr_p = None
        if trace:
            rounds = (OrcRound * MAX_ROUNDS)()
            vl = dl = None
            if logits:
                vl = np.zeros((MAX_ROUNDS, TRACE_ROWS, self.V), dtype=np.float64)
                dl = np.zeros((MAX_ROUNDS, TRACE_ROWS, self.V), dtype=np.float64)
            tr = OrcTrace(rounds, vl.ctypes.data_as(ctypes.POINTER(ctypes.c_double)) if logits else None,
                          dl.ctypes.data_as(ctypes.POINTER(ctypes.c_double)) if logits else None, MAX_ROUNDS, 0)
            tr_p = ctypes.byref(tr)
        cb = PROBE_FN(probe) if probe is not None else PROBE_FN()
        _check(lib().orc_spec_frame(self._h, _ptr(f), int(c0), _ptr(u), _ptr(out), ctypes.byref(st), tr_p, cb, None),
               "orc_spec_frame")
        tdict = None
        if trace:
            rs = []
            for i in range(tr.n_rounds):
                r = rounds[i]
                rs.append(dict(m=r.m, kp=r.kp, n_rows=r.n_rows, m_new=r.m_new, drafts=list(r.drafts[:r.kp]),
                               accepted=r.accepted, token=r.token, margin=r.margin, topk_gap=r.topk_gap))
            tdict = {"rounds": rs}
            if logits:
                tdict["verify_logits"] = vl[:tr.n_rounds]
                tdict["draft_logits"] = dl[:tr.n_rounds]
        return out, st.as_dict(), tdict


def tree_mask(tree: OrcTree) -> np.ndarray:
    n = tree.n_nodes + 1
    out = np.zeros(n * n, dtype=np.int32)
    _check(lib().orc_tree_mask(ctypes.byref(tree), _ptr(out)), "orc_tree_mask")
    return out.reshape(n, n)


def _tree_frame(self, tree: OrcTree, f, c0: int, uni, trace: bool = False, probe=None, logits: bool = False):
    """Speculative frame with sparse-tree drafting. Returns (codes, stats, trace dict or None)."""
    f = np.ascontiguousarray(f, dtype=np.float32)
    u = np.ascontiguousarray(uni, dtype=np.float32)
    out = np.zeros(self.n, dtype=np.int32)
    st = OrcStats()
    tr_p = None
    if trace:
        rounds = (OrcTreeRound * MAX_ROUNDS)()
        vl = dl = None
        if logits:
            vl = np.zeros((MAX_ROUNDS, MAX_TREE + 1, self.V), dtype=np.float64)
            dl = np.zeros((MAX_ROUNDS, TRACE_ROWS, self.V), dtype=np.float64)
        tr = OrcTreeTrace(rounds, vl.ctypes.data_as(ctypes.POINTER(ctypes.c_double)) if logits else None,
                          dl.ctypes.data_as(ctypes.POINTER(ctypes.c_double)) if logits else None, MAX_ROUNDS, 0)
        tr_p = ctypes.byref(tr)
    cb = PROBE_FN(probe) if probe is not None else PROBE_FN()
    _check(lib().orc_tree_frame(self._h, ctypes.byref(tree), _ptr(f), int(c0), _ptr(u), _ptr(out), ctypes.byref(st),
                                tr_p, cb, None), "orc_tree_frame")
    tdict = None
    if trace:
        rs = []
        for i in range(tr.n_rounds):
            r = rounds[i]
            rs.append(dict(m=r.m, depth=r.depth, n_rows=r.n_rows, n_cand=r.n_cand, m_new=r.m_new,
                           accepted=r.accepted, token=r.token, tokens=list(r.tokens[:max(r.n_cand, r.n_rows)]), path=list(r.path[:r.accepted]), margin=r.margin,
                           topk_gap=r.topk_gap))
        tdict = {"rounds": rs}
        if logits:
            tdict["verify_logits"] = vl[:tr.n_rounds]
            tdict["draft_logits"] = dl[:tr.n_rounds]
    return out, st.as_dict(), tdict


def _tree_hidden(self, tree: OrcTree, f, committed, tokens) -> np.ndarray:
    """Hidden states of the packed rows: committed = c_0..c_m, tokens = tokens of rows 1..R-1."""
    f = np.ascontiguousarray(f, dtype=np.float32)
    cm = np.ascontiguousarray(np.asarray(committed, dtype=np.int32))
    tk = np.ascontiguousarray(np.asarray([0] + list(tokens), dtype=np.int32))
    n_rows = tk.size
    out = np.zeros((n_rows, self.H), dtype=np.float64)
    _check(lib().orc_tree_hidden(self._h, ctypes.byref(tree), _ptr(f), _ptr(cm), cm.size - 1, _ptr(tk), n_rows,
                                 _ptr(out)), "orc_tree_hidden")
    return out


Oracle.tree_frame = _tree_frame
Oracle.tree_hidden = _tree_hidden


def topk_softmax(logits, topk: int, temperature: float):
    lg = np.ascontiguousarray(logits, dtype=np.float64)
    idx = np.zeros(lg.size, dtype=np.int32)
    pr = np.zeros(lg.size, dtype=np.float64)
    k = _check(lib().orc_topk_softmax(_ptr(lg), lg.size, topk, temperature, _ptr(idx), _ptr(pr)), "topk_softmax")
    return idx[:k].copy(), pr[:k].copy()


def sample(idx, prob, u: float) -> int:
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    prob = np.ascontiguousarray(prob, dtype=np.float64)
    return _check(lib().orc_sample(_ptr(idx), _ptr(prob), idx.size, float(u)), "sample")


def accept_or_resample(pidx, pp, qidx, qp, d: int, u_acc: float, u_samp: float):
    """(accepted: bool, token): token = d when accepted, else the residual sample."""
    pidx = np.ascontiguousarray(pidx, dtype=np.int32)
    pp = np.ascontiguousarray(pp, dtype=np.float64)
    qidx = np.ascontiguousarray(qidx, dtype=np.int32)
    qp = np.ascontiguousarray(qp, dtype=np.float64)
    tok = ctypes.c_int32(-1)
    a = _check(lib().orc_accept_or_resample(_ptr(pidx), _ptr(pp), pidx.size, _ptr(qidx), _ptr(qp), qidx.size,
                                            int(d), float(u_acc), float(u_samp), ctypes.byref(tok)),
               "accept_or_resample")
    return (True, int(d)) if a == 1 else (False, int(tok.value))


def uniforms_from_seed(seed: int, n_codes: int = 15) -> np.ndarray:
    out = np.zeros((n_codes, 3), dtype=np.float32)
    lib().orc_uniforms_from_seed(ctypes.c_uint64(seed), n_codes, _ptr(out))
    return out


def splitmix64_at(seed: int, n: int) -> int:
    return int(lib().orc_splitmix64_at(ctypes.c_uint64(seed), ctypes.c_uint64(n)))


def set_threads(n: int):
    lib().orc_set_threads(int(n))


def get_threads() -> int:
    return int(lib().orc_get_threads())


def pipeline_frames(outer: Oracle, emb0: np.ndarray, tables: np.ndarray, inner: Oracle, t: np.ndarray,
                    u_c0: np.ndarray, uni: np.ndarray, topk: int, temperature: float):
    """The full per-frame pipeline of Fig. 1 from scratch (test reference).

    Frame i: the outer decoder's input is x_i = t_i + E_0[c_0] + sum_j E_j[c_j] of frame
    i - 1 (x_0 = t_0); the outer decoder runs over x_0..x_i (positions 0..i) and its
    final-normed hidden h_i gives the c_0 logits through its head; entries at or above
    the inner codebook size are masked (codes the inner tables cannot embed); c_0 is the
    top-k, temperature-T sample at u_c0[i]; the inner loop decodes c_1..c_15 from
    (float32(h_i), c_0) with the frame's uniforms.  emb0: [V_outer][H] (outer E_0);
    tables: [15][V_inner][H].  Returns codes [n][16], inner stats, and the h_i [n][H].
    """
    n, H = t.shape
    V_in = inner.V
    rows, codes, stats, hs = [], [], [], []
    prev = None
    for i in range(n):
        x = t[i].astype(np.float64)
        if prev is not None:
            x = x + emb0[prev[0]].astype(np.float64)
            for j in range(1, len(prev)):
                x = x + tables[j - 1][prev[j]].astype(np.float64)
        rows.append(x)
        h = outer.forward_vectors(np.stack(rows))[-1]
        lg = outer.logits(h, 1)
        lg[V_in:] = -np.inf
        idx, p = topk_softmax(lg, topk, temperature)
        c0 = sample(idx, p, float(u_c0[i]))
        c, st, _ = inner.spec_frame(h.astype(np.float32), c0, uni[i])
        prev = [c0] + [int(v) for v in c]
        codes.append(prev)
        stats.append(st)
        hs.append(h)
    return np.array(codes, dtype=np.int32), stats, np.stack(hs)
