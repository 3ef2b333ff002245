"""ctypes wrapper around ``mot_oracle.c`` (plain C, double precision).

TEST INFRASTRUCTURE ONLY (tests, smoke check, CPU-baseline timing).

Array conventions (all numpy, C-contiguous):
  src_k, src_v : float32 [L_src][B][T][H_src][D_src]  (or [L][B][H][T][D])
  w1 : float32 [L_tgt][2][E][hidden][d_in]     b1 : [L_tgt][2][E][hidden]
  w2 : float32 [L_tgt][2][E][d_out][hidden]    b2 : [L_tgt][2][E][d_out]
  wr : float32 [L_tgt][2][E][d_in]             br : [L_tgt][2][E]
  index 1 of every weight is 0 = keys, 1 = values; biases may be None.
  With dims.streams = 1 (the MoT-h activation stream) index 1 has size 1,
  src_v may be None and the returned dst_v is None.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mot_oracle.c")
_LIB = os.path.join(_HERE, "libmot_oracle.so")


def oracle_lib_path() -> str:
    return _LIB


def build_oracle(force: bool = True) -> str:
    """Compile the oracle with gcc.  IEEE semantics: no fast-math, no FMA
    contraction, so every sum is evaluated exactly as written."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", "-o", tmp, _SRC, "-lm", "-lpthread"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    return _LIB


class _Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "L_src", "L_tgt", "B", "T", "H_src", "D_src", "H_tgt", "D_tgt", "E",
        "top_k", "hidden", "src_layout", "dst_layout", "act", "streams")]


@dataclass
class OracleDims:
    L_src: int
    L_tgt: int
    B: int
    T: int
    H_src: int
    D_src: int
    H_tgt: int
    D_tgt: int
    E: int
    hidden: int
    top_k: int = 0          # 0 means "all E translators"
    src_layout: int = 0     # 0 = BTHD, 1 = BHTD
    dst_layout: int = 0
    act: int = 0            # 0 = exact-erf GELU, 1 = identity
    streams: int = 2        # 2 = keys and values; 1 = one activation stream (MoT-h)

    @property
    def d_in(self) -> int:
        return self.H_src * self.D_src

    @property
    def d_out(self) -> int:
        return self.H_tgt * self.D_tgt

    def _c(self) -> _Dims:
        return _Dims(self.L_src, self.L_tgt, self.B, self.T, self.H_src, self.D_src,
                     self.H_tgt, self.D_tgt, self.E, self.top_k or self.E, self.hidden,
                     self.src_layout, self.dst_layout, self.act, self.streams)


_lib = None


def _load():
    global _lib
    if _lib is None:
        # MOT_ORACLE_LIB: a mutated build of this oracle, used only by the
        # mutation tests to show that the pins fail on planted mistakes
        path = os.environ.get("MOT_ORACLE_LIB") or _LIB
        if path == _LIB and not os.path.exists(_LIB):
            build_oracle(force=False)
        _lib = ctypes.CDLL(path)
        _lib.mot_oracle_backbone_param_count.restype = ctypes.c_size_t
        _lib.mot_oracle_backbone_param_count.argtypes = [ctypes.c_int32] * 4
        _lib.mot_oracle_backbone_window_param_count.restype = ctypes.c_size_t
        _lib.mot_oracle_backbone_window_param_count.argtypes = [ctypes.c_int32] * 5
        for fn in (_lib.mot_oracle_translate, _lib.mot_oracle_rows,
                   _lib.mot_oracle_depth_ratio_map, _lib.mot_oracle_restore_kv,
                   _lib.mot_oracle_topS_select, _lib.mot_oracle_replay_attention,
                   _lib.mot_oracle_replay_attention_rows, _lib.mot_oracle_topS_rows,
                   _lib.mot_oracle_backbone_translate, _lib.mot_oracle_backbone_window, _lib.mot_oracle_usage,
                   _lib.mot_oracle_usage_stats):
            fn.restype = ctypes.c_int
    return _lib


def _f32(a, name):
    if a is None:
        return None
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.c_void_p)


def _threads(n):
    if n is None or n <= 0:
        n = os.cpu_count() or 1
    return int(n)


def oracle_translate(dims: OracleDims, src_k, src_v, layer_map, w1, b1, w2, b2, wr, br,
                     dst_k=None, dst_v=None, nthreads=None):
    """Full translation.  Returns (dst_k, dst_v) as float64 arrays in the
    dst layout; target layers with layer_map[j] < 0 keep the given contents
    (NaN when dst_k/dst_v are not supplied)."""
    lib = _load()
    arrs = [_f32(a, n) for a, n in ((src_k, "src_k"), (src_v, "src_v"), (w1, "w1"), (b1, "b1"),
                                    (w2, "w2"), (b2, "b2"), (wr, "wr"), (br, "br"))]
    lm = np.ascontiguousarray(layer_map, dtype=np.int32)
    shape = ((dims.L_tgt, dims.B, dims.T, dims.H_tgt, dims.D_tgt) if dims.dst_layout == 0
             else (dims.L_tgt, dims.B, dims.H_tgt, dims.T, dims.D_tgt))
    if dst_k is None:
        dst_k = np.full(shape, np.nan)
    if dst_v is None:
        dst_v = np.full(shape, np.nan)
    dst_k = np.ascontiguousarray(dst_k, dtype=np.float64)
    dst_v = np.ascontiguousarray(dst_v, dtype=np.float64)
    if dims.streams == 1:
        dst_v = None
    c = dims._c()
    rc = lib.mot_oracle_translate(*[_ptr(a) for a in arrs[:2]], _ptr(lm),
                                  *[_ptr(a) for a in arrs[2:]], _ptr(dst_k), _ptr(dst_v),
                                  ctypes.byref(c), _threads(nthreads))
    if rc != 0:
        raise ValueError("mot_oracle_translate failed with code %d" % rc)
    return dst_k, dst_v


def oracle_rows(dims: OracleDims, src_k, src_v, layer_map, w1, b1, w2, b2, wr, br,
                units, rows, nthreads=None, want_gates=False):
    """Sampled translation of the listed (j, x) units and flattened rows.
    Returns out[n_units][n_rows][d_out] (and gates[n_units][n_rows][E])."""
    lib = _load()
    arrs = [_f32(a, n) for a, n in ((src_k, "src_k"), (src_v, "src_v"), (w1, "w1"), (b1, "b1"),
                                    (w2, "w2"), (b2, "b2"), (wr, "wr"), (br, "br"))]
    lm = np.ascontiguousarray(layer_map, dtype=np.int32)
    uj = np.ascontiguousarray([u[0] for u in units], dtype=np.int32)
    ux = np.ascontiguousarray([u[1] for u in units], dtype=np.int32)
    rr = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.zeros((len(units), len(rr), dims.d_out))
    gates = np.zeros((len(units), len(rr), dims.E)) if want_gates else None
    c = dims._c()
    rc = lib.mot_oracle_rows(*[_ptr(a) for a in arrs[:2]], _ptr(lm),
                             *[_ptr(a) for a in arrs[2:]], ctypes.byref(c),
                             _ptr(uj), _ptr(ux), ctypes.c_int32(len(units)),
                             _ptr(rr), ctypes.c_int64(len(rr)), _ptr(out), _ptr(gates),
                             _threads(nthreads))
    if rc != 0:
        raise ValueError("mot_oracle_rows failed with code %d" % rc)
    return (out, gates) if want_gates else out


def oracle_depth_ratio_map(L_src: int, L_tgt: int) -> np.ndarray:
    lib = _load()
    out = np.zeros(L_tgt, dtype=np.int32)
    rc = lib.mot_oracle_depth_ratio_map(ctypes.c_int32(L_src), ctypes.c_int32(L_tgt), _ptr(out))
    if rc != 0:
        raise ValueError("mot_oracle_depth_ratio_map failed with code %d" % rc)
    return out


def oracle_restore_kv(act, layer_map, wk, bk, wv, bv, B, T, H_tgt, D_tgt, dst_layout=0,
                      dst_k=None, dst_v=None):
    """MoT-h key/value restoration (App. C.5): K = W^K a + b^K, V = W^V a + b^V
    per restored layer.  act [L][B][T][d_act]; wk, wv [L][d_kv][d_act];
    bk, bv [L][d_kv] or None; layer_map int[L] or None (every layer).
    Returns (dst_k, dst_v) as float64 in the dst layout; layers that are not
    restored keep the given contents (NaN when dst_k/dst_v are not supplied)."""
    lib = _load()
    act = _f32(act, "act")
    L, d_act = act.shape[0], act.shape[-1]
    arrs = [_f32(a, n) for a, n in ((wk, "wk"), (bk, "bk"), (wv, "wv"), (bv, "bv"))]
    lm = None if layer_map is None else np.ascontiguousarray(layer_map, dtype=np.int32)
    shape = (L, B, T, H_tgt, D_tgt) if dst_layout == 0 else (L, B, H_tgt, T, D_tgt)
    dst_k = np.full(shape, np.nan) if dst_k is None else np.array(dst_k, dtype=np.float64)
    dst_v = np.full(shape, np.nan) if dst_v is None else np.array(dst_v, dtype=np.float64)
    i32 = ctypes.c_int32
    rc = lib.mot_oracle_restore_kv(_ptr(act), _ptr(lm), *[_ptr(a) for a in arrs],
                                   _ptr(dst_k), _ptr(dst_v), i32(L), i32(B), i32(T), i32(d_act),
                                   i32(H_tgt), i32(D_tgt), i32(dst_layout))
    if rc != 0:
        raise ValueError("mot_oracle_restore_kv failed with code %d" % rc)
    return dst_k, dst_v


def oracle_topS_select(A, S: int) -> np.ndarray:
    """Top-S source-guided key sets (App. C.4): A [B][T][T] head-averaged
    source attention; returns int32 [B][T][S], each row the S positions
    v <= u with the largest A[b][u][v] (ties: lower v), ascending, padded -1."""
    lib = _load()
    A = _f32(A, "A")
    B, T = A.shape[0], A.shape[1]
    idx = np.zeros((B, T, S), dtype=np.int32)
    rc = lib.mot_oracle_topS_select(_ptr(A), ctypes.c_int32(B), ctypes.c_int32(T), ctypes.c_int32(S),
                                    _ptr(idx))
    if rc != 0:
        raise ValueError("mot_oracle_topS_select failed with code %d" % rc)
    return idx


def oracle_replay_attention(q, k, v, idx=None, kv_layout: int = 0) -> np.ndarray:
    """Replay attention of one target layer over the key sets idx [B][T][S]
    (-1 padded), or the full causal set when idx is None (App. C.4).
    q [B][T][H_q][D]; k, v [B][T][H_kv][D] (kv_layout 0) or [B][H_kv][T][D] (1).
    Returns float64 [B][T][H_q][D]."""
    lib = _load()
    q = _f32(q, "q"); k = _f32(k, "k"); v = _f32(v, "v")
    B, T, H_q, D = q.shape
    H_kv = k.shape[2] if kv_layout == 0 else k.shape[1]
    S = 0
    if idx is not None:
        idx = np.ascontiguousarray(idx, dtype=np.int32)
        S = idx.shape[2]
    o = np.zeros((B, T, H_q, D))
    i32 = ctypes.c_int32
    rc = lib.mot_oracle_replay_attention(_ptr(q), _ptr(k), _ptr(v), _ptr(idx), _ptr(o), i32(B), i32(T),
                                         i32(H_q), i32(H_kv), i32(D), i32(S), i32(kv_layout))
    if rc != 0:
        raise ValueError("mot_oracle_replay_attention failed with code %d" % rc)
    return o


def oracle_topS_rows(A, S: int, rows) -> np.ndarray:
    """Top-S sets of the listed (b, u) rows only: int32 [n][S]."""
    lib = _load()
    A = _f32(A, "A")
    B, T = A.shape[0], A.shape[1]
    rb = np.ascontiguousarray([r[0] for r in rows], dtype=np.int32)
    ru = np.ascontiguousarray([r[1] for r in rows], dtype=np.int32)
    out = np.zeros((len(rows), S), dtype=np.int32)
    i32 = ctypes.c_int32
    rc = lib.mot_oracle_topS_rows(_ptr(A), i32(B), i32(T), i32(S), _ptr(rb), _ptr(ru), i32(len(rows)), _ptr(out))
    if rc != 0:
        raise ValueError("mot_oracle_topS_rows failed with code %d" % rc)
    return out


def oracle_replay_attention_rows(q, k, v, idx, rows, kv_layout: int = 0) -> np.ndarray:
    """oracle_replay_attention for the listed (b, u) rows only: float64 [n][H_q][D]."""
    lib = _load()
    q = _f32(q, "q"); k = _f32(k, "k"); v = _f32(v, "v")
    B, T, H_q, D = q.shape
    H_kv = k.shape[2] if kv_layout == 0 else k.shape[1]
    S = 0
    if idx is not None:
        idx = np.ascontiguousarray(idx, dtype=np.int32)
        S = idx.shape[2]
    rb = np.ascontiguousarray([r[0] for r in rows], dtype=np.int32)
    ru = np.ascontiguousarray([r[1] for r in rows], dtype=np.int32)
    out = np.zeros((len(rows), H_q, D))
    i32 = ctypes.c_int32
    rc = lib.mot_oracle_replay_attention_rows(_ptr(q), _ptr(k), _ptr(v), _ptr(idx), i32(B), i32(T), i32(H_q),
                                              i32(H_kv), i32(D), i32(S), i32(kv_layout), _ptr(rb), _ptr(ru),
                                              i32(len(rows)), _ptr(out))
    if rc != 0:
        raise ValueError("mot_oracle_replay_attention_rows failed with code %d" % rc)
    return out


def oracle_backbone_param_count(d_in: int, d_h: int, d_ff: int, d_out: int) -> int:
    """Parameters per (unit, expert) of the backbone translator body."""
    return int(_load().mot_oracle_backbone_param_count(d_in, d_h, d_ff, d_out))


def oracle_backbone_translate(dims: OracleDims, src_k, src_v, layer_map, params, wr, br,
                              d_h: int, n_heads: int, d_ff: int):
    """Mixture of backbone translators (App. C.2, one channel-window slot per
    unit): params float32 [L_tgt][2][E][P] packed as documented in
    mot_oracle.c.  Returns (dst_k, dst_v) float64 in the dst layout (NaN in
    layers with layer_map[j] < 0)."""
    lib = _load()
    arrs = [_f32(a, n) for a, n in ((src_k, "src_k"), (src_v, "src_v"), (params, "params"), (wr, "wr"),
                                    (br, "br"))]
    lm = np.ascontiguousarray(layer_map, dtype=np.int32)
    shape = ((dims.L_tgt, dims.B, dims.T, dims.H_tgt, dims.D_tgt) if dims.dst_layout == 0
             else (dims.L_tgt, dims.B, dims.H_tgt, dims.T, dims.D_tgt))
    dst_k = np.full(shape, np.nan)
    dst_v = np.full(shape, np.nan)
    c = dims._c()
    i32 = ctypes.c_int32
    rc = lib.mot_oracle_backbone_translate(_ptr(arrs[0]), _ptr(arrs[1]), _ptr(lm), _ptr(arrs[2]), _ptr(arrs[3]),
                                           _ptr(arrs[4]), _ptr(dst_k), _ptr(dst_v), ctypes.byref(c),
                                           i32(d_h), i32(n_heads), i32(d_ff))
    if rc != 0:
        raise ValueError("mot_oracle_backbone_translate failed with code %d" % rc)
    return dst_k, dst_v


def oracle_usage(dims: OracleDims, src_k, src_v, layer_map, wr, br) -> np.ndarray:
    """Translator selection counts per unit (paper Sec. 4, "MoT Architecture
    Ablation"): int64 [L_tgt][streams][E]; units of unmapped layers stay 0."""
    lib = _load()
    arrs = [_f32(a, n) for a, n in ((src_k, "src_k"), (src_v, "src_v"), (wr, "wr"), (br, "br"))]
    lm = np.ascontiguousarray(layer_map, dtype=np.int32)
    counts = np.zeros((dims.L_tgt, dims.streams, dims.E), np.int64)
    c = dims._c()
    rc = lib.mot_oracle_usage(_ptr(arrs[0]), _ptr(arrs[1]), _ptr(lm), _ptr(arrs[2]), _ptr(arrs[3]),
                              ctypes.byref(c), _ptr(counts))
    if rc != 0:
        raise ValueError("mot_oracle_usage failed with code %d" % rc)
    return counts


def oracle_usage_stats(counts) -> tuple:
    """(CV^2, entropy) of one unit's counts I[0..E): population variance over
    the squared mean, and -sum p ln p with p = I / sum I."""
    lib = _load()
    cnt = np.ascontiguousarray(counts, dtype=np.int64).ravel()
    cv2, ent = ctypes.c_double(), ctypes.c_double()
    rc = lib.mot_oracle_usage_stats(_ptr(cnt), ctypes.c_int32(cnt.size), ctypes.byref(cv2), ctypes.byref(ent))
    if rc != 0:
        raise ValueError("mot_oracle_usage_stats failed with code %d" % rc)
    return cv2.value, ent.value


def oracle_backbone_window_param_count(d_in: int, d_h: int, d_ff: int, d_out: int, n_slots: int) -> int:
    """Parameters per (window, X, expert) of the backbone body over a window
    of n_slots channel slots (shared input projection, one cross-attention
    block per slot, output projection of the concatenation)."""
    return int(_load().mot_oracle_backbone_window_param_count(d_in, d_h, d_ff, d_out, n_slots))


def oracle_backbone_window(dims: OracleDims, src_k, src_v, layer_map, params, wr, br, d_h: int, n_heads: int,
                           d_ff: int, n_slots: int):
    """Mixture of backbone translators over channel windows of n_slots slots
    (App. C.2): window w covers target layers w*N .. w*N+N-1, slot r reads
    source layer layer_map[w*N + r]; params float32 [L_tgt/N][2][E][P]; router
    weights [L_tgt/N][2][E][N*d_in], bias [L_tgt/N][2][E].  Returns (dst_k,
    dst_v) float64 in the dst layout (NaN in skipped windows)."""
    lib = _load()
    arrs = [_f32(a, n) for a, n in ((src_k, "src_k"), (src_v, "src_v"), (params, "params"), (wr, "wr"),
                                    (br, "br"))]
    lm = np.ascontiguousarray(layer_map, dtype=np.int32)
    shape = ((dims.L_tgt, dims.B, dims.T, dims.H_tgt, dims.D_tgt) if dims.dst_layout == 0
             else (dims.L_tgt, dims.B, dims.H_tgt, dims.T, dims.D_tgt))
    dst_k = np.full(shape, np.nan)
    dst_v = np.full(shape, np.nan)
    c = dims._c()
    i32 = ctypes.c_int32
    rc = lib.mot_oracle_backbone_window(_ptr(arrs[0]), _ptr(arrs[1]), _ptr(lm), _ptr(arrs[2]), _ptr(arrs[3]),
                                        _ptr(arrs[4]), _ptr(dst_k), _ptr(dst_v), ctypes.byref(c), i32(d_h),
                                        i32(n_heads), i32(d_ff), i32(n_slots))
    if rc != 0:
        raise ValueError("mot_oracle_backbone_window failed with code %d" % rc)
    return dst_k, dst_v
