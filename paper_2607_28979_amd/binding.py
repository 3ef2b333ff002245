"""Thin ctypes binding of libmot (argument marshalling only).

Every step of the translation runs in the HIP kernels of ``csrc/libmot.so``.
This module turns torch tensors into device pointers and the current torch
stream into a ``hipStream_t``; it has no compute path of its own and raises
``MotError`` when the library is missing or a call fails.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(HERE, "csrc", "libmot.so")

MOT_F32, MOT_BF16 = 0, 1
LAYOUT_BTHD, LAYOUT_BHTD = 0, 1
ACT_GELU, ACT_IDENTITY = 0, 1
ALGO_AUTO, ALGO_UNFUSED, ALGO_FUSED, ALGO_ROUTED = 0, 1, 2, 3

STATUS = {0: "MOT_OK", 1: "MOT_ERR_NULL_ARG", 2: "MOT_ERR_BAD_SHAPE", 3: "MOT_ERR_BAD_LAYER_MAP",
          4: "MOT_ERR_UNSUPPORTED", 5: "MOT_ERR_MISALIGNED", 6: "MOT_ERR_WORKSPACE_TOO_SMALL",
          7: "MOT_ERR_HIP"}

EXPORTED = ("mot_translate", "mot_workspace_bytes", "mot_depth_ratio_map", "mot_status_string",
            "mot_last_error", "mot_abi_version", "mot_restore_kv", "mot_topS_select",
            "mot_replay_attention", "mot_backbone_param_count", "mot_backbone_translate",
            "mot_usage_stats", "mot_replay_workspace_bytes", "mot_backbone_workspace_bytes",
            "mot_replay_attention_noalloc")


class MotError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        self.name = STATUS.get(status, "MOT_ERR_%d" % status)
        super().__init__("%s: %s" % (self.name, detail))


class _Shapes(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "L_src", "L_tgt", "B", "T", "H_src", "D_src", "H_tgt", "D_tgt", "E", "top_k", "hidden",
        "dtype", "src_layout", "dst_layout", "act", "algo", "streams")] + [
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t), ("usage", ctypes.c_void_p)]


class _RestoreShapes(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("L", "B", "T", "d_act", "H_tgt", "D_tgt", "dtype",
                                             "dst_layout")]


class _BackboneDims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("d_h", "n_heads", "d_ff", "n_slots")]


class _ReplayShapes(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("B", "T", "H_q", "H_kv", "D", "S", "kv_layout")] + [
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t)]


class _TW(ctypes.Structure):
    _fields_ = [("w1", ctypes.c_void_p), ("b1", ctypes.c_void_p), ("w2", ctypes.c_void_p),
                ("b2", ctypes.c_void_p)]


class _RW(ctypes.Structure):
    _fields_ = [("w", ctypes.c_void_p), ("b", ctypes.c_void_p)]


@dataclass
class Shapes:
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
    dtype: int = MOT_BF16
    top_k: int = 0            # 0 = E
    src_layout: int = LAYOUT_BTHD
    dst_layout: int = LAYOUT_BTHD
    act: int = ACT_GELU
    algo: int = ALGO_AUTO
    streams: int = 2          # 2 = keys and values; 1 = one activation stream (MoT-h)

    def c(self, workspace=None, workspace_bytes=0, usage=None) -> _Shapes:
        return _Shapes(self.L_src, self.L_tgt, self.B, self.T, self.H_src, self.D_src, self.H_tgt,
                       self.D_tgt, self.E, self.top_k or self.E, self.hidden, self.dtype,
                       self.src_layout, self.dst_layout, self.act, self.algo, self.streams,
                       workspace, workspace_bytes, usage)

    @classmethod
    def from_workload(cls, w, **kw) -> "Shapes":
        return cls(w.L_src, w.L_tgt, w.B, w.T, w.H_src, w.D_src, w.H_tgt, w.D_tgt, w.E, w.hidden,
                   dtype=MOT_F32 if w.dtype == "f32" else MOT_BF16, src_layout=w.src_layout,
                   dst_layout=w.dst_layout, **{"top_k": w.top_k, "streams": w.streams, **kw})


_lib = None


def lib_path() -> str:
    return _LIB_PATH


def _hip_runtimes() -> set:
    """Distinct files of the HIP runtime mapped into this process (Linux)."""
    try:
        with open("/proc/self/maps") as f:
            return {os.path.realpath(ln.split()[-1]) for ln in f
                    if "libamdhip64.so" in ln and ln.split()[-1].startswith("/")}
    except OSError:
        return set()


def load_library():
    """Load libmot.so; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise MotError(-1, "libmot.so not found at %s; build it with "
                               "`python -m paper_2607_28979_amd.build`" % _LIB_PATH)
        # PyTorch for ROCm ships its own HIP runtime.  Loading torch first lets
        # libmot bind to that same runtime (the dynamic linker matches its
        # soname), so streams and device pointers from torch are valid here;
        # loading libmot first would bring a second, separate runtime into
        # the process.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        lib = ctypes.CDLL(_LIB_PATH)
        runtimes = _hip_runtimes()
        if len(runtimes) > 1:
            raise MotError(-1, "two HIP runtimes are loaded in this process (%s); import torch "
                               "before loading libmot" % ", ".join(sorted(runtimes)))
        lib.mot_translate.restype = ctypes.c_int
        lib.mot_translate.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.POINTER(_TW), ctypes.POINTER(_RW), ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.POINTER(_Shapes), ctypes.c_void_p]
        lib.mot_workspace_bytes.restype = ctypes.c_size_t
        lib.mot_workspace_bytes.argtypes = [ctypes.POINTER(_Shapes)]
        lib.mot_depth_ratio_map.restype = ctypes.c_int
        lib.mot_depth_ratio_map.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]
        lib.mot_status_string.restype = ctypes.c_char_p
        lib.mot_status_string.argtypes = [ctypes.c_int]
        lib.mot_last_error.restype = ctypes.c_char_p
        lib.mot_abi_version.restype = ctypes.c_int
        lib.mot_restore_kv.restype = ctypes.c_int
        lib.mot_restore_kv.argtypes = [ctypes.c_void_p] * 8 + [ctypes.POINTER(_RestoreShapes),
                                                               ctypes.c_void_p]
        lib.mot_topS_select.restype = ctypes.c_int
        lib.mot_topS_select.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(_ReplayShapes),
                                        ctypes.c_void_p]
        lib.mot_backbone_param_count.restype = ctypes.c_size_t
        lib.mot_backbone_param_count.argtypes = [ctypes.POINTER(_Shapes), ctypes.POINTER(_BackboneDims)]
        lib.mot_backbone_translate.restype = ctypes.c_int
        lib.mot_backbone_translate.argtypes = [ctypes.c_void_p] * 4 + [ctypes.POINTER(_RW), ctypes.c_void_p,
                                                                       ctypes.c_void_p, ctypes.POINTER(_Shapes),
                                                                       ctypes.POINTER(_BackboneDims), ctypes.c_void_p]
        lib.mot_replay_workspace_bytes.restype = ctypes.c_size_t
        lib.mot_replay_workspace_bytes.argtypes = [ctypes.POINTER(_ReplayShapes), ctypes.c_int]
        lib.mot_backbone_workspace_bytes.restype = ctypes.c_size_t
        lib.mot_backbone_workspace_bytes.argtypes = [ctypes.POINTER(_Shapes), ctypes.POINTER(_BackboneDims)]
        lib.mot_usage_stats.restype = ctypes.c_int
        lib.mot_usage_stats.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p]
        for fn in (lib.mot_replay_attention, lib.mot_replay_attention_noalloc):
            fn.restype = ctypes.c_int
            fn.argtypes = [ctypes.c_void_p] * 5 + [ctypes.POINTER(_ReplayShapes), ctypes.c_void_p]
        _lib = lib
    return _lib


def abi_version() -> int:
    return load_library().mot_abi_version()


def status_string(status: int) -> str:
    return load_library().mot_status_string(status).decode()


def _check(rc: int):
    if rc != 0:
        raise MotError(rc, load_library().mot_last_error().decode())


def depth_ratio_map(L_src: int, L_tgt: int):
    import numpy as np
    out = np.zeros(L_tgt, dtype=np.int32)
    _check(load_library().mot_depth_ratio_map(L_src, L_tgt, out.ctypes.data))
    return out


def workspace_bytes(shapes: Shapes) -> int:
    c = shapes.c()
    n = load_library().mot_workspace_bytes(ctypes.byref(c))
    if n == ctypes.c_size_t(-1).value:
        raise MotError(2, load_library().mot_last_error().decode())
    return int(n)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def translate_raw(src_k, src_v, layer_map, w1, b1, w2, b2, wr, br, dst_k, dst_v,
                  shapes: Shapes, stream=None, workspace=None, workspace_bytes_=0, usage=None) -> None:
    """Call mot_translate with raw device addresses (ints) or tensors.  No
    checks beyond the library's own (used by the ABI validation tests)."""
    import numpy as np
    lib = load_library()
    lm = np.ascontiguousarray(layer_map, dtype=np.int32)
    tw = _TW(_ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2))
    rw = _RW(_ptr(wr), _ptr(br))
    c = shapes.c(_ptr(workspace), workspace_bytes_, _ptr(usage))
    _check(lib.mot_translate(_ptr(src_k), _ptr(src_v), lm.ctypes.data if lm.size else None,
                             ctypes.byref(tw), ctypes.byref(rw), _ptr(dst_k), _ptr(dst_v),
                             ctypes.byref(c), stream))


def translate(src_k, src_v, layer_map: Sequence[int], w1, b1, w2, b2, wr, br, dst_k, dst_v,
              shapes: Shapes, workspace=None, usage=None) -> None:
    """Translate on the current torch stream.  Tensors must live on the
    current HIP device, be contiguous and have the dtype named by
    ``shapes.dtype`` (torch.float32 or torch.bfloat16).  ``usage``: optional
    int32 tensor [L_tgt][streams][E] of translator selection counts that the
    call adds to (the library treats it as uint32)."""
    import torch
    want = torch.float32 if shapes.dtype == MOT_F32 else torch.bfloat16
    dev = torch.device("cuda", torch.cuda.current_device())
    for name, t in (("src_k", src_k), ("src_v", src_v), ("w1", w1), ("b1", b1), ("w2", w2),
                    ("b2", b2), ("wr", wr), ("br", br), ("dst_k", dst_k), ("dst_v", dst_v)):
        if t is None:
            continue
        if t.device != dev:
            raise MotError(1, "%s is on %s, expected %s" % (name, t.device, dev))
        if t.dtype != want:
            raise MotError(2, "%s has dtype %s, expected %s" % (name, t.dtype, want))
        if not t.is_contiguous():
            raise MotError(2, "%s is not contiguous" % name)
    ws_bytes = 0
    if workspace is not None:
        ws_bytes = workspace.numel() * workspace.element_size()
    if usage is not None and (usage.device != dev or usage.dtype != torch.int32 or not usage.is_contiguous()):
        raise MotError(2, "usage must be a contiguous int32 tensor on %s" % dev)
    stream = torch.cuda.current_stream().cuda_stream
    translate_raw(src_k, src_v, layer_map, w1, b1, w2, b2, wr, br, dst_k, dst_v, shapes,
                  stream=stream, workspace=workspace, workspace_bytes_=ws_bytes, usage=usage)


def usage_stats(counts, cv2, entropy) -> None:
    """mot_usage_stats on the current torch stream: counts int32 [n][E]
    (read as uint32), cv2 and entropy float64 [n] (outputs)."""
    import torch
    for name, t, dt in (("counts", counts, torch.int32), ("cv2", cv2, torch.float64),
                        ("entropy", entropy, torch.float64)):
        if t.dtype != dt or not t.is_contiguous():
            raise MotError(2, "%s must be a contiguous %s tensor" % (name, dt))
    n, E = counts.shape
    _check(load_library().mot_usage_stats(_ptr(counts), n, E, _ptr(cv2), _ptr(entropy),
                                          torch.cuda.current_stream().cuda_stream))


def restore_kv(act, layer_map, wk, bk, wv, bv, dst_k, dst_v, L: int, B: int, T: int, d_act: int,
               H_tgt: int, D_tgt: int, dst_layout: int = LAYOUT_BTHD) -> None:
    """mot_restore_kv on the current torch stream (bf16 tensors on the
    current device): K = W^K a + b^K and V = W^V a + b^V for every layer with
    layer_map[l] >= 0 (layer_map None = all layers)."""
    import numpy as np
    import torch
    lib = load_library()
    for name, t in (("act", act), ("wk", wk), ("bk", bk), ("wv", wv), ("bv", bv), ("dst_k", dst_k),
                    ("dst_v", dst_v)):
        if t is not None and (t.dtype != torch.bfloat16 or not t.is_contiguous()):
            raise MotError(2, "%s must be a contiguous bfloat16 tensor" % name)
    lm = None if layer_map is None else np.ascontiguousarray(layer_map, dtype=np.int32)
    c = _RestoreShapes(L, B, T, d_act, H_tgt, D_tgt, MOT_BF16, dst_layout)
    stream = torch.cuda.current_stream().cuda_stream
    _check(lib.mot_restore_kv(_ptr(act), lm.ctypes.data if lm is not None else None, _ptr(wk),
                              _ptr(bk), _ptr(wv), _ptr(bv), _ptr(dst_k), _ptr(dst_v),
                              ctypes.byref(c), stream))


def topS_select(A, idx, B: int, T: int, S: int) -> None:
    """mot_topS_select on the current torch stream: A fp32 [B][T][T] (head-
    averaged source attention), idx int32 [B][T][S] (output)."""
    import torch
    lib = load_library()
    for name, t, dt in (("A", A, torch.float32), ("idx", idx, torch.int32)):
        if t is not None and (t.dtype != dt or not t.is_contiguous()):
            raise MotError(2, "%s must be a contiguous %s tensor" % (name, dt))
    c = _ReplayShapes(B, T, 1, 1, 128, S, LAYOUT_BTHD)
    _check(lib.mot_topS_select(_ptr(A), _ptr(idx), ctypes.byref(c),
                               torch.cuda.current_stream().cuda_stream))


def replay_workspace_bytes(B: int, T: int, H_q: int, H_kv: int, D: int, S: int = 0, with_sets: bool = False) -> int:
    c = _ReplayShapes(B, T, H_q, H_kv, D, S, LAYOUT_BTHD)
    n = load_library().mot_replay_workspace_bytes(ctypes.byref(c), int(with_sets))
    if n == ctypes.c_size_t(-1).value:
        raise MotError(2, load_library().mot_last_error().decode())
    return int(n)


def replay_attention(q, k, v, idx, o, B: int, T: int, H_q: int, H_kv: int, D: int, S: int = 0,
                     kv_layout: int = LAYOUT_BTHD, workspace=None) -> None:
    """mot_replay_attention on the current torch stream (bf16 q, k, v, o;
    int32 idx [B][T][S], or None for the full causal set; optional device
    workspace tensor for the full causal set's staging)."""
    import torch
    lib = load_library()
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o)):
        if t.dtype != torch.bfloat16 or not t.is_contiguous():
            raise MotError(2, "%s must be a contiguous bfloat16 tensor" % name)
    if idx is not None and (idx.dtype != torch.int32 or not idx.is_contiguous()):
        raise MotError(2, "idx must be a contiguous int32 tensor")
    c = _ReplayShapes(B, T, H_q, H_kv, D, S if idx is not None else 0, kv_layout, _ptr(workspace),
                      workspace.numel() * workspace.element_size() if workspace is not None else 0)
    _check(lib.mot_replay_attention(_ptr(q), _ptr(k), _ptr(v), _ptr(idx), _ptr(o), ctypes.byref(c),
                                    torch.cuda.current_stream().cuda_stream))


def replay_attention_noalloc(q, k, v, idx, o, B: int, T: int, H_q: int, H_kv: int, D: int, S: int = 0,
                             kv_layout: int = LAYOUT_BTHD) -> None:
    """mot_replay_attention_noalloc on the current torch stream: the same
    operation as replay_attention, with the full causal path's staging in the
    library's static per-device scratch (no allocation)."""
    import torch
    lib = load_library()
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o)):
        if t.dtype != torch.bfloat16 or not t.is_contiguous():
            raise MotError(2, "%s must be a contiguous bfloat16 tensor" % name)
    if idx is not None and (idx.dtype != torch.int32 or not idx.is_contiguous()):
        raise MotError(2, "idx must be a contiguous int32 tensor")
    c = _ReplayShapes(B, T, H_q, H_kv, D, S if idx is not None else 0, kv_layout)
    _check(lib.mot_replay_attention_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(idx), _ptr(o), ctypes.byref(c),
                                            torch.cuda.current_stream().cuda_stream))


def backbone_param_count(shapes: Shapes, d_h: int, n_heads: int, d_ff: int, n_slots: int = 1) -> int:
    """Elements per expert of the packed backbone parameters."""
    c = shapes.c()
    return int(load_library().mot_backbone_param_count(ctypes.byref(c),
                                                       ctypes.byref(_BackboneDims(d_h, n_heads, d_ff, n_slots))))


def backbone_workspace_bytes(shapes: Shapes, d_h: int, n_heads: int, d_ff: int, n_slots: int = 1) -> int:
    c = shapes.c()
    n = load_library().mot_backbone_workspace_bytes(ctypes.byref(c),
                                                    ctypes.byref(_BackboneDims(d_h, n_heads, d_ff, n_slots)))
    if n == ctypes.c_size_t(-1).value:
        raise MotError(2, load_library().mot_last_error().decode())
    return int(n)


def backbone_translate(src_k, src_v, layer_map, params, wr, br, dst_k, dst_v, shapes: Shapes, d_h: int,
                       n_heads: int, d_ff: int, usage=None, workspace=None, n_slots: int = 1) -> None:
    """mot_backbone_translate on the current torch stream (bf16 tensors)."""
    import numpy as np
    import torch
    lib = load_library()
    for name, t in (("src_k", src_k), ("src_v", src_v), ("params", params), ("wr", wr), ("br", br),
                    ("dst_k", dst_k), ("dst_v", dst_v)):
        if t is not None and (t.dtype != torch.bfloat16 or not t.is_contiguous()):
            raise MotError(2, "%s must be a contiguous bfloat16 tensor" % name)
    lm = np.ascontiguousarray(layer_map, dtype=np.int32)
    rw = _RW(_ptr(wr), _ptr(br))
    c = shapes.c(_ptr(workspace), workspace.numel() * workspace.element_size() if workspace is not None else 0,
                 _ptr(usage))
    _check(lib.mot_backbone_translate(_ptr(src_k), _ptr(src_v), lm.ctypes.data, _ptr(params), ctypes.byref(rw),
                                      _ptr(dst_k), _ptr(dst_v), ctypes.byref(c),
                                      ctypes.byref(_BackboneDims(d_h, n_heads, d_ff, n_slots)),
                                      torch.cuda.current_stream().cuda_stream))
