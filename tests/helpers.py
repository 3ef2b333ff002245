"""Shared test plumbing: device upload, GPU calls through the C ABI, oracle
calls, and the per-unit relative Frobenius error."""
from __future__ import annotations

import numpy as np

from paper_2607_28979_amd import binding as mb
from paper_2607_28979_amd.inputs import Inputs, bf16_bits

SENTINEL = -3.75   # exactly representable in bf16 and fp32

TOL = {"f32": 1e-5, "bf16": 2e-2}


def to_dev(a: np.ndarray, dtype: str):
    import torch
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    bits = bf16_bits(a)
    return torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16)


def dst_shape(w):
    if w.dst_layout == 0:
        return (w.L_tgt, w.B, w.T, w.H_tgt, w.D_tgt)
    return (w.L_tgt, w.B, w.H_tgt, w.T, w.D_tgt)


def run_gpu(w, inp: Inputs, layer_map, algo=mb.ALGO_AUTO, act=mb.ACT_GELU, with_bias=True,
            dev=None):
    """Translate on the GPU through the C ABI; returns (dst_k, dst_v) as
    float64 numpy arrays in the dst layout (unmapped layers hold SENTINEL)."""
    import torch
    d = dev or {}
    if not d:
        for name in ("src_k", "src_v", "w1", "b1", "w2", "b2", "wr", "br"):
            d[name] = to_dev(getattr(inp, name), w.dtype)
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    dk = torch.full(dst_shape(w), SENTINEL, dtype=tdt, device="cuda")
    dv = torch.full(dst_shape(w), SENTINEL, dtype=tdt, device="cuda")
    shapes = mb.Shapes.from_workload(w, algo=algo, act=act)
    mb.translate(d["src_k"], d["src_v"], layer_map, d["w1"], d["b1"] if with_bias else None,
                 d["w2"], d["b2"] if with_bias else None, d["wr"], d["br"] if with_bias else None,
                 dk, dv, shapes)
    torch.cuda.synchronize()
    return dk.float().cpu().numpy().astype(np.float64), dv.float().cpu().numpy().astype(np.float64)


def oracle_dims(w, act=0):
    from oracle import OracleDims
    return OracleDims(L_src=w.L_src, L_tgt=w.L_tgt, B=w.B, T=w.T, H_src=w.H_src, D_src=w.D_src,
                      H_tgt=w.H_tgt, D_tgt=w.D_tgt, E=w.E, hidden=w.hidden,
                      src_layout=w.src_layout, dst_layout=w.dst_layout, act=act,
                      top_k=w.top_k, streams=w.streams)


def unit_rows(dst, w, j):
    """Target layer j of a dst array as [B*T][d_out] (layout-aware)."""
    a = dst[j]
    if w.dst_layout == 1:
        a = a.transpose(0, 2, 1, 3)
    return a.reshape(w.B * w.T, w.d_out)


def rel_frob(got: np.ndarray, ref: np.ndarray) -> float:
    num = np.linalg.norm((got - ref).ravel())
    den = np.linalg.norm(ref.ravel())
    return float(num / den) if den > 0 else float(num)


def max_unit_error(gpu_k, gpu_v, ref_k, ref_v, w, layer_map):
    worst = 0.0
    for j in range(w.L_tgt):
        if layer_map[j] < 0:
            continue
        for g, r in ((gpu_k, ref_k), (gpu_v, ref_v)):
            worst = max(worst, rel_frob(unit_rows(g, w, j), unit_rows(r, w, j)))
    return worst
