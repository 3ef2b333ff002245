"""Seeded synthetic inputs for the KV-cache translation workloads.

This module only draws random numbers and rounds them to the storage type.
It holds none of the translation arithmetic; both the GPU library's callers
and the CPU oracle receive exactly the arrays produced here.

Draw order (numpy ``Generator(PCG64(seed))``), all float32:
  1. source keys   [L_src][B][T][H_src][D_src] ~ N(0, 1)
  2. source values  same shape                 ~ N(0, 1)
  3. key channel scales   [L_src][d_in] = exp(key_sigma * N(0,1))   (if key_sigma > 0)
  4. value channel scales [L_src][d_in] = exp(val_sigma * N(0,1))   (if val_sigma > 0)
  5. key outlier rows: for each batch row b, ceil(frac*T) positions = {0} plus
     ceil(frac*T)-1 positions drawn without replacement from 1..T-1; the same
     positions in every layer; those key rows are multiplied by key_outlier_mult
  6. weights, for j = 0..L_tgt-1, x = keys, values:
       router W [E][d_in]  Xavier-uniform  U(+-sqrt(6/(d_in+E)))
       router b [E]        U(+-1/sqrt(d_in))
       for m = 0..E-1:
         W1 [hidden][d_in]  Xavier-uniform U(+-sqrt(6/(d_in+hidden)))
         b1 [hidden]        U(+-1/sqrt(d_in))
         W2 [d_out][hidden] Xavier-uniform U(+-sqrt(6/(hidden+d_out)))
         b2 [d_out]         U(+-1/sqrt(hidden))
Then, for bf16 workloads, every array is rounded to bfloat16 (round to
nearest even) and returned widened back to float32 (exact).
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional

import numpy as np

from .configs import Workload


@dataclass
class Inputs:
    src_k: np.ndarray      # float32, layout per workload.src_layout
    src_v: Optional[np.ndarray]   # None for a single activation stream
    w1: np.ndarray         # [L_tgt][2][E][hidden][d_in]
    b1: np.ndarray         # [L_tgt][2][E][hidden]
    w2: np.ndarray         # [L_tgt][2][E][d_out][hidden]
    b2: np.ndarray         # [L_tgt][2][E][d_out]
    wr: np.ndarray         # [L_tgt][2][E][d_in]
    br: np.ndarray         # [L_tgt][2][E]
    dtype: str             # "f32" or "bf16": the storage type the values fit


def round_to_bf16(a: np.ndarray, chunk: int = 1 << 24) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), in place;
    returns the array (still float32, now exactly bf16-representable)."""
    flat = a.reshape(-1)
    u = flat.view(np.uint32)
    for s in range(0, u.size, chunk):
        blk = u[s:s + chunk].astype(np.uint64)
        blk = (blk + 0x7FFF + ((blk >> 16) & 1)) >> 16
        u[s:s + chunk] = (blk << 16).astype(np.uint32)
    return a


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of a float32 array whose values are exactly
    bf16-representable (as produced by ``round_to_bf16``)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("array holds values that are not bf16-representable")
    return (u >> 16).astype(np.uint16)


def _uniform(rng: np.random.Generator, out: np.ndarray, bound: float) -> None:
    rng.random(out=out, dtype=np.float32)
    out *= np.float32(2.0 * bound)
    out -= np.float32(bound)


def generate(w: Workload, with_bias: bool = True, streams: Optional[int] = None) -> Inputs:
    """streams (default: the workload's) = 1 draws only the key-side arrays
    (the one activation stream of the MoT-h variant): src_v is None, weights
    have size 1 on axis 1, and the value-side draws (items 2 and 4, the
    x = values weights) are skipped."""
    streams = streams or w.streams
    rng = np.random.Generator(np.random.PCG64(w.seed))
    shp = (w.L_src, w.B, w.T, w.H_src, w.D_src)
    src_k = rng.standard_normal(shp, dtype=np.float32)
    src_v = rng.standard_normal(shp, dtype=np.float32) if streams == 2 else None
    d_in, d_out, E, Hd = w.d_in, w.d_out, w.E, w.hidden
    if w.key_sigma > 0:
        s = np.exp(np.float32(w.key_sigma) * rng.standard_normal((w.L_src, d_in), dtype=np.float32))
        src_k *= s.reshape(w.L_src, 1, 1, w.H_src, w.D_src)
    if w.val_sigma > 0 and streams == 2:
        s = np.exp(np.float32(w.val_sigma) * rng.standard_normal((w.L_src, d_in), dtype=np.float32))
        src_v *= s.reshape(w.L_src, 1, 1, w.H_src, w.D_src)
    if w.key_outlier_frac > 0 and w.T > 0:
        n_out = int(math.ceil(w.key_outlier_frac * w.T))
        for b in range(w.B):
            rest = rng.choice(np.arange(1, w.T), size=max(0, min(n_out - 1, w.T - 1)), replace=False)
            pos = np.concatenate([[0], np.sort(rest)]).astype(np.int64)
            src_k[:, b, pos] *= np.float32(w.key_outlier_mult)

    L = w.L_tgt
    w1 = np.empty((L, streams, E, Hd, d_in), np.float32)
    b1 = np.empty((L, streams, E, Hd), np.float32)
    w2 = np.empty((L, streams, E, d_out, Hd), np.float32)
    b2 = np.empty((L, streams, E, d_out), np.float32)
    wr = np.empty((L, streams, E, d_in), np.float32)
    br = np.empty((L, streams, E), np.float32)
    for j in range(L):
        for x in range(streams):
            _uniform(rng, wr[j, x], math.sqrt(6.0 / (d_in + E)))
            _uniform(rng, br[j, x], 1.0 / math.sqrt(d_in))
            for m in range(E):
                _uniform(rng, w1[j, x, m], math.sqrt(6.0 / (d_in + Hd)))
                _uniform(rng, b1[j, x, m], 1.0 / math.sqrt(d_in))
                _uniform(rng, w2[j, x, m], math.sqrt(6.0 / (Hd + d_out)))
                _uniform(rng, b2[j, x, m], 1.0 / math.sqrt(Hd))
    if not with_bias:
        b1[:] = 0
        b2[:] = 0
        br[:] = 0
    if w.src_layout == 1:
        src_k = np.ascontiguousarray(src_k.transpose(0, 1, 3, 2, 4))
        if src_v is not None:
            src_v = np.ascontiguousarray(src_v.transpose(0, 1, 3, 2, 4))
    if w.dtype == "bf16":
        for a in (src_k, src_v, w1, b1, w2, b2, wr, br):
            if a is not None:
                round_to_bf16(a)
    return Inputs(src_k, src_v, w1, b1, w2, b2, wr, br, w.dtype)


def sample_rows(n_tok: int, n: int, seed: int) -> np.ndarray:
    """A seeded sorted sample of flattened token rows that always includes
    the first and the last row (the ragged tail of the last token tile)."""
    if n >= n_tok:
        return np.arange(n_tok, dtype=np.int64)
    rng = np.random.Generator(np.random.PCG64(10_000 + seed))
    mid = rng.choice(np.arange(1, n_tok - 1), size=max(0, n - 2), replace=False)
    return np.unique(np.concatenate([[0, n_tok - 1], mid]).astype(np.int64))


def projection_weights(L: int, d_act: int, d_kv: int, seed: int, dtype: str = "bf16"):
    """Stand-in target key/value projections for the activation variant:
    W^K, W^V [L][d_kv][d_act] Xavier-uniform U(+-sqrt(6/(d_act+d_kv))) and
    b^K, b^V [L][d_kv] U(+-1/sqrt(d_act)), drawn in that order per layer
    (W^K, b^K, W^V, b^V), from PCG64(20_000 + seed); rounded like generate()."""
    rng = np.random.Generator(np.random.PCG64(20_000 + seed))
    wk = np.empty((L, d_kv, d_act), np.float32)
    wv = np.empty((L, d_kv, d_act), np.float32)
    bk = np.empty((L, d_kv), np.float32)
    bv = np.empty((L, d_kv), np.float32)
    for l in range(L):
        _uniform(rng, wk[l], math.sqrt(6.0 / (d_act + d_kv)))
        _uniform(rng, bk[l], 1.0 / math.sqrt(d_act))
        _uniform(rng, wv[l], math.sqrt(6.0 / (d_act + d_kv)))
        _uniform(rng, bv[l], 1.0 / math.sqrt(d_act))
    if dtype == "bf16":
        for a in (wk, bk, wv, bv):
            round_to_bf16(a)
    return wk, bk, wv, bv


def activations(L: int, B: int, T: int, d_act: int, seed: int, dtype: str = "bf16") -> np.ndarray:
    """Intermediate activation rows [L][B][T][d_act] ~ N(0, 1) from
    PCG64(30_000 + seed), rounded like generate()."""
    rng = np.random.Generator(np.random.PCG64(30_000 + seed))
    a = rng.standard_normal((L, B, T, d_act), dtype=np.float32)
    if dtype == "bf16":
        round_to_bf16(a)
    return a


def replay_inputs(B: int, T: int, H_q: int, H_kv: int, D: int, seed: int, kv_layout: int = 0):
    """Replay-attention operands from PCG64(40_000 + seed), drawn in the order
    q [B][T][H_q][D], k, v [B][T][H_kv][D], all N(0, 1) and rounded to bf16;
    k and v are returned transposed to [B][H_kv][T][D] when kv_layout = 1."""
    rng = np.random.Generator(np.random.PCG64(40_000 + seed))
    q = round_to_bf16(rng.standard_normal((B, T, H_q, D), dtype=np.float32))
    k = round_to_bf16(rng.standard_normal((B, T, H_kv, D), dtype=np.float32))
    v = round_to_bf16(rng.standard_normal((B, T, H_kv, D), dtype=np.float32))
    if kv_layout == 1:
        k = np.ascontiguousarray(k.transpose(0, 2, 1, 3))
        v = np.ascontiguousarray(v.transpose(0, 2, 1, 3))
    return q, k, v


def source_attention(B: int, T: int, seed: int, window: float = 64.0, sink: float = 4.0,
                     hitters: float = 2.0, noise: float = 0.5) -> np.ndarray:
    """Stand-in for a source model's head-averaged causal attention map,
    fp32 [B][T][T] from PCG64(50_000 + seed): row u is a softmax over v <= u
    of  -|u - v|/window + sink*[v = 0] + hitters*h[b][v] + noise*eps[b][u][v]
    (locality, an attention sink at position 0, per-position heavy hitters
    h ~ N(0, 1), entry noise eps ~ N(0, 1)); entries v > u are 0.  Drawn:
    h [B][T], then eps row block by row block."""
    rng = np.random.Generator(np.random.PCG64(50_000 + seed))
    h = rng.standard_normal((B, T), dtype=np.float32)
    A = np.empty((B, T, T), np.float32)
    pos = np.arange(T, dtype=np.float32)
    blk = max(1, min(T, (1 << 22) // max(T, 1)))
    lg = np.empty((blk, T), np.float32)
    eps = np.empty((blk, T), np.float32)
    fut = np.empty((blk, T), bool)
    for b in range(B):
        col = hitters * h[b]
        col[0] += sink
        for u0 in range(0, T, blk):
            n = min(T, u0 + blk) - u0
            g, e, f = lg[:n], eps[:n], fut[:n]
            rng.standard_normal(out=e, dtype=np.float32)
            np.subtract(pos[u0:u0 + n, None], pos[None, :], out=g)
            np.abs(g, out=g)
            g *= np.float32(-1.0 / window)
            g += col[None, :]
            e *= np.float32(noise)
            g += e
            np.greater(pos[None, :], pos[u0:u0 + n, None], out=f)
            g[f] = -np.inf
            g -= g.max(axis=1, keepdims=True)
            np.exp(g, out=g)
            g /= g.sum(axis=1, keepdims=True)
            A[b, u0:u0 + n] = g
    return A


def backbone_params(w: Workload, d_h: int, d_ff: int, seed: int, n_slots: int = 1) -> np.ndarray:
    """Packed parameters of the backbone experts, float32 [L_tgt/N][2][E][P]
    (bf16-representable), from PCG64(60_000 + seed), N = n_slots slots per
    channel window: for each (window, x, m), in the packed order (the shared
    input projection, one cross-attention block per slot, the output
    projection of the N slots' concatenation), LayerNorm gains U(0.8, 1.2) and
    shifts U(+-0.1), weight matrices Xavier-uniform
    U(+-sqrt(6/(fan_in+fan_out))), biases U(+-1/sqrt(fan_in))."""
    d_in, d_out, N = w.d_in, w.d_out, n_slots
    cab = [("ln", d_h), ("ln", d_h),
           ("w", (d_h, d_h)), ("b", (d_h, d_h)), ("w", (d_h, d_h)), ("b", (d_h, d_h)),
           ("w", (d_h, d_h)), ("b", (d_h, d_h)), ("w", (d_h, d_h)), ("b", (d_h, d_h)), ("ln", d_h),
           ("w", (d_ff, d_h)), ("b", (d_ff, d_h)), ("w", (d_h, d_ff)), ("b", (d_h, d_ff))]
    parts = ([("ln", d_in), ("w", (d_h, d_in)), ("b", (d_h, d_in))] + cab * N +
             [("ln", N * d_h), ("w", (N * d_out, N * d_h)), ("b", (N * d_out, N * d_h))])
    P = sum(2 * a if k == "ln" else (a[0] * a[1] if k == "w" else a[0]) for k, a in parts)
    rng = np.random.Generator(np.random.PCG64(60_000 + seed))
    out = np.empty((w.L_tgt // N, 2, w.E, P), np.float32)
    for j in range(w.L_tgt // N):
        for x in range(2):
            for m in range(w.E):
                dst = out[j, x, m]
                o = 0
                for k, a in parts:
                    if k == "ln":
                        dst[o:o + a] = rng.uniform(0.8, 1.2, a).astype(np.float32)
                        dst[o + a:o + 2 * a] = rng.uniform(-0.1, 0.1, a).astype(np.float32)
                        o += 2 * a
                    elif k == "w":
                        n = a[0] * a[1]
                        _uniform(rng, dst[o:o + n], math.sqrt(6.0 / (a[0] + a[1])))
                        o += n
                    else:
                        _uniform(rng, dst[o:o + a[0]], 1.0 / math.sqrt(a[1]))
                        o += a[0]
    return round_to_bf16(out)


def window_router(w: Workload, n_slots: int, seed: int):
    """Router of the channel-window backbone: weights [L_tgt/N][2][E][N*d_in]
    Xavier-uniform and bias [L_tgt/N][2][E] U(+-1/sqrt(N*d_in)), drawn per
    (window, x) in that order from PCG64(70_000 + seed), bf16-rounded."""
    N, d = n_slots, n_slots * w.d_in
    rng = np.random.Generator(np.random.PCG64(70_000 + seed))
    wr = np.empty((w.L_tgt // N, 2, w.E, d), np.float32)
    br = np.empty((w.L_tgt // N, 2, w.E), np.float32)
    for j in range(w.L_tgt // N):
        for x in range(2):
            _uniform(rng, wr[j, x], math.sqrt(6.0 / (d + w.E)))
            _uniform(rng, br[j, x], 1.0 / math.sqrt(d))
    return round_to_bf16(wr), round_to_bf16(br)
