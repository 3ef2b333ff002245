"""Pins of the oracle's backbone translator over a multi-slot channel window
(paper App. C.2, "Backbone Translator": z_r = GELU(W_In LN_In(X_r)), the
recurrent scan h_0 = z_1, h_r = CAB_r(h_{r-1}, z_r), then
GELU(W_Out LN_Out(Concat(h_1..h_N)))), as the experts of the mixture whose
router reads the window's concatenated source rows.  None of them restates
the oracle: N = 1 is the single-slot function (itself pinned elsewhere), and
the other expectations are closed forms of inputs built so that each block
adds nothing or a known constant."""
import math

import numpy as np
import pytest

from oracle import OracleDims

EPS = 1e-5


def G(a):
    return 0.5 * a * (1.0 + math.erf(a / math.sqrt(2.0)))


def _dims(L_tgt, T, d, E=1, top_k=1, B=1):
    return OracleDims(L_src=L_tgt, L_tgt=L_tgt, B=B, T=T, H_src=1, D_src=d, H_tgt=1, D_tgt=d, E=E, hidden=d,
                      top_k=top_k)


def _pack(d, N, *, w_in=None, cab=None, w_out=None, b_out=None):
    """Packed parameters of one expert with d_in = d_h = d_ff = d_out = d:
    unit LayerNorms and W_in = I unless given; each slot's block from
    cab(r) -> dict of overrides (default: every projection and bias zero, so
    the block adds nothing); W_out = I and b_out = 0 unless given."""
    I = np.eye(d, dtype=np.float32)
    Z = np.zeros((d, d), np.float32)
    one, zero = np.ones(d, np.float32), np.zeros(d, np.float32)
    parts = [one, zero, I if w_in is None else w_in, zero]
    for r in range(N):
        c = dict(ln_q_g=one, ln_q_b=zero, ln_c_g=one, ln_c_b=zero, wq=Z, bq=zero, wk=Z, bk=zero, wv=Z, bv=zero,
                 wo=Z, bo=zero, ln_f_g=one, ln_f_b=zero, w_f1=Z, b_f1=zero, w_f2=Z, b_f2=zero)
        if cab:
            c.update(cab(r))
        parts += [c[k] for k in ("ln_q_g", "ln_q_b", "ln_c_g", "ln_c_b", "wq", "bq", "wk", "bk", "wv", "bv", "wo",
                                 "bo", "ln_f_g", "ln_f_b", "w_f1", "b_f1", "w_f2", "b_f2")]
    parts += [np.ones(N * d, np.float32), np.zeros(N * d, np.float32),
              np.eye(N * d, dtype=np.float32) if w_out is None else w_out,
              np.zeros(N * d, np.float32) if b_out is None else b_out]
    p = np.concatenate([np.asarray(a, np.float32).ravel() for a in parts])
    from oracle import oracle_backbone_window_param_count
    assert p.size == oracle_backbone_window_param_count(d, d, d, d, N)
    return p


def _run(src, params, N, n_heads=1, wr=None, br=None, E=1, top_k=1):
    """src float32 [L][B][T][1][d]; params [L/N][2][E][P] (or one expert's
    vector, used for every window, X and expert)."""
    from oracle import oracle_backbone_window
    L, B, T, _, d = src.shape
    W = L // N
    if params.ndim == 1:
        params = np.broadcast_to(params, (W, 2, E, params.size)).copy()
    wr = np.zeros((W, 2, E, N * d), np.float32) if wr is None else wr
    br = np.zeros((W, 2, E), np.float32) if br is None else br
    dk, dv = oracle_backbone_window(_dims(L, T, d, E, top_k, B), src, src, np.arange(L, dtype=np.int32), params, wr,
                                    br, d, n_heads, d, N)
    return dk


def test_one_slot_is_the_single_slot_backbone(oracle_built):
    """N = 1: the window function is mot_oracle_backbone_translate bit for bit
    (same parameters, router, Top-K and gates)."""
    from oracle import oracle_backbone_param_count, oracle_backbone_translate, oracle_backbone_window
    rng = np.random.default_rng(61)
    d_in, d_h, d_ff, d_out, nh = 8, 8, 16, 8, 2
    dims = OracleDims(L_src=2, L_tgt=3, B=2, T=6, H_src=1, D_src=d_in, H_tgt=2, D_tgt=d_out // 2, E=3, hidden=d_h,
                      top_k=2)
    P = oracle_backbone_param_count(d_in, d_h, d_ff, d_out)
    params = (rng.standard_normal((3, 2, 3, P)) * 0.4).astype(np.float32)
    src_k = rng.standard_normal((2, 2, 6, 1, d_in)).astype(np.float32)
    src_v = rng.standard_normal((2, 2, 6, 1, d_in)).astype(np.float32)
    wr = rng.standard_normal((3, 2, 3, d_in)).astype(np.float32)
    br = rng.standard_normal((3, 2, 3)).astype(np.float32)
    lm = np.array([1, -1, 0], np.int32)
    a = oracle_backbone_translate(dims, src_k, src_v, lm, params, wr, br, d_h, nh, d_ff)
    b = oracle_backbone_window(dims, src_k, src_v, lm, params, wr, br, d_h, nh, d_ff, 1)
    for u, v in zip(a, b):
        assert np.array_equal(np.nan_to_num(u, nan=7.0), np.nan_to_num(v, nan=7.0))


@pytest.mark.parametrize("N", [2, 3])
def test_blocks_adding_nothing_repeat_the_first_slot(N, oracle_built):
    """Every block zero (no attention output, no FFN): h_r = h_{r-1} = z_1, so
    F = (z_1, ..., z_1) and, since repeating a vector keeps its mean and
    population variance, every target layer of the window receives
    GELU(LN(z_1)), whatever the later slots hold.  x_1 = (3, 1, 3, 1):
    z_1 alternates GELU(c), GELU(-c) with c = 1/sqrt(1 + eps), their
    difference is c, so LN gives +-e, e = (c/2)/sqrt(c^2/4 + eps)."""
    d, T = 4, 2
    rng = np.random.default_rng(62)
    src = rng.standard_normal((N, 1, T, 1, d)).astype(np.float32)
    src[0, 0, :, 0] = [3, 1, 3, 1]
    got = _run(src, _pack(d, N), N)
    c = 1 / math.sqrt(1 + EPS)
    e = (c / 2) / math.sqrt(c * c / 4 + EPS)
    want = [G(e), G(-e), G(e), G(-e)]
    for r in range(N):
        for t in range(T):
            np.testing.assert_allclose(got[r, 0, t, 0], want, rtol=1e-12, atol=1e-14)


def test_scan_accumulates_slot_by_slot(oracle_built):
    """N = 3, attention zero, FFN reduced to its bias b_f2 = delta e_0 in every
    block: h_r = h_{r-1} + delta e_0, so h_r = z_1 + r delta e_0 (the
    recurrence builds on the previous state, not on z_r).  With
    x_1 = (3, 1, 3, 1), F = (z_1 + delta e_0, z_1 + 2 delta e_0, z_1 + 3 delta e_0)
    and the output is GELU(LN_out(F)) over the 12 values, cut into three
    layers."""
    d, N, delta = 4, 3, 0.5
    e0 = np.zeros(d, np.float32)
    e0[0] = delta
    src = np.zeros((N, 1, 1, 1, d), np.float32)
    src[0, 0, 0, 0] = [3, 1, 3, 1]
    src[1, 0, 0, 0] = [9, -4, 2, 0]      # later slots must not matter here
    src[2, 0, 0, 0] = [-1, 5, 5, -7]
    got = _run(src, _pack(d, N, cab=lambda r: dict(b_f2=e0)), N)
    c = 1 / math.sqrt(1 + EPS)
    p, q = G(c), G(-c)
    F = []
    for r in range(1, N + 1):
        F += [p + r * delta, q, p, q]
    mu = sum(F) / len(F)
    var = sum((a - mu) ** 2 for a in F) / len(F)
    want = [G((a - mu) / math.sqrt(var + EPS)) for a in F]
    np.testing.assert_allclose(got[:, 0, 0, 0].ravel(), want, rtol=1e-12, atol=1e-14)


def test_zero_output_weights_give_the_bias_per_slot(oracle_built):
    """W_out = 0: target layer r of the window receives GELU(b_out[r d_out ..])
    whatever the sources and blocks."""
    d, N = 4, 2
    rng = np.random.default_rng(63)
    b_out = rng.standard_normal(N * d).astype(np.float32)
    src = rng.standard_normal((2 * N, 2, 3, 1, d)).astype(np.float32)
    got = _run(src, _pack(d, N, w_out=np.zeros((N * d, N * d), np.float32), b_out=b_out), N)
    for w in range(2):
        for r in range(N):
            want = [G(float(v)) for v in b_out[r * d:(r + 1) * d]]
            np.testing.assert_allclose(got[w * N + r].reshape(-1, d), np.broadcast_to(want, (6, d)), rtol=1e-13)


def test_router_reads_the_concatenated_window(oracle_built):
    """Two experts that output constants (W_out = 0, b_out = 1 or -1 ones), a
    router that looks only at the first channel of slot 2 (router column
    d_in): Top-1 picks expert 0 where that value is positive, expert 1 where
    it is negative, regardless of slot 1."""
    d, N, T = 4, 2, 5
    src = np.zeros((N, 1, T, 1, d), np.float32)
    src[0, 0, :, 0, 0] = [5, -5, 5, -5, 5]              # slot 1: the opposite pattern
    src[1, 0, :, 0, 0] = [1, 1, -1, -1, 2]
    src[1, 0, :, 0, 1] = 1.0
    Zo = np.zeros((N * d, N * d), np.float32)
    params = np.stack([_pack(d, N, w_out=Zo, b_out=np.full(N * d, s, np.float32)) for s in (1.0, -1.0)])
    params = np.broadcast_to(params, (1, 2, 2, params.shape[-1])).copy()
    wr = np.zeros((1, 2, 2, N * d), np.float32)
    wr[..., 0, d] = 4.0
    wr[..., 1, d] = -4.0
    got = _run(src, params, N, wr=wr, E=2, top_k=1)
    sign = np.array([1, 1, -1, -1, 1], np.float64)
    for r in range(N):
        np.testing.assert_allclose(got[r, 0, :, 0, 0], [G(s) for s in sign], rtol=1e-13)


def test_slot_order_matters_and_windows_are_checked(oracle_built):
    """Swapping the two slots of a window changes its output (the scan is
    ordered); a window with some unmapped slots is refused."""
    from oracle import oracle_backbone_window, oracle_backbone_window_param_count
    rng = np.random.default_rng(64)
    d, N = 8, 2
    P = oracle_backbone_window_param_count(d, d, 16, d, N)
    params = (rng.standard_normal((1, 2, 1, P)) * 0.4).astype(np.float32)
    src = rng.standard_normal((2, 1, 5, 1, d)).astype(np.float32)
    wr = np.zeros((1, 2, 1, N * d), np.float32)
    br = np.zeros((1, 2, 1), np.float32)
    dims = _dims(2, 5, d)
    a, _ = oracle_backbone_window(dims, src, src, np.array([0, 1], np.int32), params, wr, br, d, 2, 16, N)
    b, _ = oracle_backbone_window(dims, src, src, np.array([1, 0], np.int32), params, wr, br, d, 2, 16, N)
    assert not np.allclose(a, b) and not np.allclose(a, b[::-1])
    with pytest.raises(ValueError):
        oracle_backbone_window(dims, src, src, np.array([0, -1], np.int32), params, wr, br, d, 2, 16, N)
