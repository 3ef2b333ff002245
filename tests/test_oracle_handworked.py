"""Hand-worked pins of the backbone translator body (paper App. C.2) and of
replay attention (App. C.4) that do not restate the oracle's formulas: the
inputs are chosen so that every LayerNorm sees a two-level pattern and every
softmax two scores, and the expected values are closed forms worked out on
paper (GELU itself is pinned against tabulated normal-CDF values elsewhere,
so it is evaluated here through math.erf).  Each pin fails under a plausible
slip in the oracle: unbiased instead of population variance, epsilon outside
the square root, a 1/width or 1/d_h attention scale instead of 1/sqrt(width),
heads split in the wrong place, a 1/D replay scale."""
import math

import numpy as np
import pytest

from oracle import OracleDims

EPS = 1e-5


def G(a):
    """Exact GELU a * Phi(a)."""
    return 0.5 * a * (1.0 + math.erf(a / math.sqrt(2.0)))


def ln_pair(delta):
    """LayerNorm (unit gain, zero shift) of a vector alternating m + delta,
    m - delta: mean m, population variance delta^2, so the entries are
    +-delta / sqrt(delta^2 + eps)."""
    return delta / math.sqrt(delta * delta + EPS)


def _identity_backbone(d, n_heads, T, wq_zero=True, bq=None, wk_identity=False, wv_identity=False,
                       wo_identity=False):
    """Packed parameters of one expert with widths d_in = d_h = d_ff = d_out =
    d: unit LayerNorms, W_in = W_out = I, zero biases, the FFN switched off
    (W_f1 = W_f2 = 0), attention projections as requested."""
    from oracle import oracle_backbone_param_count
    I = np.eye(d, dtype=np.float32)
    Z = np.zeros((d, d), np.float32)
    one, zero = np.ones(d, np.float32), np.zeros(d, np.float32)
    parts = [one, zero, I, zero,                                   # LN_in, W_in, b_in
             one, zero, one, zero,                                 # LN_Q, LN_C
             Z if wq_zero else I, zero if bq is None else np.asarray(bq, np.float32),
             I if wk_identity else Z, zero, I if wv_identity else Z, zero,
             I if wo_identity else Z, zero,                        # Wo, bo
             one, zero, Z, zero, Z, zero,                          # LN_F, W_f1, b_f1, W_f2, b_f2
             one, zero, I, zero]                                   # LN_out, W_out, b_out
    p = np.concatenate([a.ravel() for a in parts]).astype(np.float32)
    assert p.size == oracle_backbone_param_count(d, d, d, d)
    return p


def _run_backbone(x_rows, params, n_heads):
    """One unit (target layer 0, keys), one expert (gate 1), one batch row."""
    from oracle import oracle_backbone_translate
    T, d = x_rows.shape
    dims = OracleDims(L_src=1, L_tgt=1, B=1, T=T, H_src=1, D_src=d, H_tgt=1, D_tgt=d, E=1, hidden=d, top_k=1)
    src = x_rows.reshape(1, 1, T, 1, d).astype(np.float32)
    P = params.reshape(1, 1, 1, -1)
    P = np.concatenate([P, P], axis=1)                             # keys and values share the expert
    wr = np.zeros((1, 2, 1, d), np.float32)
    br = np.zeros((1, 2, 1), np.float32)
    dk, _ = oracle_backbone_translate(dims, src, src, np.zeros(1, np.int32), P, wr, br, d, n_heads, d)
    return dk[0, 0, :, 0, :]


def test_backbone_layernorms(oracle_built):
    """T positions see no attention (W_v = 0) and no FFN, so each output row is
    GELU(LN_out(GELU(LN_in(x)))).  x = (3, 1, 3, 1): LN_in gives +-c with
    c = 1/sqrt(1 + eps) (unbiased variance would give +-0.866); z alternates
    GELU(c), GELU(-c), whose difference is c exactly, so LN_out gives +-e with
    e = (c/2)/sqrt(c^2/4 + eps).  x = 1 +- 2^-7: delta^2 = 6.1e-5 is comparable
    to eps, which makes the placement of eps visible (inside the root:
    c = 0.92694; outside it: 0.99872)."""
    d = 4
    P = _identity_backbone(d, 1, 2)
    x = np.array([[3, 1, 3, 1], [1 + 2 ** -7, 1 - 2 ** -7, 1 + 2 ** -7, 1 - 2 ** -7]], np.float32)
    got = _run_backbone(x, P, 1)
    for t, delta in enumerate((1.0, 2.0 ** -7)):
        c = ln_pair(delta)
        e = ln_pair(c / 2)
        want = [G(e), G(-e), G(e), G(-e)]
        np.testing.assert_allclose(got[t], want, rtol=1e-12, atol=1e-14)
    assert abs(ln_pair(2.0 ** -7) - 0.9269437) < 1e-7
    assert abs(got[1, 0] - G(ln_pair(ln_pair(2.0 ** -7) / 2))) < 1e-12


def test_backbone_attention_scale_and_heads(oracle_built):
    """Two positions, two heads of width 2 (d_h = 4).  x_0 = (3, 1, 3, 1) and
    x_1 = (1, 3, 1, 3) give z_0 = (p, q, p, q), z_1 = (q, p, q, p) with
    p - q = c, and LN_C(z_0) = (e, -e, e, -e) = -LN_C(z_1).  K = V = LN_C(z)
    (W_k = W_v = I); Q = b_q = (b0, 0, 0, b1) at both positions (W_q = 0).
    Position 1 of head 0 scores keys 0 and 1 as +-b0 e / sqrt(2), so its
    attention output is tanh(b0 e / sqrt 2) (e, -e); head 1 scores them as
    -+b1 e / sqrt(2) and gives -tanh(b1 e / sqrt 2) (e, -e).  Position 0 sees
    only key 0: (e, -e, e, -e).  With W_o = I the block output is
    h = z + attention, and the row is GELU(LN_out(h))."""
    d, b0, b1 = 4, 1.5, -0.75
    P = _identity_backbone(d, 2, 2, bq=[b0, 0, 0, b1], wk_identity=True, wv_identity=True, wo_identity=True)
    x = np.array([[3, 1, 3, 1], [1, 3, 1, 3]], np.float32)
    got = _run_backbone(x, P, 2)
    c = ln_pair(1.0)
    p, q = G(c), G(-c)
    e = ln_pair(c / 2)
    t0 = math.tanh(b0 * e / math.sqrt(2.0))
    t1 = -math.tanh(b1 * e / math.sqrt(2.0))
    h = [np.array([p + e, q - e, p + e, q - e]), np.array([q + t0 * e, p - t0 * e, q + t1 * e, p - t1 * e])]
    for t in range(2):
        v = h[t]
        mu = sum(v) / 4
        var = sum((a - mu) ** 2 for a in v) / 4
        want = [G((a - mu) / math.sqrt(var + EPS)) for a in v]
        np.testing.assert_allclose(got[t], want, rtol=1e-12, atol=1e-14)
    # the scale matters: with 1/width the head-0 factor would be tanh(0.75 e) = 0.635, not 0.786
    assert abs(t0 - 0.78585) < 1e-4 and abs(math.tanh(b0 * e / 2) - 0.63515) < 1e-4


@pytest.mark.parametrize("sparse", [False, True])
def test_replay_attention_scale(sparse, oracle_built):
    """D = 64, one head: q_1 = (2, 0, ...), k_0 = 0, k_1 = (4, 0, ...), so the
    scores of position 1 are 0 and 8 / sqrt(64) = 1 and its output is
    (1, e) / (1 + e) on v_0 = (1, 0, ...), v_1 = (0, 1, 0, ...); position 0
    returns v_0.  A 1/D scale would give weights (1, e^0.125) / (1 + e^0.125)."""
    from oracle import oracle_replay_attention
    D = 64
    q = np.zeros((1, 2, 1, D), np.float32)
    k = np.zeros((1, 2, 1, D), np.float32)
    v = np.zeros((1, 2, 1, D), np.float32)
    q[0, :, 0, 0] = 2.0
    k[0, 1, 0, 0] = 4.0
    v[0, 0, 0, 0] = 1.0
    v[0, 1, 0, 1] = 1.0
    idx = np.array([[[0, -1], [0, 1]]], np.int32) if sparse else None
    o = oracle_replay_attention(q, k, v, idx)
    want1 = np.zeros(D)
    want1[0], want1[1] = 1 / (1 + math.e), math.e / (1 + math.e)
    want0 = np.zeros(D)
    want0[0] = 1.0
    np.testing.assert_allclose(o[0, 1, 0], want1, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(o[0, 0, 0], want0, rtol=1e-14, atol=1e-15)
    assert abs(want1[1] - 0.7310585786300049) < 1e-15
