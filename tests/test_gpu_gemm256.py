"""GPU parity of the two-GEMM path's 256 x 256-tile kernels (the layer-1 GEMM
with its gated GELU epilogue and the layer-2 GEMM over every expert's hidden
units, paper Sec. 3 Eq. mot_definition with App. C.2's GELU) against the
oracle.

The library runs these kernels when one launch of the two-GEMM path holds
at least 128 workgroups of 256 x 256 layer-1 tiles (ceil(n_tok / 256) *
ceil(E * hidden / 256) * units >= 128); smaller launches take the 128 x
128-tile kernels, which the other parity files cover.  Every case here is
sized past that threshold (asserted below) and has ragged edges: token
counts that are not multiples of 256, E * hidden and d_out that are not
multiples of 256, both cache layouts, no-bias and identity-activation
forms, Top-K < E, and the largest expert count (E = 16, where the gate-mixed
output bias spans both halves of the bias product's K axis)."""
import numpy as np
import pytest

from paper_2607_28979_amd import binding as mb
from paper_2607_28979_amd.configs import Workload
from paper_2607_28979_amd.inputs import generate

from helpers import (ROW_TOL, TOL, check_topk_rows, max_unit_error, oracle_dims, rel_frob, row_errors, run_gpu,
                     unit_rows)

pytestmark = pytest.mark.gpu


def _w(**kw):
    base = dict(L_src=3, L_tgt=4, B=1, T=1100, H_src=4, D_src=64, H_tgt=3, D_tgt=32, E=3, hidden=320, seed=21)
    base.update(kw)
    return Workload("gemm256", "bf16", **base)


def _big_tiles(w, lm):
    units = 2 * int((np.asarray(lm) >= 0).sum())
    return -(-w.n_tok // 256) * -(-(w.E * w.hidden) // 256) * units >= 128


def _oracle(w, inp, lm, act=0, with_bias=True):
    from oracle import oracle_translate
    b = (lambda a: a) if with_bias else (lambda a: None)
    return oracle_translate(oracle_dims(w, act), inp.src_k, inp.src_v, lm, inp.w1, b(inp.b1), inp.w2, b(inp.b2),
                            inp.wr, b(inp.br))


def _check(w, lm, g, r):
    err = max_unit_error(g[0], g[1], r[0], r[1], w, lm)
    worst = 0.0
    for j in range(w.L_tgt):
        if lm[j] < 0:
            continue
        for a, b in zip(g, r):
            worst = max(worst, float(row_errors(unit_rows(a, w, j), unit_rows(b, w, j)).max()))
    print("  max unit rel-Frobenius error %.3e, max row error %.3e" % (err, worst), flush=True)
    assert err <= TOL["bf16"] and worst <= ROW_TOL["bf16"], (err, worst)
    assert np.isfinite(g[0]).all() and np.isfinite(g[1]).all()


CASES = {
    # 1100 tokens (4 full tiles + 76), E*hidden = 960 (3 full tiles + 192), d_out = 96
    "ragged": (_w(), np.array([0, 1, 2, 2], np.int32)),
    # E = 16 experts of 64 hidden units, d_in 512 -> d_out 256
    "e16": (_w(E=16, hidden=64, H_src=8, H_tgt=2, D_tgt=128, T=1300, seed=22), np.array([2, 0, 1, 1], np.int32)),
    # an unmapped layer, d_out 512 = two output tiles
    "skip": (_w(H_tgt=4, D_tgt=128, E=2, hidden=1024, T=700, seed=23), np.array([1, -1, 0, 2], np.int32)),
    # d_in = E * hidden = 64: two 32-wide K slices per product, fewer than the
    # slices the pipeline keeps in flight (the prologue reloads the last one)
    "short_k": (_w(L_src=2, L_tgt=3, H_src=1, D_src=64, H_tgt=1, D_tgt=64, E=1, hidden=64, B=4, T=4100, seed=25),
                np.array([1, 0, 1], np.int32)),
}


@pytest.mark.parametrize("name", list(CASES))
def test_gemm256_parity(name, oracle_built):
    w, lm = CASES[name]
    assert _big_tiles(w, lm)
    print("case", name, "n_tok", w.n_tok, "E*hidden", w.E * w.hidden, "d_out", w.d_out, flush=True)
    inp = generate(w)
    g = run_gpu(w, inp, lm, algo=mb.ALGO_UNFUSED)
    _check(w, lm, g, _oracle(w, inp, lm))
    if (lm < 0).any():
        from helpers import SENTINEL
        j = int(np.nonzero(lm < 0)[0][0])
        assert (g[0][j] == SENTINEL).all() and (g[1][j] == SENTINEL).all()


def test_gemm256_no_bias_identity(oracle_built):
    """No biases (the accumulators start at zero, no gate-mixed b2) and the
    identity activation."""
    w, lm = CASES["ragged"]
    print("case ragged, no bias, identity activation", flush=True)
    inp = generate(w)
    g = run_gpu(w, inp, lm, algo=mb.ALGO_UNFUSED, act=mb.ACT_IDENTITY, with_bias=False)
    _check(w, lm, g, _oracle(w, inp, lm, act=1, with_bias=False))


def test_gemm256_layouts_are_permutations():
    """BHTD source and target caches give the BTHD results permuted, bit for
    bit (the kernels read heads through a separate offset term)."""
    w, lm = CASES["ragged"]
    print("case ragged, BTHD vs BHTD", flush=True)
    g = run_gpu(w, generate(w), lm, algo=mb.ALGO_UNFUSED)
    wh = w.with_(src_layout=1, dst_layout=1)
    h = run_gpu(wh, generate(wh), lm, algo=mb.ALGO_UNFUSED)
    assert np.array_equal(h[0], g[0].transpose(0, 1, 3, 2, 4))
    assert np.array_equal(h[1], g[1].transpose(0, 1, 3, 2, 4))


@pytest.mark.parametrize("k", [1, 2])
def test_gemm256_topk(k, oracle_built):
    """Dense-masked Top-K on the large tiles: every row meets the per-row
    bar, near-tie rows match one of their admissible sets."""
    w, lm = CASES["ragged"]
    w = w.with_(top_k=k)
    print("case ragged, top_k", k, flush=True)
    inp = generate(w)
    gk, gv = run_gpu(w, inp, lm, algo=mb.ALGO_UNFUSED)
    rk, rv = _oracle(w, inp, lm)
    worst, n_tie, n_all = 0.0, 0, 0
    for j in range(w.L_tgt):
        for x, (g, r) in enumerate(((gk, rk), (gv, rv))):
            gr, rr = unit_rows(g, w, j), unit_rows(r, w, j)
            keep, _, nt = check_topk_rows(w, inp, lm, j, x, gr, rr)
            n_tie += nt
            n_all += keep.size
            worst = max(worst, rel_frob(gr[keep], rr[keep]))
    print("  max unit rel-Frobenius error %.3e (%d near-tie rows of %d)" % (worst, n_tie, n_all), flush=True)
    assert worst <= TOL["bf16"] and n_tie <= max(2, n_all // 100)


def test_gemm256_matches_fused_kernel():
    """A shape both paths serve (d_in 256 -> d_out 512): the two-GEMM path
    on large tiles and the fused kernel agree to bf16 rounding."""
    w = _w(H_src=4, D_src=64, H_tgt=4, D_tgt=128, E=8, hidden=256, T=1500, seed=24)
    lm = np.array([0, 1, 2, 2], np.int32)
    assert _big_tiles(w, lm)
    print("case fused vs two-GEMM, n_tok", w.n_tok, flush=True)
    inp = generate(w)
    f = run_gpu(w, inp, lm, algo=mb.ALGO_FUSED)
    u = run_gpu(w, inp, lm, algo=mb.ALGO_UNFUSED)
    assert max_unit_error(f[0], f[1], u[0], u[1], w, lm) <= 1e-2


# ---------------------------------------------------------------------------
# routed (Top-K sparse) two-GEMM path: each translator runs only on the
# tokens that selected it, in plan tiles of up to 256 (token, translator)
# assignments (paper Sec. 3, Definition "Mixture-of-Translators", K < E)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name,k", [("ragged", 1), ("ragged", 2), ("e16", 1), ("e16", 3), ("skip", 1)])
def test_routed_two_gemm_parity(name, k, oracle_built):
    """Routed two-GEMM rows against the oracle: the per-row bar everywhere,
    near-tie rows matched to one of their admissible sets."""
    w, lm = CASES[name]
    w = w.with_(top_k=k)
    print("case", name, "top_k", k, "routed two-GEMM", flush=True)
    inp = generate(w)
    gk, gv = run_gpu(w, inp, lm, algo=mb.ALGO_ROUTED)
    rk, rv = _oracle(w, inp, lm)
    worst, worst_row, n_tie, n_all = 0.0, 0.0, 0, 0
    for j in range(w.L_tgt):
        if lm[j] < 0:
            from helpers import SENTINEL
            assert (gk[j] == SENTINEL).all() and (gv[j] == SENTINEL).all()
            continue
        for x, (g, r) in enumerate(((gk, rk), (gv, rv))):
            gr, rr = unit_rows(g, w, j), unit_rows(r, w, j)
            assert np.isfinite(gr).all()
            keep, wr_, nt = check_topk_rows(w, inp, lm, j, x, gr, rr)
            n_tie += nt
            n_all += keep.size
            worst_row = max(worst_row, wr_)
            worst = max(worst, rel_frob(gr[keep], rr[keep]))
    print("  max unit rel-Frobenius error %.3e, max row error %.3e (%d near-tie rows of %d)"
          % (worst, worst_row, n_tie, n_all), flush=True)
    assert worst <= TOL["bf16"] and n_tie <= max(2, n_all // 100)


def test_routed_two_gemm_auto_layouts_and_dense_agreement():
    """AUTO takes the routed path for top_k < E on these shapes (same bits
    as ALGO_ROUTED); BHTD caches give the BTHD rows permuted, bit for bit;
    the dense-masked two-GEMM path agrees to bf16 rounding."""
    w, lm = CASES["ragged"]
    w = w.with_(top_k=2)
    print("case ragged top_k 2: AUTO vs ROUTED vs dense-masked, BTHD vs BHTD", flush=True)
    inp = generate(w)
    r = run_gpu(w, inp, lm, algo=mb.ALGO_ROUTED)
    a = run_gpu(w, inp, lm, algo=mb.ALGO_AUTO)
    assert np.array_equal(r[0], a[0]) and np.array_equal(r[1], a[1])
    d = run_gpu(w, inp, lm, algo=mb.ALGO_UNFUSED)
    assert max_unit_error(r[0], r[1], d[0], d[1], w, lm) <= 1e-2
    wh = w.with_(src_layout=1, dst_layout=1)
    h = run_gpu(wh, generate(wh), lm, algo=mb.ALGO_ROUTED)
    assert np.array_equal(h[0], r[0].transpose(0, 1, 3, 2, 4))
    assert np.array_equal(h[1], r[1].transpose(0, 1, 3, 2, 4))


def test_routed_two_gemm_skewed_and_deterministic(oracle_built):
    """A router bias that sends every token to translator 1 (Top-1): the other
    translators' assignment lists are empty and their tiles absent; the result
    equals the oracle and is bit-identical on a second run."""
    w, lm = CASES["ragged"]
    w = w.with_(top_k=1)
    print("case ragged top_k 1, all tokens to translator 1", flush=True)
    inp = generate(w)
    inp.br = np.zeros_like(inp.br)
    inp.br[..., 1] = 50.0
    a = run_gpu(w, inp, lm, algo=mb.ALGO_ROUTED)
    b = run_gpu(w, inp, lm, algo=mb.ALGO_ROUTED)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    _check(w, lm, a, _oracle(w, inp, lm))
