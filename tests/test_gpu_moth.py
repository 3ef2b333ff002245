"""GPU parity of the activation-translation variant MoT-h (paper App. C.5).

MoT-h translates one intermediate-activation stream per channel with the
same Mixture-of-Translators (mot_translate with streams = 1) and restores the
target key/value caches from it through the target's fixed projections
(mot_restore_kv): K = W^K a + b^K, V = W^V a + b^V.

* streams = 1 translation on every kernel path against the oracle run with
  one stream;
* restoration against the oracle: ragged token and output tiles, both
  target layouts, a layer map with skipped layers, with and without bias;
* identity projection: K and V are the activation cut into heads, bit-exact;
* the chain translate -> restore against the oracle's chain.
Bar: bf16, relative Frobenius error per (layer, K/V) <= 2e-2; skipped layers
and identity projections bit-exact.
"""
import numpy as np
import pytest

from paper_2607_28979_amd import binding as mb
from paper_2607_28979_amd.configs import Workload
from paper_2607_28979_amd.inputs import activations, generate, projection_weights

from helpers import ROW_TOL, SENTINEL, TOL, oracle_dims, rel_frob, row_errors, to_dev

pytestmark = pytest.mark.gpu

# activation rows 256 -> 512 wide (fused, routed and unfused paths) and
# 384 -> 640 (unfused path only); 300 tokens leave a ragged last tile
MOTH = [
    Workload("moth-256-512", "bf16", L_src=3, L_tgt=4, B=2, T=150, H_src=1, D_src=256, H_tgt=1,
             D_tgt=512, E=4, hidden=256, seed=71, layer_map="depth_ratio", streams=1),
    Workload("moth-384-640", "bf16", L_src=2, L_tgt=2, B=1, T=300, H_src=1, D_src=384, H_tgt=1,
             D_tgt=640, E=3, hidden=320, seed=72, streams=1),
]


def _lm(w):
    if w.layer_map == "identity":
        return np.arange(w.L_tgt, dtype=np.int32) % w.L_src
    return mb.depth_ratio_map(w.L_src, w.L_tgt)


def _translate_act(w, inp, lm, algo, top_k=0):
    """streams = 1 translation of the activation inp.src_k (inputs drawn with
    streams = 1); returns (device tensor [L_tgt][B][T][1][d_out], float64 copy)."""
    import torch
    one = lambda a: to_dev(a, "bf16")
    a = to_dev(inp.src_k, "bf16")
    dst = torch.full((w.L_tgt, w.B, w.T, w.H_tgt, w.D_tgt), SENTINEL, dtype=torch.bfloat16,
                     device="cuda")
    shapes = mb.Shapes.from_workload(w, algo=algo, top_k=top_k)
    mb.translate(a, None, lm, one(inp.w1), one(inp.b1), one(inp.w2), one(inp.b2), one(inp.wr),
                 one(inp.br), dst, None, shapes)
    torch.cuda.synchronize()
    return dst, dst.float().cpu().numpy().astype(np.float64)


def _algos(w):
    if w.d_in in (128, 256, 512) and w.d_out in (128, 256, 512):
        return [mb.ALGO_FUSED, mb.ALGO_ROUTED, mb.ALGO_UNFUSED]
    return [mb.ALGO_ROUTED, mb.ALGO_UNFUSED]


@pytest.mark.parametrize("w", MOTH, ids=[w.name for w in MOTH])
def test_activation_translation_streams1(w, oracle_built):
    from oracle import oracle_translate
    inp = generate(w)
    lm = _lm(w)
    ref, _ = oracle_translate(oracle_dims(w), inp.src_k, None, lm, inp.w1, inp.b1, inp.w2, inp.b2,
                              inp.wr, inp.br)
    for algo in _algos(w):
        print("case", w.name, "streams 1 algo", algo, flush=True)
        _, got = _translate_act(w, inp, lm, algo)
        worst = max(rel_frob(got[j].reshape(w.n_tok, -1), ref[j].reshape(w.n_tok, -1))
                    for j in range(w.L_tgt))
        worst_row = max(float(row_errors(got[j].reshape(w.n_tok, -1), ref[j].reshape(w.n_tok, -1)).max())
                        for j in range(w.L_tgt))
        print("  max layer rel-Frobenius error %.3e, max row error %.3e" % (worst, worst_row), flush=True)
        assert worst <= TOL["bf16"], (w.name, algo, worst)
        assert worst_row <= ROW_TOL["bf16"], (w.name, algo, worst_row)


def _restore_gpu(act, lm, wk, bk, wv, bv, L, B, T, H, D, layout):
    import torch
    shape = (L, B, T, H, D) if layout == 0 else (L, B, H, T, D)
    dk = torch.full(shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
    dv = torch.full(shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
    dev = lambda x: None if x is None else to_dev(x, "bf16")
    a = act if not isinstance(act, np.ndarray) else dev(act)
    mb.restore_kv(a, lm, dev(wk), dev(bk), dev(wv), dev(bv), dk, dv, L=L, B=B, T=T,
                  d_act=act.shape[-1], H_tgt=H, D_tgt=D, dst_layout=layout)
    torch.cuda.synchronize()
    return (dk.float().cpu().numpy().astype(np.float64),
            dv.float().cpu().numpy().astype(np.float64))


RESTORE = [  # (L, B, T, d_act, H_tgt, D_tgt, layout, bias)
    (3, 2, 150, 512, 4, 128, 0, True),      # 300 tokens: ragged token tile
    (3, 1, 300, 512, 4, 128, 1, True),
    (2, 1, 200, 192, 5, 40, 0, True),       # d_kv = 200: ragged output tile
    (2, 3, 70, 256, 5, 40, 1, False),
    (1, 1, 129, 1536, 4, 128, 0, True),     # Qwen2.5-7B K/V width from a 1536-wide activation
    # launches of >= 128 workgroups with d_kv % 256 == 0: the 256 x 256-tile kernel, ragged token tiles
    (4, 2, 2100, 512, 4, 128, 0, True),
    (5, 1, 5000, 384, 2, 128, 1, False),
]


@pytest.mark.parametrize("case", RESTORE, ids=["L%d-B%d-T%d-a%d-H%d-D%d-l%d-b%d" % c for c in RESTORE])
def test_restore_parity(case, oracle_built):
    from oracle import oracle_restore_kv
    L, B, T, d_act, H, D, layout, bias = case
    print("case restore", case, flush=True)
    act = activations(L, B, T, d_act, seed=L + T)
    wk, bk, wv, bv = projection_weights(L, d_act, H * D, seed=d_act + H)
    if not bias:
        bk = bv = None
    lm = np.arange(L, dtype=np.int32)
    if L > 2:
        lm[1] = -1
    gk, gv = _restore_gpu(act, lm, wk, bk, wv, bv, L, B, T, H, D, layout)
    rk, rv = oracle_restore_kv(act, lm, wk, bk, wv, bv, B=B, T=T, H_tgt=H, D_tgt=D,
                               dst_layout=layout)
    for l in range(L):
        if lm[l] < 0:
            assert (gk[l] == SENTINEL).all() and (gv[l] == SENTINEL).all()
            continue
        ek, ev = rel_frob(gk[l], rk[l]), rel_frob(gv[l], rv[l])
        print("  layer %d rel-Frobenius K %.3e V %.3e" % (l, ek, ev), flush=True)
        assert ek <= TOL["bf16"] and ev <= TOL["bf16"], (case, l, ek, ev)


@pytest.mark.parametrize("layout,T,D", [(0, 190, 64), (1, 190, 64), (0, 8200, 128), (1, 8200, 128)])
def test_restore_identity_is_exact(layout, T, D):
    """W^K = W^V = I, no bias: each output is one exact product plus zeros,
    so K and V are the bf16 activation cut into heads, bit for bit (T = 8200
    with two heads of 128: the 256 x 256-tile kernel)."""
    L, B, H = 2, 1, 2
    act = activations(L, B, T, H * D, seed=3)
    eye = np.broadcast_to(np.eye(H * D, dtype=np.float32), (L, H * D, H * D)).copy()
    gk, gv = _restore_gpu(act, None, eye, None, eye, None, L, B, T, H, D, layout)
    want = act.astype(np.float64).reshape(L, B, T, H, D)
    if layout == 1:
        want = want.transpose(0, 1, 3, 2, 4)
    assert np.array_equal(gk, want) and np.array_equal(gv, want)


def test_moth_chain_translate_then_restore(oracle_built):
    """The whole MoT-h path on the GPU (streams = 1 translation on the fused
    path, then restoration from the translated activation kept on the
    device) against the same chain in the oracle."""
    from oracle import oracle_restore_kv, oracle_translate
    w = MOTH[0]
    inp = generate(w)
    lm = _lm(w)
    H, D = 4, 64
    wk, bk, wv, bv = projection_weights(w.L_tgt, w.d_out, H * D, seed=w.seed)
    a_dev, _ = _translate_act(w, inp, lm, mb.ALGO_FUSED)
    gk, gv = _restore_gpu(a_dev, None, wk, bk, wv, bv, w.L_tgt, w.B, w.T, H, D, 0)
    a_ref, _ = oracle_translate(oracle_dims(w), inp.src_k, None, lm, inp.w1, inp.b1, inp.w2, inp.b2,
                                inp.wr, inp.br)
    rk, rv = oracle_restore_kv(a_ref.reshape(w.L_tgt, w.B, w.T, w.d_out), None, wk, bk, wv, bv,
                               B=w.B, T=w.T, H_tgt=H, D_tgt=D)
    worst = max(max(rel_frob(gk[l], rk[l]), rel_frob(gv[l], rv[l])) for l in range(w.L_tgt))
    print("  chain max layer rel-Frobenius error %.3e" % worst, flush=True)
    assert worst <= TOL["bf16"]


def test_moth_full_width_sampled(oracle_built):
    """The MoT-h benchmark's widths (1536-wide source activation, E = 8
    translators 1536 -> 2048 -> 3584, restored to 4 x 128 keys and values)
    on two layers and 700 tokens, through the benchmark's calls; sampled rows
    of the translated activation and of the restored K/V against the oracle."""
    import torch
    from oracle import oracle_restore_kv, oracle_rows
    from paper_2607_28979_amd.configs import MOTH, small_variant
    from paper_2607_28979_amd.inputs import sample_rows
    w = small_variant(MOTH.act, L_src=2, L_tgt=2, B=1, T=700)
    print("case", w.name, "L 2 T 700", flush=True)
    inp = generate(w)
    lm = _lm(w)
    wk, bk, wv, bv = projection_weights(w.L_tgt, w.d_out, MOTH.d_kv, seed=w.seed)
    a_dev, a_got = _translate_act(w, inp, lm, mb.ALGO_AUTO)
    gk, gv = _restore_gpu(a_dev, None, wk, bk, wv, bv, w.L_tgt, w.B, w.T, MOTH.kv_heads,
                          MOTH.head_dim, 0)
    rows = sample_rows(w.n_tok, 16, w.seed)
    ref = oracle_rows(oracle_dims(w), inp.src_k, None, lm, inp.w1, inp.b1, inp.w2, inp.b2, inp.wr,
                      inp.br, units=[(j, 0) for j in range(w.L_tgt)], rows=rows)
    rk, rv = oracle_restore_kv(ref.reshape(w.L_tgt, 1, len(rows), w.d_out), None, wk, bk, wv, bv,
                               B=1, T=len(rows), H_tgt=MOTH.kv_heads, D_tgt=MOTH.head_dim)
    for j in range(w.L_tgt):
        ea = rel_frob(a_got[j].reshape(w.n_tok, -1)[rows], ref[j])
        assert float(row_errors(a_got[j].reshape(w.n_tok, -1)[rows], ref[j]).max()) <= ROW_TOL["bf16"], j
        ek = rel_frob(gk[j].reshape(w.n_tok, -1)[rows], rk[j].reshape(len(rows), -1))
        ev = rel_frob(gv[j].reshape(w.n_tok, -1)[rows], rv[j].reshape(len(rows), -1))
        print("  layer %d rel-Frobenius act %.3e K %.3e V %.3e" % (j, ea, ek, ev), flush=True)
        assert max(ea, ek, ev) <= TOL["bf16"], (j, ea, ek, ev)
    del a_dev
    torch.cuda.empty_cache()
