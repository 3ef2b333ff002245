"""Seeded randomized parity sweep through the C ABI against the oracle:
translation shapes on every path (two-GEMM with small and large tiles,
fused, routed Top-K < E, fp32), both cache layouts, skipped layers, and Top-S
selection on structured, quantised and few-valued maps.  Each case prints
its shape; the bars are the per-path ones of the other parity files.  Under
Top-K routing the rows whose K-th and (K+1)-th scores are within 1e-3 are
checked against the oracle under each admissible set; their count is
bounded at 4 % of the rows plus two (a K in the middle of 16 experts puts
over 1 % of the rows in a near tie).  A second sweep covers replay attention
and the backbone experts."""
import numpy as np
import pytest

from paper_2607_28979_amd import binding as mb
from paper_2607_28979_amd.configs import Workload
from paper_2607_28979_amd.inputs import backbone_params, generate, replay_inputs, source_attention, window_router

from helpers import (SENTINEL, TOL, check_topk_rows, dst_shape, max_unit_error, oracle_dims, rel_frob, row_errors,
                     run_gpu, to_dev, unit_rows)

pytestmark = pytest.mark.gpu

N_CASES = 240


def _translation_case(rng, kind):
    dtype = "f32" if kind == "f32" else "bf16"
    if kind == "fused":
        d_in, d_out = int(rng.choice([128, 256, 512])), int(rng.choice([128, 256, 512]))
    else:
        d_in = int(rng.choice([64, 128, 192, 256, 384, 512, 1024]))
        d_out = int(rng.choice([32, 64, 96, 128, 256, 320, 512]))
    D_src = int(rng.choice([d for d in (32, 64, 128) if d_in % d == 0]))
    D_tgt = int(rng.choice([d for d in (32, 64, 128) if d_out % d == 0]))
    E = int(rng.choice([1, 2, 3, 4, 8, 16] if dtype == "bf16" else [1, 2, 4]))
    hidden = int(rng.choice([64, 128, 192, 256, 512]))
    big = kind == "two_gemm" and rng.random() < 0.7   # large-tile launches
    T = int(rng.integers(600, 2600)) if big else int(rng.integers(20, 700))
    B = int(rng.integers(1, 3))
    L_src, L_tgt = int(rng.integers(1, 4)), int(rng.integers(1, 3))
    top_k = int(rng.integers(1, E)) if kind == "routed" and E > 1 else 0
    w = Workload("sweep", dtype, L_src=L_src, L_tgt=L_tgt, B=B, T=T, H_src=d_in // D_src, D_src=D_src,
                 H_tgt=d_out // D_tgt, D_tgt=D_tgt, E=E, hidden=hidden, seed=int(rng.integers(1 << 30)),
                 top_k=top_k, src_layout=int(rng.integers(0, 2)), dst_layout=int(rng.integers(0, 2)))
    lm = rng.integers(-1, L_src, L_tgt).astype(np.int32)
    if (lm < 0).all():
        lm[0] = 0
    return w, lm


def _check_translation(w, lm, algo):
    from oracle import oracle_translate
    inp = generate(w)
    g = run_gpu(w, inp, lm, algo=algo)
    r = oracle_translate(oracle_dims(w), inp.src_k, inp.src_v, lm, inp.w1, inp.b1, inp.w2, inp.b2, inp.wr, inp.br)
    for j in range(w.L_tgt):
        if lm[j] < 0:
            assert (g[0][j] == SENTINEL).all() and (g[1][j] == SENTINEL).all()
    if not w.top_k:
        err = max_unit_error(g[0], g[1], r[0], r[1], w, lm)
        print("  unit error %.3e" % err, flush=True)
        assert err <= TOL[w.dtype] and np.isfinite(g[0]).all() and np.isfinite(g[1]).all()
        return
    worst, n_tie, n_all = 0.0, 0, 0
    for j in range(w.L_tgt):
        if lm[j] < 0:
            continue
        for x, (gg, rr) in enumerate(((g[0], r[0]), (g[1], r[1]))):
            gr, rr2 = unit_rows(gg, w, j), unit_rows(rr, w, j)
            keep, _, nt = check_topk_rows(w, inp, lm, j, x, gr, rr2)   # near-tie rows: admissible sets
            n_tie += nt
            n_all += keep.size
            worst = max(worst, rel_frob(gr[keep], rr2[keep]))
    print("  unit error %.3e, %d near-tie rows of %d" % (worst, n_tie, n_all), flush=True)
    assert worst <= TOL[w.dtype] and n_tie <= 2 + n_all // 25


def _check_select(rng):
    import torch
    from oracle import oracle_topS_select
    B, T = int(rng.integers(1, 3)), int(rng.integers(40, 900))
    S = int(rng.choice([32, 64, 96, 128, 160, 256]))
    mode = str(rng.choice(["structured", "quantised", "few values"]))
    if mode == "structured":
        A = source_attention(B, T, seed=int(rng.integers(1 << 30)))
    elif mode == "quantised":
        A = (np.round(rng.random((B, T, T)) * int(rng.integers(2, 40))) / 40).astype(np.float32)
    else:
        vals = np.asarray(rng.random(int(rng.integers(1, 4))), np.float32)
        A = vals[rng.integers(0, len(vals), (B, T, T))]
    print("  select %s B=%d T=%d S=%d" % (mode, B, T, S), flush=True)
    idx = torch.empty((B, T, S), dtype=torch.int32, device="cuda")
    mb.topS_select(torch.from_numpy(A).cuda(), idx, B, T, S)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), oracle_topS_select(A, S))


def test_randomized_sweep(oracle_built):
    rng = np.random.default_rng(20260)
    algos = {"two_gemm": mb.ALGO_UNFUSED, "fused": mb.ALGO_FUSED, "routed": mb.ALGO_AUTO, "f32": mb.ALGO_AUTO}
    for case in range(N_CASES):
        kind = str(rng.choice(["two_gemm", "two_gemm", "fused", "routed", "f32", "select"]))
        if kind == "select":
            print("case %d" % case, flush=True)
            _check_select(rng)
            continue
        w, lm = _translation_case(rng, kind)
        print("case %d %s %s B=%d T=%d d_in=%d(%dx%d) E=%d hidden=%d d_out=%d(%dx%d) top_k=%d layouts=%d%d map=%s"
              % (case, kind, w.dtype, w.B, w.T, w.d_in, w.H_src, w.D_src, w.E, w.hidden, w.d_out, w.H_tgt,
                 w.D_tgt, w.top_k, w.src_layout, w.dst_layout, lm.tolist()), flush=True)
        _check_translation(w, lm, algos[kind])


N_REPLAY_BACKBONE = 90


def _attention(q, k, v, idx, lay):
    import torch
    B, T, Hq, D = q.shape
    Hkv = k.shape[2] if lay == 0 else k.shape[1]
    o = torch.full((B, T, Hq, D), 9.0, dtype=torch.bfloat16, device="cuda")
    ii = None if idx is None else torch.from_numpy(np.ascontiguousarray(idx, dtype=np.int32)).cuda()
    mb.replay_attention(to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16"), ii, o, B=B, T=T, H_q=Hq,
                        H_kv=Hkv, D=D, S=0 if idx is None else idx.shape[2], kv_layout=lay)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64)


def _check_replay(rng, kind):
    from oracle import oracle_replay_attention, oracle_topS_select
    B, T = int(rng.integers(1, 3)), int(rng.integers(2, 600))
    Hkv, G = int(rng.choice([1, 2, 4])), int(rng.choice([1, 2, 3, 4, 7, 8, 16]))
    D, lay = int(rng.choice([64, 128])), int(rng.integers(0, 2))
    q, k, v = replay_inputs(B, T, Hkv * G, Hkv, D, seed=int(rng.integers(1 << 30)), kv_layout=lay)
    idx, desc = None, "causal"
    if kind == "sparse":
        S = int(rng.choice(list(range(32, (192 if D == 128 else 256) + 1, 32))))
        mode = str(rng.choice(["selected", "random ascending", "random unordered"]))
        if mode == "selected":
            idx = oracle_topS_select(source_attention(B, T, seed=int(rng.integers(1 << 30))), S)
        else:   # any number of entries, -1 padded
            idx = np.full((B, T, S), -1, np.int32)
            for b in range(B):
                for u in range(T):
                    n = int(rng.integers(0, min(u + 1, S) + 1))
                    sel = rng.choice(u + 1, size=n, replace=False)
                    idx[b, u, :n] = np.sort(sel) if mode == "random ascending" else sel
        desc = "S=%d %s" % (S, mode)
    print("  %s B=%d T=%d H_q=%d H_kv=%d D=%d layout=%d" % (desc, B, T, Hkv * G, Hkv, D, lay), flush=True)
    got = _attention(q, k, v, idx, lay)
    want = oracle_replay_attention(q, k, v, idx, kv_layout=lay)
    worst = max(rel_frob(got[b, u], want[b, u]) for b in range(B) for u in range(T))
    assert rel_frob(got, want) <= TOL["bf16"] and worst <= 2 * TOL["bf16"], worst


def _check_backbone(rng):
    import torch
    from oracle import oracle_backbone_window
    N = int(rng.choice([1, 1, 2, 3]))
    hw = int(rng.choice([64, 128]))
    nh = int(rng.choice([1, 2, 3])) if 3 * hw * N <= 1024 else 1
    d_h, d_ff = nh * hw, int(rng.choice([64, 128, 256, 512]))
    L_src, L_tgt = int(rng.integers(1, 4)), N * int(rng.integers(1, 3))
    w = Workload("sweep-bb", "bf16", L_src=L_src, L_tgt=L_tgt, B=int(rng.integers(1, 3)), T=int(rng.integers(10, 300)),
                 H_src=int(rng.integers(1, 4)), D_src=int(rng.choice([64, 128])), H_tgt=int(rng.integers(1, 4)),
                 D_tgt=int(rng.choice([32, 64, 96, 128])), E=int(rng.integers(1, 4)), hidden=128,
                 seed=int(rng.integers(1 << 30)))
    lm = []
    for win in range(L_tgt // N):   # a window is mapped or skipped as a whole
        lm += [-1] * N if win > 0 and rng.random() < 0.2 else [int(x) for x in rng.integers(0, L_src, N)]
    lm = np.array(lm, np.int32)
    print("  backbone N=%d d_h=%d (%dx%d) d_ff=%d d_in=%d d_out=%d E=%d B=%d T=%d map=%s"
          % (N, d_h, nh, hw, d_ff, w.d_in, w.d_out, w.E, w.B, w.T, lm.tolist()), flush=True)
    inp = generate(w)
    params = backbone_params(w, d_h, d_ff, seed=w.seed, n_slots=N)
    wr, br = window_router(w, N, seed=w.seed)
    dk = torch.full(dst_shape(w), SENTINEL, dtype=torch.bfloat16, device="cuda")
    dv = torch.full(dst_shape(w), SENTINEL, dtype=torch.bfloat16, device="cuda")
    mb.backbone_translate(to_dev(inp.src_k, "bf16"), to_dev(inp.src_v, "bf16"), lm, to_dev(params, "bf16"),
                          to_dev(wr, "bf16"), to_dev(br, "bf16"), dk, dv, mb.Shapes.from_workload(w), d_h, nh, d_ff,
                          n_slots=N)
    torch.cuda.synchronize()
    gk, gv = (a.float().cpu().numpy().astype(np.float64) for a in (dk, dv))
    rk, rv = oracle_backbone_window(oracle_dims(w), inp.src_k, inp.src_v, lm, params, wr, br, d_h, nh, d_ff, N)
    for j in range(L_tgt):
        if lm[j] < 0:
            assert (gk[j] == SENTINEL).all() and (gv[j] == SENTINEL).all()
            continue
        for g, r in ((gk, rk), (gv, rv)):
            assert rel_frob(unit_rows(g, w, j), unit_rows(r, w, j)) <= TOL["bf16"]
            assert float(row_errors(unit_rows(g, w, j), unit_rows(r, w, j)).max()) <= 2 * TOL["bf16"]


def test_randomized_replay_and_backbone_sweep(oracle_built):
    """Replay attention over selected, random ascending and unordered sets
    (any fill, -1 padded) and the full causal set, grouped-query ratios 1-16,
    D = 64 and 128, both layouts; the backbone experts over windows of 1-3
    slots with 1-3 heads, skipped windows and ragged sizes."""
    rng = np.random.default_rng(20261)
    for case in range(N_REPLAY_BACKBONE):
        kind = str(rng.choice(["sparse", "sparse", "causal", "backbone"]))
        print("case %d %s" % (case, kind), flush=True)
        if kind == "backbone":
            _check_backbone(rng)
        else:
            _check_replay(rng, kind)
