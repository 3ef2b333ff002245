"""GPU parity of the context-replay step (paper App. C.4): Top-S source-guided
key selection and replay attention, through the C ABI, against the oracle.

* selection (mot_topS_select): bit-exact key sets on maps with many ties,
  ragged row lengths (rows shorter than S, rows across 256-element chunks),
  and a 16500-token map (rows longer than the LDS row cache) on sampled
  rows;
* sparse attention over the selected sets (grouped-query heads, both KV
  layouts, head dims 64 and 128, S = 32 .. 256), sets with padding and
  out-of-range entries, an all-empty set (zeros);
* full causal attention (the bottom L_Full layers) with a ragged last tile;
* the replay benchmark's layer shape (Qwen2.5-7B target heads, T = 8192,
  S = 128) on sampled rows.
Bar: key sets bit-exact; attention outputs (bf16) within a relative
Frobenius error of 2e-2 of the fp64 oracle.
"""
import numpy as np
import pytest

from paper_2607_28979_amd import binding as mb
from paper_2607_28979_amd.inputs import replay_inputs, source_attention

from helpers import TOL, rel_frob, to_dev

pytestmark = pytest.mark.gpu


def _gpu_select(A, S):
    import torch
    B, T = A.shape[0], A.shape[1]
    a = torch.from_numpy(np.ascontiguousarray(A, dtype=np.float32)).cuda()
    idx = torch.full((B, T, S), -7, dtype=torch.int32, device="cuda")
    mb.topS_select(a, idx, B, T, S)
    torch.cuda.synchronize()
    return idx


def _gpu_attention(q, k, v, idx, kv_layout=0):
    """idx: None, or a device / numpy int32 [B][T][S] array."""
    import torch
    B, T, Hq, D = q.shape
    Hkv = k.shape[2] if kv_layout == 0 else k.shape[1]
    o = torch.full((B, T, Hq, D), 9.0, dtype=torch.bfloat16, device="cuda")
    ii = idx
    if isinstance(idx, np.ndarray):
        ii = torch.from_numpy(np.ascontiguousarray(idx, dtype=np.int32)).cuda()
    S = 0 if idx is None else idx.shape[2]
    mb.replay_attention(to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16"), ii, o, B=B, T=T, H_q=Hq,
                        H_kv=Hkv, D=D, S=S, kv_layout=kv_layout)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("B,T,S", [(2, 300, 32), (1, 517, 128), (3, 70, 64)])
def test_topS_select_bit_exact(B, T, S, oracle_built):
    """Coarsely quantised maps (many equal values) so the lower-position tie
    rule decides many sets."""
    from oracle import oracle_topS_select
    print("case select", B, T, S, flush=True)
    rng = np.random.default_rng(T + S)
    A = (np.round(rng.random((B, T, T)) * 16) / 16).astype(np.float32)
    got = _gpu_select(A, S).cpu().numpy()
    want = oracle_topS_select(A, S)
    assert np.array_equal(got, want), int((got != want).sum())


@pytest.mark.parametrize("values", [(0.25,), (0.25, 0.5), (0.3, 0.3000001, 0.7)])
def test_topS_select_heavy_ties(values, oracle_built):
    """Maps of one to three distinct values: the boundary bin of the first
    radix digit holds more than 256 keys on the long rows (the kernel's radix
    fallback) and fewer on the short ones (its direct ranking); the sets
    follow the lower-position rule."""
    from oracle import oracle_topS_select
    B, T, S = 2, 700, 128
    print("case select heavy ties", values, flush=True)
    rng = np.random.default_rng(len(values))
    A = np.asarray(values, np.float32)[rng.integers(0, len(values), (B, T, T))]
    got = _gpu_select(A, S).cpu().numpy()
    want = oracle_topS_select(A, S)
    assert np.array_equal(got, want), int((got != want).sum())


@pytest.mark.parametrize("T", [2500, 2133])
def test_topS_select_every_row_of_long_maps(T, oracle_built):
    """Every row of maps of a few thousand positions (key caches of 10 and
    8.5 KB; T = 2133 takes the unaligned key fill), against the oracle."""
    from oracle import oracle_topS_select
    print("case select long map T", T, flush=True)
    rng = np.random.default_rng(T)
    A = (np.round(rng.random((1, T, T)) * 64) / 64).astype(np.float32)
    got = _gpu_select(A, 128).cpu().numpy()
    want = oracle_topS_select(A, 128)
    assert np.array_equal(got, want), int((got != want).sum())


def test_topS_select_structured_map(oracle_built):
    from oracle import oracle_topS_select
    A = source_attention(2, 600, seed=1)
    got = _gpu_select(A, 128).cpu().numpy()
    assert np.array_equal(got, oracle_topS_select(A, 128))


def test_topS_select_long_rows_sampled(oracle_built):
    """T = 16500 exceeds the LDS row cache: the uncached kernel, on sampled
    rows (first, last, and around 16384)."""
    from oracle import oracle_topS_rows
    T, S = 16500, 128
    print("case select long T", T, flush=True)
    A = source_attention(1, T, seed=2)
    got = _gpu_select(A, S).cpu().numpy()
    rows = [(0, u) for u in (0, 127, 128, 5000, 16383, 16384, 16385, T - 1)]
    want = oracle_topS_rows(A, S, rows)
    for i, (b, u) in enumerate(rows):
        assert np.array_equal(got[b, u], want[i]), u


ATTN = [  # B, T, H_q, H_kv, D, S, kv_layout
    (2, 200, 8, 2, 128, 64, 0),
    (1, 260, 28, 4, 128, 128, 1),     # Qwen2.5-7B heads (7 per KV head)
    (2, 150, 4, 4, 64, 32, 0),        # one query head per KV head, 2 of 4 waves without key blocks
    (1, 300, 12, 2, 64, 128, 1),      # Qwen2.5-1.5B heads
    # sets above 128 keys: the larger register-array instantiations
    (1, 280, 14, 2, 128, 192, 0),     # the largest S at D = 128
    (1, 230, 7, 1, 128, 160, 0),      # 10 key blocks: waves with 3 and with 2
    (1, 270, 8, 4, 64, 256, 1),       # the largest S at D = 64
    # set sizes whose chunk count per row is not a power of two (a row-local
    # LDS swizzle is needed): 12 and 28 chunks
    (1, 240, 6, 2, 64, 96, 0),
    (1, 300, 4, 1, 64, 224, 1),
    # an odd context: the last position of the two-position kernel is alone
    (1, 201, 8, 2, 128, 64, 0),
    (2, 99, 16, 2, 64, 128, 1),       # 8 query heads per KV head: the pair fills all 16 columns
]


@pytest.mark.parametrize("case", ATTN, ids=["B%d-T%d-Hq%d-Hkv%d-D%d-S%d-l%d" % c for c in ATTN])
def test_sparse_attention_parity(case, oracle_built):
    from oracle import oracle_replay_attention, oracle_topS_select
    B, T, Hq, Hkv, D, S, lay = case
    print("case sparse", case, flush=True)
    q, k, v = replay_inputs(B, T, Hq, Hkv, D, seed=T + D, kv_layout=lay)
    A = source_attention(B, T, seed=T)
    idx = oracle_topS_select(A, S)
    got = _gpu_attention(q, k, v, idx, lay)
    want = oracle_replay_attention(q, k, v, idx, kv_layout=lay)
    err = rel_frob(got, want)
    print("  rel-Frobenius %.3e" % err, flush=True)
    assert err <= TOL["bf16"]
    # per position too: no row may be off even when the total is fine
    worst = max(rel_frob(got[b, u], want[b, u]) for b in range(B) for u in range(T))
    assert worst <= 2 * TOL["bf16"], worst


@pytest.mark.parametrize("order", ["ascending", "shuffled", "duplicates"])
def test_sparse_pair_union_and_two_pass(order, oracle_built):
    """The two-position kernel on random sets (neighbouring positions share
    few keys, so most pairs' unions exceed its 192-key limit and it runs one
    pass per position), on shuffled sets and on sets with a repeated entry
    (both taken as listed, one pass per position), for an odd context:
    every position against the oracle, which attends each listed entry."""
    from oracle import oracle_replay_attention
    B, T, Hq, Hkv, D, S = 1, 401, 14, 2, 128, 128
    print("case pair kernel", order, flush=True)
    q, k, v = replay_inputs(B, T, Hq, Hkv, D, seed=17)
    rng = np.random.default_rng(17)
    idx = np.full((B, T, S), -1, np.int32)
    for u in range(T):
        n = min(u + 1, S)
        sel = rng.choice(u + 1, size=n, replace=False)
        if order == "ascending":
            sel = np.sort(sel)
        if order == "duplicates" and n >= 2:
            sel[-1] = sel[0]
        idx[0, u, :n] = sel
    got = _gpu_attention(q, k, v, idx)
    want = oracle_replay_attention(q, k, v, idx)
    worst = max(rel_frob(got[0, u], want[0, u]) for u in range(T))
    print("  worst position rel-Frobenius %.3e" % worst, flush=True)
    assert rel_frob(got, want) <= TOL["bf16"] and worst <= 2 * TOL["bf16"], worst


def test_sparse_attention_padding_and_invalid_entries(oracle_built):
    """Entries that are -1 or lie after the query position are skipped; a set
    with no valid entry gives zeros."""
    from oracle import oracle_replay_attention
    B, T, Hq, Hkv, D, S = 1, 96, 4, 2, 128, 32
    q, k, v = replay_inputs(B, T, Hq, Hkv, D, seed=5)
    rng = np.random.default_rng(5)
    idx = np.full((B, T, S), -1, np.int32)
    for u in range(T):
        n = int(rng.integers(1, min(u + 1, S - 1) + 1))
        idx[0, u, :n] = np.sort(rng.choice(u + 1, size=n, replace=False))
    bad = idx.copy()
    bad[0, :, S - 1] = np.minimum(np.arange(T) + 5, T + 100)   # after u (or past T): skipped
    bad[0, 10] = -1                                             # empty set
    got = _gpu_attention(q, k, v, bad)
    want = oracle_replay_attention(q, k, v, idx)
    assert np.array_equal(got[0, 10], np.zeros((Hq, D)))
    keep = np.ones(T, bool)
    keep[10] = False
    assert rel_frob(got[0, keep], want[0, keep]) <= TOL["bf16"]


@pytest.mark.parametrize("B,T,Hq,Hkv,D,lay", [(1, 200, 4, 2, 128, 0), (2, 130, 6, 1, 64, 1), (1, 64, 2, 2, 128, 0),
                                              # several 128-position tile pairs, a ragged last tile,
                                              # seven query heads per KV head
                                              (1, 1000, 14, 2, 128, 1), (2, 333, 4, 4, 64, 0)])
def test_causal_attention_parity(B, T, Hq, Hkv, D, lay, oracle_built):
    from oracle import oracle_replay_attention
    print("case causal", B, T, Hq, Hkv, D, lay, flush=True)
    q, k, v = replay_inputs(B, T, Hq, Hkv, D, seed=3 * T + D, kv_layout=lay)
    got = _gpu_attention(q, k, v, None, lay)
    want = oracle_replay_attention(q, k, v, None, kv_layout=lay)
    err = rel_frob(got, want)
    print("  rel-Frobenius %.3e" % err, flush=True)
    assert err <= TOL["bf16"]
    worst = max(rel_frob(got[b, u], want[b, u]) for b in range(B) for u in range(T))
    assert worst <= 2 * TOL["bf16"], worst


def test_sparse_with_full_sets_equals_causal(oracle_built):
    """With S >= T every set is the whole causal prefix, so the sparse kernel
    and the causal kernel compute the same attention."""
    B, T, Hq, Hkv, D = 1, 120, 4, 2, 64
    q, k, v = replay_inputs(B, T, Hq, Hkv, D, seed=9)
    A = source_attention(B, T, seed=9)
    idx = _gpu_select(A, 128)
    sp = _gpu_attention(q, k, v, idx)
    fu = _gpu_attention(q, k, v, None)
    assert rel_frob(sp, fu) <= 1e-2


def test_replay_layer_full_size_sampled(oracle_built):
    """The replay benchmark's layer: Qwen2.5-7B target (28 query heads on 4
    KV heads of 128), T = 8192, S = 128: selection and sparse attention over
    the whole layer on the GPU, sampled rows checked against the oracle; the
    causal kernel on the same layer, sampled rows."""
    from oracle import oracle_replay_attention_rows, oracle_topS_rows
    from paper_2607_28979_amd.configs import REPLAY
    w = REPLAY
    print("case replay layer full size", flush=True)
    q, k, v = replay_inputs(w.B, w.T, w.H_q, w.H_kv, w.D, seed=w.seed)
    A = source_attention(w.B, w.T, seed=w.seed)
    idx = _gpu_select(A, w.S)
    rows = [(0, u) for u in (0, 1, 127, 128, 129, 4095, 6000, w.T - 1)]
    want_idx = oracle_topS_rows(A, w.S, rows)
    idx_h = idx.cpu().numpy()
    for i, (b, u) in enumerate(rows):
        assert np.array_equal(idx_h[b, u], want_idx[i]), u
    got = _gpu_attention(q, k, v, idx)
    want = oracle_replay_attention_rows(q, k, v, idx_h, rows)
    for i, (b, u) in enumerate(rows):
        assert rel_frob(got[b, u], want[i]) <= TOL["bf16"], u
    got_c = _gpu_attention(q, k, v, None)
    rows_c = [(0, u) for u in (0, 63, 64, 3000, w.T - 1)]
    want_c = oracle_replay_attention_rows(q, k, v, None, rows_c)
    for i, (b, u) in enumerate(rows_c):
        assert rel_frob(got_c[b, u], want_c[i]) <= TOL["bf16"], u


def test_causal_caller_workspace_equals_owned(oracle_built):
    """The full causal path with a caller-owned workspace (the V staging of
    mot_replay_workspace_bytes) gives the same bits as with the library's
    own buffer, and a smaller workspace is refused before any launch."""
    import torch
    B, T, Hq, Hkv, D = 2, 333, 8, 2, 128
    q, k, v = replay_inputs(B, T, Hq, Hkv, D, seed=5, kv_layout=0)
    dq, dk, dv = (to_dev(a, "bf16") for a in (q, k, v))
    need = mb.replay_workspace_bytes(B, T, Hq, Hkv, D)
    assert need == B * Hkv * D * ((T + 63) // 64 * 64) * 2
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    ws.fill_(0x5A)
    outs = []
    for wsp in (None, ws):
        o = torch.zeros((B, T, Hq, D), dtype=torch.bfloat16, device="cuda")
        mb.replay_attention(dq, dk, dv, None, o, B, T, Hq, Hkv, D, workspace=wsp)
        torch.cuda.synchronize()
        outs.append(o.cpu())
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
    o = torch.zeros((B, T, Hq, D), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(mb.MotError) as e:
        mb.replay_attention(dq, dk, dv, None, o, B, T, Hq, Hkv, D, workspace=ws[: need - 16])
    assert e.value.name == "MOT_ERR_WORKSPACE_TOO_SMALL"
