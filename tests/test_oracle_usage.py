"""Pins of the oracle's translator-usage statistics (paper Sec. 4, paragraph
"MoT Architecture Ablation"): I_m = the cumulative Top-K selection count of
translator m, CV^2 = Var_m(I_m) / Mean_m(I_m)^2, entropy = -sum_m p_m ln p_m
with p_m = I_m / sum I.  Pinned by the paper's printed MoT-Uni row, closed
forms, and a pure-Python count of Top-K selections."""
import math
import os

import numpy as np
import pytest

from oracle import OracleDims

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "mot_usage_table.txt")


def _stats(counts):
    from oracle import oracle_usage_stats
    return oracle_usage_stats(np.asarray(counts, np.int64))


def test_paper_mot_uni_row(oracle_built):
    """MoT-Uni uses both translators equally: I_1 = I_2 gives CV^2 = 0 and
    entropy ln 2; printed as 0.00 and 0.69."""
    rows = {l.split()[0]: (float(l.split()[1]), float(l.split()[2]))
            for l in open(GOLDEN) if l.strip() and not l.startswith("#")}
    for n in (1, 7, 123456):
        cv2, ent = _stats([n, n])
        assert round(cv2, 2) == rows["MoT-Uni"][0] and round(ent, 2) == rows["MoT-Uni"][1]
        assert cv2 == 0.0 and abs(ent - math.log(2)) < 1e-15


@pytest.mark.parametrize("E", [1, 2, 3, 4, 8, 16])
def test_balanced_and_one_hot(E, oracle_built):
    """Balanced counts: CV^2 = 0, entropy = ln E.  All selections on one
    translator: mean N/E, population variance N^2 (E-1)/E^2, so CV^2 = E - 1,
    and entropy 0 (the empty translators contribute 0 ln 0 = 0)."""
    cv2, ent = _stats([5] * E)
    assert cv2 == 0.0 and abs(ent - math.log(E)) < 1e-14
    one = [0] * E
    one[E // 2] = 4096
    cv2, ent = _stats(one)
    assert abs(cv2 - (E - 1)) < 1e-12 and ent == 0.0


def test_two_translator_closed_form(oracle_built):
    """E = 2, counts (a, b): CV^2 = ((a - b) / (a + b))^2 and the entropy is
    the binary entropy of p = a / (a + b)."""
    for a, b in ((3, 1), (1, 3), (900, 100), (1, 999), (50, 51)):
        p = a / (a + b)
        cv2, ent = _stats([a, b])
        assert abs(cv2 - ((a - b) / (a + b)) ** 2) < 1e-14
        assert abs(ent - (-p * math.log(p) - (1 - p) * math.log(1 - p))) < 1e-14


def test_invariances_and_empty(oracle_built):
    """Permuting translators or scaling every count changes neither statistic;
    no selections at all leaves both undefined (NaN)."""
    c = [7, 0, 3, 11, 1]
    base = _stats(c)
    assert np.allclose(_stats(c[::-1]), base, rtol=0, atol=1e-14)
    assert np.allclose(_stats([10 * v for v in c]), base, rtol=0, atol=1e-14)
    assert all(math.isnan(v) for v in _stats([0, 0, 0]))


def _py_counts(src, wr, br, lm, K, streams):
    """Pure-Python Top-K selection counts: logits, softmax, K rounds of
    argmax with the lower index winning ties."""
    L_tgt, _, E, d_in = wr.shape
    counts = np.zeros((L_tgt, streams, E), np.int64)
    for j in range(L_tgt):
        if lm[j] < 0:
            continue
        for x in range(streams):
            rows = src[x][lm[j]].reshape(-1, d_in)
            for z in rows:
                lg = [sum(float(wr[j, x, m, c]) * float(z[c]) for c in range(d_in)) + float(br[j, x, m])
                      for m in range(E)]
                mx = max(lg)
                g = [math.exp(v - mx) for v in lg]
                g = [v / sum(g) for v in g]
                taken = []
                for _ in range(K):
                    best = None
                    for m in range(E):
                        if m not in taken and (best is None or g[m] > g[best]):
                            best = m
                    taken.append(best)
                for m in taken:
                    counts[j, x, m] += 1
    return counts


@pytest.mark.parametrize("K,streams", [(1, 2), (2, 2), (3, 2), (1, 1)])
def test_counts_match_brute_force(K, streams, oracle_built):
    from oracle import oracle_usage
    rng = np.random.default_rng(53 + K)
    L_src, L_tgt, B, T, H, D, E = 2, 3, 2, 5, 2, 2, 3
    d_in = H * D
    src = [rng.standard_normal((L_src, B, T, H, D)).astype(np.float32) for _ in range(streams)]
    wr = rng.standard_normal((L_tgt, streams, E, d_in)).astype(np.float32)
    br = rng.standard_normal((L_tgt, streams, E)).astype(np.float32)
    lm = np.array([1, -1, 0], np.int32)
    dims = OracleDims(L_src=L_src, L_tgt=L_tgt, B=B, T=T, H_src=H, D_src=D, H_tgt=1, D_tgt=4, E=E, hidden=4,
                      top_k=K, streams=streams)
    got = oracle_usage(dims, src[0], src[1] if streams == 2 else None, lm, wr, br)
    assert np.array_equal(got, _py_counts(src, wr, br, lm, K, streams))
    assert (got[1] == 0).all() and (got[[0, 2]].sum(axis=-1) == K * B * T).all()


def test_counts_ties_go_to_the_lower_index(oracle_built):
    """A zero router gives every token equal scores: Top-1 selects translator
    0 for every token, Top-2 translators 0 and 1."""
    from oracle import oracle_usage
    B, T, E = 1, 9, 4
    src = np.ones((1, B, T, 1, 8), np.float32)
    wr = np.zeros((1, 2, E, 8), np.float32)
    br = np.zeros((1, 2, E), np.float32)
    for K, want in ((1, [T, 0, 0, 0]), (2, [T, T, 0, 0]), (4, [T] * 4)):
        dims = OracleDims(L_src=1, L_tgt=1, B=B, T=T, H_src=1, D_src=8, H_tgt=1, D_tgt=8, E=E, hidden=8, top_k=K)
        got = oracle_usage(dims, src, src, np.zeros(1, np.int32), wr, br)
        assert got[0, 0].tolist() == want and got[0, 1].tolist() == want
