"""CPU checks of the near-tie handling the Top-K parity tests use (paper
Sec. 3, Definition "Mixture-of-Translators": the K largest gates,
renormalised).  A row whose K-th and (K+1)-th scores are nearly equal may
select either set at fp32 precision; the GPU tests then accept the oracle row
of any admissible set and nothing else.  Here the "device" rows are oracle
rows themselves, so the acceptance rule is exercised without a GPU."""
import numpy as np
import pytest

from paper_2607_28979_amd.configs import Workload
from paper_2607_28979_amd.inputs import generate

from helpers import (ROW_TOL, admissible_sets, check_topk_rows, forced_set_router_bias, oracle_dims,
                     unit_logits, unit_rows)


def _tie_case(K):
    w = Workload("ties", "bf16", L_src=1, L_tgt=1, B=1, T=6, H_src=1, D_src=64, H_tgt=1, D_tgt=64, E=4,
                 hidden=64, seed=11, top_k=K)
    inp = generate(w)
    lm = np.zeros(1, np.int32)
    # row 2 of unit (0, K): translators 1 and 3 share the K-th place up to 1e-5
    lg = unit_logits(w, inp, lm, 0, 0, rows=[2])[0]
    order = np.argsort(-lg)
    if K == 1:
        want = {1: lg.max() + 0.5, 3: lg.max() + 0.5 + 1e-5}
    else:   # translator 0 clearly first, then the 1/3 near tie
        want = {0: lg.max() + 2.0, 1: lg.max() + 0.5, 3: lg.max() + 0.5 + 1e-5}
    for m, t in want.items():
        inp.br[0, 0, m] = np.float32(float(inp.br[0, 0, m]) + (t - lg[m]))
    return w, inp, lm


def _oracle(w, inp, lm, br):
    from oracle import oracle_translate
    rk, _ = oracle_translate(oracle_dims(w), inp.src_k, inp.src_v, lm, inp.w1, inp.b1, inp.w2, inp.b2,
                             inp.wr, br)
    return unit_rows(rk, w, 0)


@pytest.mark.parametrize("K", [1, 2])
def test_near_tie_accepts_either_admissible_set(K, oracle_built):
    w, inp, lm = _tie_case(K)
    lg = unit_logits(w, inp, lm, 0, 0, rows=[2])[0]
    sets = admissible_sets(lg, K)
    assert len(sets) == 2 and all(1 in s or 3 in s for s in sets)
    ref = _oracle(w, inp, lm, inp.br)
    for chosen in sets:
        dev = ref.copy()
        dev[2] = _oracle(w, inp, lm, forced_set_router_bias(inp, lg, 0, 0, chosen, K))[2]
        keep, worst, n_tie = check_topk_rows(w, inp, lm, 0, 0, dev, ref)
        assert n_tie == 1 and not keep[2] and worst <= ROW_TOL["bf16"]


@pytest.mark.parametrize("K", [1, 2])
def test_near_tie_rejects_other_sets_and_wrong_rows(K, oracle_built):
    w, inp, lm = _tie_case(K)
    lg = unit_logits(w, inp, lm, 0, 0, rows=[2])[0]
    ref = _oracle(w, inp, lm, inp.br)
    # a set outside the admissible ones: translator 2 in place of the tied pair
    bad = (2,) if K == 1 else (0, 2)
    br = inp.br.copy()
    for m in range(4):
        br[0, 0, m] = np.float32(float(br[0, 0, m]) + (10.0 if m in bad else -10.0))
    dev = ref.copy()
    dev[2] = _oracle(w, inp, lm, br)[2]
    with pytest.raises(AssertionError):
        check_topk_rows(w, inp, lm, 0, 0, dev, ref)
    # a clear row that is off by 5 % fails the per-row bar
    dev = ref.copy()
    dev[4] *= 1.05
    with pytest.raises(AssertionError):
        check_topk_rows(w, inp, lm, 0, 0, dev, ref)
