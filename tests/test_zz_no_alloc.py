"""mot_replay_attention_noalloc (the replay attention entry point for callers
that cannot allocate) against mot_replay_attention, through the C ABI.

The no-allocation entry point stages the full causal path's V in the
library's static per-device scratch; its output must equal the existing
entry point's bit for bit (same kernels, same arithmetic), on two calls in a
row, the second smaller than the first, so that the static array's leftovers
from the first call cannot leak into the second."""
import numpy as np
import pytest

from paper_2607_28979_amd import binding as mb
from paper_2607_28979_amd.inputs import replay_inputs, source_attention

from helpers import TOL, rel_frob, to_dev

pytestmark = pytest.mark.gpu


def _pair(B, T, Hq, Hkv, D, lay, seed, S=0):
    import torch
    q, k, v = replay_inputs(B, T, Hq, Hkv, D, seed=seed, kv_layout=lay)
    dq, dk, dv = (to_dev(a, "bf16") for a in (q, k, v))
    idx = None
    if S:
        from oracle import oracle_topS_select
        idx = torch.from_numpy(oracle_topS_select(source_attention(B, T, seed=seed), S)).cuda()
    outs = []
    for fn in (mb.replay_attention, mb.replay_attention_noalloc):
        o = torch.full((B, T, Hq, D), -3.75, dtype=torch.bfloat16, device="cuda")
        fn(dq, dk, dv, idx, o, B, T, Hq, Hkv, D, S=S, kv_layout=lay)
        torch.cuda.synchronize()
        outs.append(o.cpu())
    return outs, (q, k, v, idx)


@pytest.mark.parametrize("lay", [0, 1])
def test_noalloc_equals_replay_attention_two_calls(lay, oracle_built):
    from oracle import oracle_replay_attention
    # first call: 1 x 1000 positions, 4 KV heads of 128 (1 MiB of staged V);
    # second: a smaller one (300 positions, 2 KV heads of 64)
    for case in ((1, 1000, 8, 4, 128, 11), (2, 300, 4, 2, 64, 12)):
        B, T, Hq, Hkv, D, seed = case
        print("case noalloc causal", case, "layout", lay, flush=True)
        (ref, got), (q, k, v, _) = _pair(B, T, Hq, Hkv, D, lay, seed)
        assert np.array_equal(ref.view(dtype=__import__("torch").int16).numpy(),
                              got.view(dtype=__import__("torch").int16).numpy())
        err = rel_frob(got.float().numpy().astype(np.float64),
                       oracle_replay_attention(q, k, v, None, kv_layout=lay))
        print("  bit-exact with mot_replay_attention; rel-Frobenius vs oracle %.3e" % err, flush=True)
        assert err <= TOL["bf16"]


def test_noalloc_with_key_sets(oracle_built):
    (ref, got), _ = _pair(1, 260, 8, 2, 128, 0, 13, S=64)
    import torch
    assert torch.equal(ref.view(torch.int16), got.view(torch.int16))
