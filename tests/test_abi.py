"""CPU tests of the C-ABI boundary: the library loads, exports every symbol
the header declares, and rejects bad arguments before touching the GPU
(nothing here launches a kernel)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2607_28979_amd import binding as mb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mot.h")

FAKE = 0x7F0000000000       # 16-byte aligned address that is never dereferenced


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(mb.lib_path()):
        pytest.skip("libmot.so not built (run __graft_entry__.build())")
    return mb.load_library()


def _decls():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(mot_[A-Za-z_]+)\s*\(", txt)))


def test_exports_every_declared_symbol(lib):
    names = _decls()
    assert set(mb.EXPORTED) == set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_abi_version(lib):
    assert mb.abi_version() == 5


def test_status_strings(lib):
    for code, name in mb.STATUS.items():
        assert mb.status_string(code) == name


@pytest.mark.parametrize("L_src,L_tgt", [(24, 28), (28, 28), (12, 12), (28, 24), (1, 7), (256, 3)])
def test_depth_ratio_map_bit_exact_vs_oracle(lib, oracle_built, L_src, L_tgt):
    from oracle import oracle_depth_ratio_map
    assert np.array_equal(mb.depth_ratio_map(L_src, L_tgt), oracle_depth_ratio_map(L_src, L_tgt))


def test_depth_ratio_map_rejects(lib):
    with pytest.raises(mb.MotError) as e:
        mb.depth_ratio_map(0, 4)
    assert e.value.name == "MOT_ERR_BAD_SHAPE"


def _shapes(**kw):
    base = dict(L_src=2, L_tgt=2, B=1, T=8, H_src=2, D_src=64, H_tgt=2, D_tgt=64, E=4, hidden=128,
                dtype=mb.MOT_BF16)
    base.update(kw)
    return mb.Shapes(**base)


def _call(shapes, layer_map=(0, 1), ptrs=None, ws=None, ws_bytes=0):
    p = dict(src_k=FAKE, src_v=FAKE + (1 << 30), w1=FAKE + (2 << 30), b1=None, w2=FAKE + (3 << 30),
             b2=None, wr=FAKE + (4 << 30), br=None, dst_k=FAKE + (5 << 30), dst_v=FAKE + (6 << 30))
    p.update(ptrs or {})
    mb.translate_raw(p["src_k"], p["src_v"], layer_map, p["w1"], p["b1"], p["w2"], p["b2"], p["wr"],
                     p["br"], p["dst_k"], p["dst_v"], shapes, workspace=ws, workspace_bytes_=ws_bytes)


def _expect(code, **kw):
    with pytest.raises(mb.MotError) as e:
        _call(**kw)
    assert e.value.name == code, str(e.value)


def test_null_pointers(lib):
    _expect("MOT_ERR_NULL_ARG", shapes=_shapes(), ptrs={"src_k": None})
    _expect("MOT_ERR_NULL_ARG", shapes=_shapes(), ptrs={"dst_v": None})
    _expect("MOT_ERR_NULL_ARG", shapes=_shapes(), ptrs={"w1": None})
    _expect("MOT_ERR_NULL_ARG", shapes=_shapes(), ptrs={"wr": None})


@pytest.mark.parametrize("kw", [dict(L_src=0), dict(L_tgt=257), dict(B=-1), dict(E=0), dict(E=17),
                                dict(hidden=0), dict(dtype=7), dict(src_layout=2), dict(act=5),
                                dict(algo=9), dict(top_k=5), dict(top_k=-1)])
def test_bad_shapes(lib, kw):
    _expect("MOT_ERR_BAD_SHAPE", shapes=_shapes(**kw), layer_map=[0] * 300)


@pytest.mark.parametrize("kw", [dict(D_src=60), dict(hidden=96),
                                dict(H_tgt=1, D_tgt=24), dict(dtype=mb.MOT_F32, D_src=6, H_src=2),
                                dict(algo=mb.ALGO_FUSED, dtype=mb.MOT_F32),
                                dict(algo=mb.ALGO_FUSED, H_src=12, D_src=64)])
def test_unsupported(lib, kw):
    _expect("MOT_ERR_UNSUPPORTED", shapes=_shapes(**kw))


@pytest.mark.parametrize("lm", [(0, 2), (-2, 0), (5, 5)])
def test_bad_layer_map(lib, lm):
    _expect("MOT_ERR_BAD_LAYER_MAP", shapes=_shapes(), layer_map=lm)


def test_misaligned(lib):
    _expect("MOT_ERR_MISALIGNED", shapes=_shapes(), ptrs={"src_k": FAKE + 8})
    _expect("MOT_ERR_MISALIGNED", shapes=_shapes(), ptrs={"w2": FAKE + 4})
    _expect("MOT_ERR_MISALIGNED", shapes=_shapes(), ptrs={"b1": FAKE + 1})


def test_overlapping_destinations(lib):
    _expect("MOT_ERR_BAD_SHAPE", shapes=_shapes(), ptrs={"dst_v": FAKE + (5 << 30) + 64})
    _expect("MOT_ERR_BAD_SHAPE", shapes=_shapes(), ptrs={"dst_k": FAKE})


def test_workspace_too_small(lib):
    s = _shapes(algo=mb.ALGO_UNFUSED)
    need = mb.workspace_bytes(s)
    assert need > 0
    _expect("MOT_ERR_WORKSPACE_TOO_SMALL", shapes=s, ws=FAKE + (7 << 30), ws_bytes=1024)


def test_workspace_bytes(lib):
    assert mb.workspace_bytes(_shapes()) == 0                    # fused: none
    s = _shapes(algo=mb.ALGO_UNFUSED)
    n_pad = 128
    gates = (4 * n_pad * 4 * 4 + 255) // 256 * 256                # 4 units, E=4, fp32
    hid = n_pad * 4 * 128 * 2
    assert mb.workspace_bytes(s) == gates + 4 * hid
    with pytest.raises(mb.MotError):
        mb.workspace_bytes(_shapes(E=0))


def test_streams_field(lib):
    """streams selects one activation stream (MoT-h) or keys and values."""
    _expect("MOT_ERR_BAD_SHAPE", shapes=_shapes(streams=3))
    _expect("MOT_ERR_BAD_SHAPE", shapes=_shapes(streams=-1))
    one, two = (mb.workspace_bytes(_shapes(algo=mb.ALGO_UNFUSED, streams=n)) for n in (1, 2))
    assert 0 < one < two
    _expect("MOT_ERR_NULL_ARG", shapes=_shapes(streams=2), ptrs={"src_v": None})


def _restore(ptrs=None, lm=None, **kw):
    base = dict(L=2, B=1, T=8, d_act=128, H_tgt=2, D_tgt=64, dtype=mb.MOT_BF16, dst_layout=0)
    base.update(kw)
    p = dict(act=FAKE, wk=FAKE + (1 << 30), bk=None, wv=FAKE + (2 << 30), bv=None,
             dst_k=FAKE + (3 << 30), dst_v=FAKE + (4 << 30))
    p.update(ptrs or {})
    c = mb._RestoreShapes(*[base[k] for k in ("L", "B", "T", "d_act", "H_tgt", "D_tgt", "dtype",
                                              "dst_layout")])
    arr = None if lm is None else np.ascontiguousarray(lm, dtype=np.int32)
    mb._check(mb.load_library().mot_restore_kv(p["act"], None if arr is None else arr.ctypes.data,
                                               p["wk"], p["bk"], p["wv"], p["bv"], p["dst_k"], p["dst_v"],
                                               ctypes.byref(c), None))


@pytest.mark.parametrize("kw,code", [
    (dict(L=0), "MOT_ERR_BAD_SHAPE"), (dict(L=257), "MOT_ERR_BAD_SHAPE"), (dict(T=-1), "MOT_ERR_BAD_SHAPE"),
    (dict(d_act=0), "MOT_ERR_BAD_SHAPE"), (dict(dst_layout=2), "MOT_ERR_BAD_SHAPE"),
    (dict(dtype=5), "MOT_ERR_BAD_SHAPE"), (dict(dtype=mb.MOT_F32), "MOT_ERR_UNSUPPORTED"),
    (dict(d_act=96), "MOT_ERR_UNSUPPORTED"), (dict(D_tgt=12), "MOT_ERR_UNSUPPORTED")])
def test_restore_rejects_shapes(lib, kw, code):
    with pytest.raises(mb.MotError) as e:
        _restore(**kw)
    assert e.value.name == code, str(e.value)


@pytest.mark.parametrize("ptrs,code", [
    (dict(act=None), "MOT_ERR_NULL_ARG"), (dict(dst_v=None), "MOT_ERR_NULL_ARG"),
    (dict(wk=FAKE + (1 << 30) + 8), "MOT_ERR_MISALIGNED"), (dict(bv=FAKE + 1), "MOT_ERR_MISALIGNED"),
    (dict(dst_v=FAKE + (3 << 30) + 256), "MOT_ERR_BAD_SHAPE"),      # dst_v inside dst_k
    (dict(dst_k=FAKE + 64), "MOT_ERR_BAD_SHAPE")])                  # dst_k inside act
def test_restore_rejects_pointers(lib, ptrs, code):
    with pytest.raises(mb.MotError) as e:
        _restore(ptrs=ptrs)
    assert e.value.name == code, str(e.value)


def test_restore_empty_is_a_no_op(lib):
    _restore(T=0, ptrs=dict(act=None, dst_k=None))     # nothing to do: no pointer is read


def _bb_raw(shapes, d_h, n_heads, d_ff):
    lm = np.array([0, 1], np.int32)
    rw = mb._RW(None, None)
    c = shapes.c()
    mb._check(mb.load_library().mot_backbone_translate(None, None, lm.ctypes.data, None, ctypes.byref(rw), None,
                                                       None, ctypes.byref(c),
                                                       ctypes.byref(mb._BackboneDims(d_h, n_heads, d_ff)), None))


def test_backbone_rejects(lib):
    """Shape checks of mot_backbone_translate run before any pointer is used."""
    s = _shapes(H_tgt=2, D_tgt=64)
    for sh, dh, nh, code in ((mb.Shapes(**{**s.__dict__, "dst_layout": 1}), 128, 2, "MOT_ERR_UNSUPPORTED"),
                             (s, 128, 4, "MOT_ERR_UNSUPPORTED"),          # head width 32
                             (s, 96, 1, "MOT_ERR_UNSUPPORTED"),           # d_h not a multiple of 64
                             (s, 128, 3, "MOT_ERR_BAD_SHAPE"),            # d_h not a multiple of n_heads
                             (mb.Shapes(**{**s.__dict__, "dtype": mb.MOT_F32, "D_src": 64}), 128, 2,
                              "MOT_ERR_UNSUPPORTED")):
        with pytest.raises(mb.MotError) as e:
            _bb_raw(sh, dh, nh, 256)
        assert e.value.name == code, (code, str(e.value))
    with pytest.raises(mb.MotError) as e:
        _bb_raw(s, 128, 2, 256)
    assert e.value.name == "MOT_ERR_NULL_ARG"
    assert mb.backbone_param_count(s, 128, 2, 256) > 0


def test_header_struct_layout_matches_binding(tmp_path):
    """sizeof and every field offset of the header's structs, as a C compiler
    lays them out, equal the ctypes mirrors in the binding."""
    import subprocess
    structs = {"mot_shapes": mb._Shapes, "mot_restore_shapes": mb._RestoreShapes,
               "mot_translator_weights": mb._TW, "mot_router_weights": mb._RW,
               "mot_replay_shapes": mb._ReplayShapes, "mot_backbone_dims": mb._BackboneDims}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "mot.h"', "int main(void) {"]
    for cname, cls in structs.items():
        lines.append('printf("%s size %%zu\\n", sizeof(%s));' % (cname, cname))
        for f, _ in cls._fields_:
            lines.append('printf("%s %s %%zu\\n", offsetof(%s, %s));' % (cname, f, cname, f))
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-D__HIP_PLATFORM_AMD__", "-I", os.path.dirname(HEADER),
                    "-I", "/opt/rocm/include", str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l.strip()}
    for cname, cls in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(cls), cname
        for f, _ in cls._fields_:
            assert got[(cname, f)] == getattr(cls, f).offset, (cname, f)


def test_bench_refuses_several_gpus():
    """bench.py measures one GPU: --gpus above 1 exits with status 2 and says why."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(os.path.dirname(HEADER), "..", "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr or "single" in r.stderr


def test_empty_contexts_are_no_ops(lib):
    """B*T == 0 returns MOT_OK without reading any pointer, for every entry point."""
    c = mb._ReplayShapes(1, 0, 4, 2, 128, 32, 0)
    mb._check(mb.load_library().mot_topS_select(None, None, ctypes.byref(c), None))
    mb._check(mb.load_library().mot_replay_attention(None, None, None, None, None, ctypes.byref(c), None))
    mb._check(mb.load_library().mot_replay_attention(None, None, None, FAKE, None, ctypes.byref(c), None))
    _bb_raw(_shapes(H_tgt=2, D_tgt=64, T=0), 128, 2, 256)


@pytest.mark.parametrize("kw,code", [
    (dict(S=48), "MOT_ERR_UNSUPPORTED"), (dict(S=256), "MOT_ERR_UNSUPPORTED"),    # D = 128: at most 192
    (dict(S=224), "MOT_ERR_UNSUPPORTED"), (dict(D=64, S=288), "MOT_ERR_UNSUPPORTED"),
    (dict(D=96), "MOT_ERR_UNSUPPORTED"), (dict(H_q=6, H_kv=4), "MOT_ERR_BAD_SHAPE"),
    (dict(H_q=34, H_kv=2), "MOT_ERR_UNSUPPORTED"), (dict(kv_layout=3), "MOT_ERR_BAD_SHAPE"),
    (dict(T=-1), "MOT_ERR_BAD_SHAPE"), (dict(H_q=8192, H_kv=8192), "MOT_ERR_UNSUPPORTED")])
def test_replay_rejects(lib, kw, code):
    base = dict(B=1, T=8, H_q=4, H_kv=2, D=128, S=32, kv_layout=0)
    base.update(kw)
    c = mb._ReplayShapes(*[base[k] for k in ("B", "T", "H_q", "H_kv", "D", "S", "kv_layout")])
    with pytest.raises(mb.MotError) as e:
        mb._check(mb.load_library().mot_replay_attention(FAKE, FAKE + (1 << 30), FAKE + (2 << 30), FAKE + (3 << 30),
                                                         FAKE + (4 << 30), ctypes.byref(c), None))
    assert e.value.name == code, str(e.value)


def test_topS_rejects(lib):
    c = mb._ReplayShapes(1, 70000, 1, 1, 128, 32, 0)
    with pytest.raises(mb.MotError) as e:
        mb._check(mb.load_library().mot_topS_select(FAKE, FAKE + (1 << 40), ctypes.byref(c), None))
    assert e.value.name == "MOT_ERR_UNSUPPORTED"
    c = mb._ReplayShapes(1, 64, 1, 1, 128, 32, 0)
    with pytest.raises(mb.MotError) as e:
        mb._check(mb.load_library().mot_topS_select(FAKE + 2, FAKE + (1 << 40), ctypes.byref(c), None))
    assert e.value.name == "MOT_ERR_MISALIGNED"
    with pytest.raises(mb.MotError) as e:
        mb._check(mb.load_library().mot_topS_select(FAKE, FAKE + 64, ctypes.byref(c), None))   # idx inside A
    assert e.value.name == "MOT_ERR_BAD_SHAPE"


_ENUM_SRC = r"""
#include <stdio.h>
#include "replay_limits.h"
using namespace mot;
int main() {
    for (int D = 64; D <= 128; D += 64)
        for (int S = 1; S <= 320; ++S) {
            const int sc = S / 8, m = replay_swizzle_mask(sc > 0 ? sc : 1);
            int perm = S % 8 == 0;                 /* every row: c -> c ^ (d & m) permutes 0..sc-1 */
            for (int d = 0; perm && d < D; ++d) {
                unsigned char seen[64] = {0};
                for (int c = 0; c < sc; ++c) {
                    const int t = c ^ (d & m);
                    if (t < 0 || t >= sc || seen[t]) { perm = 0; break; }
                    seen[t] = 1;
                }
            }
            const int inst = replay_sparse_instance(D, S);
            const int cover = replay_sparse_v_items(D, inst) * 256 >= (S / 2) * (D / 8) &&
                              replay_sparse_key_blocks(inst) * 4 >= (S + 15) / 16 && S <= inst;
            printf("%d %d %d %d %d %d\n", D, S, (int)replay_sparse_supported(D, S), perm, cover,
                   (int)replay_sparse_lds_bytes(D, S));
        }
    return 0;
}
"""


def test_replay_set_sizes_and_swizzle(lib, tmp_path):
    """Every (D, S) that mot_replay_attention admits with a key set has (i)
    an LDS swizzle that permutes the 16-byte chunks inside each row of S keys,
    (ii) register arrays in the dispatched instantiation that cover all S
    keys, and (iii) LDS within 64 KB.  The limits are read from the header the
    kernel and the host check share, compiled here as host-only C++; the
    admitted set comes from the library itself (the argument check runs
    before any device access, so NULL buffers give MOT_ERR_NULL_ARG exactly
    when the sizes are admitted).  Regression: a mask of SC - 1 moved chunks
    into the neighbouring row for S = 96, 160, 192, 224."""
    import subprocess
    src = tmp_path / "enum.cpp"
    exe = tmp_path / "enum"
    src.write_text(_ENUM_SRC)
    subprocess.run(["g++", "-std=c++17", "-O1", "-I", os.path.join(ROOT, "paper_2607_28979_amd", "csrc"),
                    str(src), "-o", str(exe)], check=True)
    rows = [tuple(int(v) for v in l.split()) for l in
            subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n") if l.strip()]
    admitted = set()
    for D, S, supported, perm, cover, lds in rows:
        c = mb._ReplayShapes(1, 4, 2, 1, D, S, 0)
        st = mb.load_library().mot_replay_attention(None, None, None, FAKE, None, ctypes.byref(c), None)
        name = mb.STATUS[st]
        assert name in ("MOT_ERR_NULL_ARG", "MOT_ERR_UNSUPPORTED", "MOT_ERR_BAD_SHAPE"), (D, S, name)
        assert (name == "MOT_ERR_NULL_ARG") == bool(supported), (D, S, name)
        if supported:
            admitted.add((D, S))
            assert perm and cover and lds <= 65536, (D, S, perm, cover, lds)
    assert admitted == {(64, s) for s in range(32, 257, 32)} | {(128, s) for s in range(32, 193, 32)}
    # the old mask (SC - 1) is not a row permutation for these sizes: the test has teeth
    for S in (96, 160, 192, 224):
        sc = S // 8
        assert any(sorted(c ^ (d & (sc - 1)) for c in range(sc)) != list(range(sc)) for d in range(64))


def test_workspace_size_queries(lib):
    """mot_replay_workspace_bytes: the V staging of the full causal path
    (B * H_kv * D * T rounded up to 64, bf16), 0 with key sets, SIZE_MAX for
    unsupported shapes; mot_backbone_workspace_bytes is positive for valid
    backbone shapes and SIZE_MAX otherwise."""
    assert mb.replay_workspace_bytes(2, 100, 8, 2, 128) == 2 * 2 * 128 * 128 * 2
    assert mb.replay_workspace_bytes(1, 64, 4, 4, 64, S=32, with_sets=True) == 0
    with pytest.raises(mb.MotError):
        mb.replay_workspace_bytes(1, 64, 4, 4, 96)
    # the causal kernel addresses a batch row's K rows with 32-bit byte
    # offsets: (T + 64) * H_kv * D * 2 < 2^31 in BTHD (here H_kv * D = 256)
    t_max = (1 << 31) // (256 * 2) - 64 - 1
    assert mb.replay_workspace_bytes(1, t_max, 4, 2, 128) == 2 * 128 * (-(-t_max // 64) * 64) * 2
    with pytest.raises(mb.MotError, match="2 GiB"):
        mb.replay_workspace_bytes(1, t_max + 1, 4, 2, 128)
    s = _shapes(H_tgt=2, D_tgt=64, T=70)
    n = mb.backbone_workspace_bytes(s, 128, 2, 256)
    assert n > 70 * (64 * 2 + 128 * 2 * 9 + 256 * 2 + 128 * 4)   # B = 1: every activation row once
    with pytest.raises(mb.MotError):
        mb.backbone_workspace_bytes(s, 96, 2, 256)


def test_usage_argument_checks(lib):
    """mot_usage_stats rejects E outside 1..MOT_MAX_EXPERTS, NULL and
    misaligned buffers before any launch; n = 0 is a no-op.  mot_translate
    rejects a usage array that is not 4-byte aligned or overlaps a
    destination cache."""
    L = mb.load_library()
    c8, d8 = FAKE, FAKE + (1 << 30)
    assert mb.STATUS[L.mot_usage_stats(None, 0, 4, None, None, None)] == "MOT_OK"
    for n, E, a, b, c, code in ((3, 0, c8, d8, d8 + 64, "MOT_ERR_BAD_SHAPE"),
                                (3, 17, c8, d8, d8 + 64, "MOT_ERR_BAD_SHAPE"),
                                (3, 4, None, d8, d8 + 64, "MOT_ERR_NULL_ARG"),
                                (3, 4, c8 + 2, d8, d8 + 64, "MOT_ERR_MISALIGNED"),
                                (3, 4, c8, d8 + 4, d8 + 64, "MOT_ERR_MISALIGNED"),
                                (3, 4, c8, d8, d8 + 8, "MOT_ERR_BAD_SHAPE")):
        assert mb.STATUS[L.mot_usage_stats(a, n, E, b, c, None)] == code, (n, E, code)
    s = _shapes(top_k=2)
    lm = np.array([0, 1], np.int32)
    for usage, code in ((FAKE + (7 << 30) + 2, "MOT_ERR_MISALIGNED"), (FAKE + (5 << 30), "MOT_ERR_BAD_SHAPE")):
        with pytest.raises(mb.MotError) as e:
            mb.translate_raw(FAKE, FAKE + (1 << 30), lm, FAKE + (2 << 30), None, FAKE + (3 << 30), None,
                             FAKE + (4 << 30), None, FAKE + (5 << 30), FAKE + (6 << 30), s, usage=usage)
        assert e.value.name == code


def test_noalloc_replay_rejects_oversized_staging(lib):
    """mot_replay_attention_noalloc refuses a full causal call whose staged V
    exceeds its 32 MiB static scratch (1 x 65536 positions x 4 KV heads of 128
    = 64 MiB) with MOT_ERR_WORKSPACE_TOO_SMALL, before touching the device;
    it applies the same argument checks as mot_replay_attention."""
    L = mb.load_library()
    big = mb._ReplayShapes(1, 65536, 8, 4, 128, 0, 0)
    st = L.mot_replay_attention_noalloc(FAKE, FAKE + (1 << 34), FAKE + (2 << 34), None, FAKE + (3 << 34),
                                        ctypes.byref(big), None)
    assert mb.STATUS[st] == "MOT_ERR_WORKSPACE_TOO_SMALL", mb.load_library().mot_last_error()
    bad = mb._ReplayShapes(1, 64, 8, 4, 96, 0, 0)
    assert mb.STATUS[L.mot_replay_attention_noalloc(FAKE, FAKE, FAKE, None, FAKE, ctypes.byref(bad), None)] == \
        "MOT_ERR_UNSUPPORTED"


def test_backbone_window_checks(lib, oracle_built):
    """Channel windows of the backbone: n_slots outside 0..8 and an L_tgt
    that is not a multiple of the window are refused; a window that mixes
    mapped and unmapped slots is MOT_ERR_BAD_LAYER_MAP; the packed parameter
    count matches the oracle's for every window size."""
    from oracle import oracle_backbone_window_param_count
    L = mb.load_library()
    s = _shapes(L_src=2, L_tgt=4, H_tgt=2, D_tgt=64)
    rw = mb._RW(FAKE + (4 << 30), None)

    def call(lm, n_slots):
        lm = np.ascontiguousarray(lm, np.int32)
        c = s.c()
        st = L.mot_backbone_translate(FAKE, FAKE + (1 << 30), lm.ctypes.data, FAKE + (2 << 30), ctypes.byref(rw),
                                      FAKE + (5 << 30), FAKE + (6 << 30), ctypes.byref(c),
                                      ctypes.byref(mb._BackboneDims(128, 2, 256, n_slots)), None)
        return mb.STATUS[st]

    assert call([0, 1, 0, 1], 9) == "MOT_ERR_BAD_SHAPE"
    assert call([0, 1, 0, 1], 3) == "MOT_ERR_BAD_SHAPE"        # 4 layers, windows of 3
    assert call([0, -1, 0, 1], 2) == "MOT_ERR_BAD_LAYER_MAP"   # window 0 half mapped
    for n_slots in (0, 1, 2, 4):
        want = oracle_backbone_window_param_count(128, 128, 256, 128, max(1, n_slots))
        assert mb.backbone_param_count(s, 128, 2, 256, n_slots) == want
