"""Brute-force scalar evaluation of the MoT translation for tiny shapes.

TEST INFRASTRUCTURE ONLY.  Pure Python (lists, ``math``), one token at a time,
used to pin the C oracle on shapes of 2 tokens and 2 channels.  It evaluates
every translator's full output first and mixes afterwards (the C oracle mixes
as it goes), and it indexes the caches through nested lists built from the
flat arrays rather than through stride arithmetic, so a stride or index slip
in either implementation shows up as a mismatch.

Paper: Sec. 3, Definition "Mixture-of-Translators" (Eq. mot_definition);
GELU is the paper's phi (App. C.2), taken as the exact erf form.
"""
from __future__ import annotations

import math


def _gelu(a: float) -> float:
    return a * 0.5 * (1.0 + math.erf(a / math.sqrt(2.0)))


def brute_translate(dims, src_k, src_v, layer_map, w1, b1, w2, b2, wr, br):
    """Returns {(j, x): [[out row] for each flattened token b*T+t]} for every
    mapped target layer; rows are python float lists of length d_out."""
    act = (lambda a: a) if dims.act == 1 else _gelu
    E, Hd = dims.E, dims.hidden
    top_k = dims.top_k or E
    res = {}
    srcs = (src_k.tolist(), src_v.tolist())
    W1, W2, WR = w1.tolist(), w2.tolist(), wr.tolist()
    B1 = b1.tolist() if b1 is not None else None
    B2 = b2.tolist() if b2 is not None else None
    BR = br.tolist() if br is not None else None
    for j in range(dims.L_tgt):
        i = int(layer_map[j])
        if i < 0:
            continue
        for x in range(2):
            rows = []
            for b in range(dims.B):
                for t in range(dims.T):
                    z = []
                    for h in range(dims.H_src):
                        for d in range(dims.D_src):
                            if dims.src_layout == 0:
                                z.append(srcs[x][i][b][t][h][d])
                            else:
                                z.append(srcs[x][i][b][h][t][d])
                    logits = []
                    for m in range(E):
                        v = sum(WR[j][x][m][c] * z[c] for c in range(len(z)))
                        if BR is not None:
                            v += BR[j][x][m]
                        logits.append(v)
                    mx = max(logits)
                    ex = [math.exp(v - mx) for v in logits]
                    g = [v / sum(ex) for v in ex]
                    order = sorted(range(E), key=lambda m: (-g[m], m))
                    chosen = sorted(order[:top_k])
                    norm = sum(g[m] for m in chosen)
                    experts = {}
                    for m in chosen:
                        hid = []
                        for k in range(Hd):
                            a = sum(W1[j][x][m][k][c] * z[c] for c in range(len(z)))
                            if B1 is not None:
                                a += B1[j][x][m][k]
                            hid.append(act(a))
                        y = []
                        for o in range(dims.H_tgt * dims.D_tgt):
                            v = sum(W2[j][x][m][o][k] * hid[k] for k in range(Hd))
                            if B2 is not None:
                                v += B2[j][x][m][o]
                            y.append(v)
                        experts[m] = y
                    out = [0.0] * (dims.H_tgt * dims.D_tgt)
                    for m in chosen:
                        for o in range(len(out)):
                            out[o] += (g[m] / norm) * experts[m][o]
                    rows.append(out)
            res[(j, x)] = rows
    return res
