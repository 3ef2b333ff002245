"""Synthetic workload shapes for the KV-cache translation hot path.

Each workload is shaped like a source/target model pair whose context KV
caches the paper translates (Sec. 4 "Experimental Setup"; the model pairs of
Table "qwen25_combined" and App. E.2).  The translator body is a per-token
Linear(d_in -> hidden) - GELU - Linear(hidden -> d_out) MLP, the router is
Linear(d_in -> E) + softmax, and every token uses all E translators.

Value recipes (consumed by ``inputs.py``):
  key_sigma / val_sigma : per-(layer, channel) log-normal scale exp(sigma*N(0,1))
  key_outlier_frac / key_outlier_mult : fraction of token positions per batch
      row whose key rows are multiplied (attention-sink-like rows); position 0
      is always one of them.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import List, Optional


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str              # "f32" or "bf16"
    L_src: int
    L_tgt: int
    B: int
    T: int
    H_src: int
    D_src: int
    H_tgt: int
    D_tgt: int
    E: int
    hidden: int
    seed: int
    layer_map: str = "identity"      # "identity" or "depth_ratio"
    key_sigma: float = 0.0
    val_sigma: float = 0.0
    key_outlier_frac: float = 0.0
    key_outlier_mult: float = 1.0
    src_layout: int = 0
    dst_layout: int = 0
    top_k: int = 0                   # translators used per token; 0 = all E (dense)
    streams: int = 2                 # 2 = keys and values; 1 = one activation stream (MoT-h)

    @property
    def d_in(self) -> int:
        return self.H_src * self.D_src

    @property
    def d_out(self) -> int:
        return self.H_tgt * self.D_tgt

    @property
    def n_tok(self) -> int:
        return self.B * self.T

    def units(self) -> int:
        return self.streams * self.L_tgt

    def gemm_flops(self) -> float:
        """Algorithmic multiply-add flops of one full translation: router,
        first and second translator layers of the translators each token
        uses (all E, or its top_k), for every unit and token."""
        used = self.top_k if 0 < self.top_k < self.E else self.E
        per_tok_unit = 2.0 * (self.d_in * self.E + used * (self.d_in * self.hidden
                                                            + self.hidden * self.d_out))
        return per_tok_unit * self.n_tok * self.units()

    def alg_bytes(self) -> float:
        """Algorithmic HBM bytes: each distinct source layer read once, all
        weights read once, the translated cache written once."""
        es = 4 if self.dtype == "f32" else 2
        n_src_layers = self.L_src if self.layer_map != "identity" else min(self.L_src, self.L_tgt)
        src = self.streams * n_src_layers * self.n_tok * self.d_in * es
        w = self.units() * self.E * (self.hidden * self.d_in + self.hidden + self.d_out * self.hidden
                                     + self.d_out + self.d_in + 1) * es
        dst = self.units() * self.n_tok * self.d_out * es
        return float(src + w + dst)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS: List[Workload] = [
    Workload("gpt2-small->opt-125m", "f32", L_src=12, L_tgt=12, B=1, T=64, H_src=12, D_src=64,
             H_tgt=12, D_tgt=64, E=2, hidden=256, seed=0),
    Workload("qwen2.5-0.5b->qwen2.5-0.5b", "bf16", L_src=24, L_tgt=24, B=4, T=1024, H_src=2,
             D_src=64, H_tgt=2, D_tgt=64, E=4, hidden=512, seed=1, key_sigma=0.5, val_sigma=0.5),
    Workload("opt-1.3b->qwen2.5-1.5b", "bf16", L_src=24, L_tgt=28, B=8, T=2048, H_src=32,
             D_src=64, H_tgt=2, D_tgt=128, E=4, hidden=1024, seed=2, layer_map="depth_ratio"),
    Workload("qwen2.5-1.5b->qwen2.5-7b", "bf16", L_src=28, L_tgt=28, B=8, T=4096, H_src=2,
             D_src=128, H_tgt=4, D_tgt=128, E=8, hidden=2048, seed=3, key_sigma=1.0),
    Workload("qwen2.5-7b->qwen2.5-7b-32k", "bf16", L_src=28, L_tgt=28, B=1, T=32768, H_src=4,
             D_src=128, H_tgt=4, D_tgt=128, E=8, hidden=2048, seed=4, key_sigma=1.0,
             key_outlier_frac=0.01, key_outlier_mult=20.0),
]

BY_NAME = {w.name: w for w in WORKLOADS}

# the headline workload: Qwen2.5-1.5B -> Qwen2.5-7B, B=8, T=4096
HEADLINE = WORKLOADS[3]


@dataclass(frozen=True)
class MothWorkload:
    """The activation variant MoT-h (App. C.5): each layer's intermediate
    activation (width d_model) is translated as one stream, then the target's
    key and value projections (kv_heads x head_dim each) restore its cache."""
    act: Workload
    kv_heads: int
    head_dim: int

    @property
    def d_kv(self) -> int:
        return self.kv_heads * self.head_dim

    def restore_flops(self) -> float:
        return 2.0 * 2 * self.d_kv * self.act.d_out * self.act.n_tok * self.act.L_tgt


# Qwen2.5-1.5B (d_model 1536) -> Qwen2.5-7B (d_model 3584, 4 KV heads of 128),
# 28 -> 28 layers, B=8, T=4096; translator width and experts as the headline
MOTH = MothWorkload(
    Workload("qwen2.5-1.5b->qwen2.5-7b activations", "bf16", L_src=28, L_tgt=28, B=8, T=4096,
             H_src=1, D_src=1536, H_tgt=1, D_tgt=3584, E=8, hidden=2048, seed=5, streams=1),
    kv_heads=4, head_dim=128)


def small_variant(w: Workload, L_src: Optional[int] = None, L_tgt: Optional[int] = None,
                  B: Optional[int] = None, T: Optional[int] = None,
                  hidden: Optional[int] = None) -> Workload:
    """Same row dimensions, experts and value recipe; fewer layers/tokens so
    the oracle finishes in seconds.  Used by the parity tests."""
    return replace(w, L_src=L_src or w.L_src, L_tgt=L_tgt or w.L_tgt, B=B or w.B,
                   T=T or w.T, hidden=hidden or w.hidden)


@dataclass(frozen=True)
class ReplayWorkload:
    """Context replay after translation (App. C.4): every target layer
    attends over the context; the bottom L_full layers over the full causal
    prefix, the others over their Top-S source-guided key sets, chosen from
    the head-averaged attention map of the source layer the depth-ratio map
    pairs with them."""
    name: str
    L_src: int
    L_tgt: int
    B: int
    T: int
    H_q: int
    H_kv: int
    D: int
    S: int
    L_full: int
    seed: int

    def attention_flops(self) -> float:
        """2 (scores) + 2 (values) flops per (query head, key, head dim)."""
        sparse = (self.L_tgt - self.L_full) * self.B * sum(min(u + 1, self.S) for u in range(self.T))
        full = self.L_full * self.B * self.T * (self.T + 1) / 2
        return 4.0 * self.H_q * self.D * (sparse + full)


# Qwen2.5-1.5B source -> Qwen2.5-7B target (28 query heads on 4 KV heads of
# 128), one 8K-token context, S = 128, L_full = 2
REPLAY = ReplayWorkload("qwen2.5-1.5b->qwen2.5-7b replay, 8K context", L_src=28, L_tgt=28, B=1, T=8192,
                        H_q=28, H_kv=4, D=128, S=128, L_full=2, seed=6)


@dataclass(frozen=True)
class BackboneWorkload:
    """The Mixture-of-Translators with the backbone translator body (App.
    C.2) as its experts: the headline model pair's cache rows, translator
    width d_h, n_heads attention heads, FFN width d_ff, E experts."""
    kv: Workload
    d_h: int
    n_heads: int
    d_ff: int

    def flops(self, n_slots: int = 1) -> float:
        """Matrix flops of one call over channel windows of n_slots slots: per
        (window, K/V) unit and expert, for each slot the input projection, Q,
        K, V, output and FFN projections and causal attention (scores and
        values) within each batch row, then the target projection of the
        slots' concatenation; every expert runs on every token."""
        w, N = self.kv, n_slots
        per_tok = 2.0 * (N * (w.d_in * self.d_h + 4 * self.d_h * self.d_h + 2 * self.d_h * self.d_ff)
                         + (N * self.d_h) * (N * w.d_out))
        attn = N * 4.0 * self.d_h * w.B * w.T * (w.T + 1) / 2
        return w.units() // N * w.E * (per_tok * w.n_tok + attn)


# Qwen2.5-1.5B -> Qwen2.5-7B cache rows (256 -> 512), B = 8, T = 4096, two
# backbone experts (the paper's N_Tr = 2), both used per token
BACKBONE = BackboneWorkload(
    Workload("qwen2.5-1.5b->qwen2.5-7b backbone experts", "bf16", L_src=28, L_tgt=28, B=8, T=4096, H_src=2,
             D_src=128, H_tgt=4, D_tgt=128, E=2, hidden=256, seed=7, key_sigma=1.0),
    d_h=256, n_heads=2, d_ff=512)
