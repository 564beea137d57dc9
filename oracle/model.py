"""Target decoder and SpecBlock drafter forward over explicit rows (oracle).

Test infrastructure: see the package docstring.

A *row* is one query position run through the network.  Every row carries
its RoPE position, the slot its K/V occupy in a per-call (or per-iteration)
*segment*, and the list of segment slots it may attend to.  On top of that,
every row sees a *prefix* of committed K/V entries in full.  This one form
covers causal prefill (a chain), tree verification (ancestor-or-self sets) and
the drafter's block attention (prefix + on-path rows of earlier blocks + own
block causal).
"""
from __future__ import annotations

import numpy as np

from .numerics import Numerics, attend, rmsnorm, rope, silu

LAYER_KEYS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wg", "wu",
              "wd")


def f64(raw: dict, prefix: str, keys) -> dict:
    return {k: np.asarray(raw[prefix + k], dtype=np.float64) for k in keys}


class Segment:
    """K/V of the rows of one call or iteration, per layer: [cap, Hkv, hd]."""

    def __init__(self, n_layers: int, cap: int, n_kv: int, hd: int):
        self.k = [np.zeros((cap, n_kv, hd)) for _ in range(n_layers)]
        self.v = [np.zeros((cap, n_kv, hd)) for _ in range(n_layers)]


class Prefix:
    """Committed K/V entries, per layer: [T, Hkv, hd] (all visible)."""

    def __init__(self, n_layers: int, n_kv: int, hd: int):
        self.k = [np.zeros((0, n_kv, hd)) for _ in range(n_layers)]
        self.v = [np.zeros((0, n_kv, hd)) for _ in range(n_layers)]

    def __len__(self):
        return self.k[0].shape[0]

    def append(self, layer: int, k, v):
        self.k[layer] = np.concatenate([self.k[layer], k[None]], axis=0)
        self.v[layer] = np.concatenate([self.v[layer], v[None]], axis=0)


def decoder_layer(lw, x, pos, slots, vis, prefix_k, prefix_v, seg_k, seg_v,
                  shape, num: Numerics):
    """One pre-norm Llama decoder layer over rows.

    x: residual stream entering the layer [R, d].  The rows' K/V are written
    to ``seg_k/seg_v[slots]`` before attention, so a row can see itself and
    any row of the same call listed in ``vis[r]``.
    """
    R = x.shape[0]
    H, Hkv, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    a = num.act(rmsnorm(x, lw["attn_norm"], shape.norm_eps))
    q = (a @ lw["wq"].T).reshape(R, H, hd)
    k = (a @ lw["wk"].T).reshape(R, Hkv, hd)
    v = (a @ lw["wv"].T).reshape(R, Hkv, hd)
    q = num.act(rope(q, pos, shape.rope_theta))
    k = num.act(rope(k, pos, shape.rope_theta))
    v = num.act(v)
    seg_k[slots] = k
    seg_v[slots] = v
    o = np.empty((R, H * hd))
    for r in range(R):
        sel = np.asarray(vis[r], dtype=np.int64)
        keys = np.concatenate([prefix_k, seg_k[sel]], axis=0)
        vals = np.concatenate([prefix_v, seg_v[sel]], axis=0)
        o[r] = attend(q[r], keys, vals)
    x = x + num.act(o) @ lw["wo"].T
    m = num.act(rmsnorm(x, lw["mlp_norm"], shape.norm_eps))
    u = num.act(silu(m @ lw["wg"].T) * (m @ lw["wu"].T))
    return x + u @ lw["wd"].T


class Target:
    """Llama-style target model M (pre-RMSNorm, rotate-half RoPE, SwiGLU,
    grouped-query attention, untied LM head, no biases)."""

    def __init__(self, raw: dict, shape, dtype: str, tap_layers):
        self.shape = shape
        self.num = Numerics(dtype)
        self.embed = np.asarray(raw["embed"], dtype=np.float64)
        self.layers = [f64(raw, f"layers.{i}.", LAYER_KEYS)
                       for i in range(shape.n_layers)]
        self.final_norm = np.asarray(raw["final_norm"], dtype=np.float64)
        self.lm_head = np.asarray(raw["lm_head"], dtype=np.float64)
        self.tap_layers = tuple(tap_layers)

    def new_prefix(self) -> Prefix:
        s = self.shape
        return Prefix(s.n_layers, s.n_kv_heads, s.head_dim)

    def new_segment(self, cap: int) -> Segment:
        s = self.shape
        return Segment(s.n_layers, cap, s.n_kv_heads, s.head_dim)

    def forward(self, tokens, pos, slots, vis, prefix: Prefix, seg: Segment):
        """Run rows through the target.

        Returns (logits [R, V], taps [R, 3, d]) where taps are the residual
        stream after the low / mid / top tap layers (pre final norm).
        """
        x = self.embed[np.asarray(tokens)]
        by_layer = {}
        for i, lw in enumerate(self.layers):
            x = decoder_layer(lw, x, np.asarray(pos), slots, vis,
                              prefix.k[i], prefix.v[i], seg.k[i], seg.v[i],
                              self.shape, self.num)
            by_layer[i] = x
        taps = np.stack([by_layer[i] for i in self.tap_layers], axis=1)
        h = self.num.act(rmsnorm(x, self.final_norm, self.shape.norm_eps))
        return h @ self.lm_head.T, taps


class Drafter:
    """SpecBlock drafter D_theta (Sec. 3.1).

    Readings taken here:
    * norm() in Eq. 2 is RMSNorm with its own gain per input;
    * one W_shift per decoder layer, applied to the state entering that
      layer, including the first (so an L = 1 drafter still carries the
      shift of Eq. 3); the shifted state replaces the layer's input;
    * a final RMSNorm precedes the drafter LM head; the cached h^(L) is the
      pre-norm state;
    * the drafter shares the target's token embedding (the paper freezes the
      drafter's embedding at the target's); its LM head covers the target's
      vocabulary or a reduced one (App. A: the most frequent target tokens)
      whose ids map to target ids through ``d2t`` (strictly increasing, so
      "smaller id" means the same in both numberings).
    """

    def __init__(self, raw: dict, shape, dtype: str, n_layers: int,
                 embed: np.ndarray):
        self.shape = shape
        self.num = Numerics(dtype)
        self.embed = embed
        g = lambda k: np.asarray(raw["d." + k], dtype=np.float64)  # noqa: E731
        self.w_cond = g("w_cond")
        self.norm_c, self.norm_e, self.norm_q = g("norm_c"), g("norm_e"), g(
            "norm_q")
        self.pos_query = g("pos_query")
        self.w_fuse = g("w_fuse")
        self.shift = [g(f"layers.{i}.w_shift") for i in range(n_layers)]
        self.layers = [f64(raw, f"d.layers.{i}.", LAYER_KEYS)
                       for i in range(n_layers)]
        self.final_norm = g("final_norm")
        self.lm_head = g("lm_head")
        self.d2t = (np.asarray(raw["d.d2t"], dtype=np.int64)
                    if "d.d2t" in raw else None)
        self.rank_w = g("rank_w")
        self.rank_b = g("rank_b")
        self.n_layers = n_layers

    def new_prefix(self) -> Prefix:
        s = self.shape
        return Prefix(self.n_layers, s.n_kv_heads, s.head_dim)

    def new_segment(self, cap: int) -> Segment:
        s = self.shape
        return Segment(self.n_layers, cap, s.n_kv_heads, s.head_dim)

    def to_target(self, ids) -> np.ndarray:
        """Target token ids of drafter output ids."""
        ids = np.asarray(ids, dtype=np.int64)
        return ids if self.d2t is None else self.d2t[ids]

    def cond_from_taps(self, taps3):
        """Eq. 1: c = W_cond [h_low, h_mid, h_top] (taps3: [3, d])."""
        return self.num.act(np.asarray(taps3).reshape(-1)) @ self.w_cond.T

    def forward(self, conds, tokens, row_start, row_k, row_pred, pos, slots,
                vis, prefix: Prefix, seg: Segment):
        """Block forward over rows (Eq. 2, Eq. 3, decoder layers, LM head).

        conds [B, d] and tokens [B] describe the starts; row r belongs to
        start row_start[r] and block position row_k[r] (1-based), and its
        shift partner is row row_pred[r] of this call (itself when k = 1,
        the convention h_{t,0} = h_{t,1}).
        Returns (logits [R, Vd] over the drafter's vocabulary, h_last [R, d]).
        """
        eps = self.shape.norm_eps
        num = self.num
        conds = np.asarray(conds, dtype=np.float64)
        row_start = np.asarray(row_start)
        row_k = np.asarray(row_k)
        nc = rmsnorm(conds, self.norm_c, eps)
        ne = rmsnorm(self.embed[np.asarray(tokens)], self.norm_e, eps)
        nq = rmsnorm(self.pos_query, self.norm_q, eps)
        fused_in = np.concatenate(
            [nc[row_start], ne[row_start], nq[row_k - 1]], axis=1)
        h = num.act(fused_in) @ self.w_fuse.T                      # Eq. 2
        pred = np.asarray(row_pred)
        for i, lw in enumerate(self.layers):
            shifted = num.act(np.concatenate([h, h[pred]], axis=1))
            x = shifted @ self.shift[i].T                            # Eq. 3
            h = decoder_layer(lw, x, np.asarray(pos), slots, vis,
                              prefix.k[i], prefix.v[i], seg.k[i], seg.v[i],
                              self.shape, num)
        z = num.act(rmsnorm(h, self.final_norm, eps)) @ self.lm_head.T
        return z, h
