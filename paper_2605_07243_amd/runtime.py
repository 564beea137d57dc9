"""Device-memory harness around libspecblock.so.

PyTorch is used for device memory and the stream only; every step of the
hot path runs in the library's HIP kernels (there is no fallback).  This
module allocates the caches, tree and output buffers the C ABI describes,
packs weights into the library's layout ([Wq; Wk; Wv] and [Wg; Wu] row
concatenations, bf16 projections fragment-packed by sb_pack_weight) and
marshals arguments.
"""
from __future__ import annotations

import ctypes as C
import zlib

import numpy as np
import torch

from . import binding as B


def _ptr(t):
    return C.c_void_p(t.data_ptr()) if t is not None else C.c_void_p(0)


def elem_dtype(dtype: str):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def device_normal(name: str, shape, seed: int, dtype: str, device,
                  std: float = 0.02):
    """Seeded N(0, std) tensor generated on the device (for model sizes
    whose host generation would dominate a run)."""
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1000003 + zlib.crc32(name.encode())) % (2 ** 63))
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    t.mul_(std)
    return t.to(elem_dtype(dtype))


class Runtime:
    """One SpecBlock context with its caches and buffers.

    weights: dict name -> array (the synth naming), host numpy or device
    tensors; ``None`` generates N(0, 0.02) weights on the device.
    """

    def __init__(self, w, weights=None, *, n_seqs=None, max_pages=None,
                 prefill_chunk=128, device="cuda", page_seed=3, seed=0,
                 adapt_cap=0, share_layers=False):
        self.lib = B.load()
        self.w = w
        self.dev = torch.device(device)
        s = w.target
        self.S = n_seqs or w.n_seqs
        self.Vd = w.draft_vocab or s.vocab
        if max_pages is None:
            max_pages = (max(w.prompt_len) + 64 * (w.M * w.K + 1) + 15) // 16
        self.max_pages = max_pages
        cfg = B.Config()
        cfg.target = B.ModelDims(s.n_layers, s.d_model, s.n_heads,
                                 s.n_kv_heads, s.head_dim, s.d_ff, s.vocab,
                                 s.rope_theta, s.norm_eps)
        cfg.drafter_layers = w.drafter_layers
        cfg.tap_layers[:] = list(w.tap_layers)
        cfg.K, cfg.M, cfg.B_max, cfg.budget = w.K, w.M, w.B_max, w.budget
        cfg.branch_map[:] = list(w.branch_map)
        cfg.dtype = B.SB_BF16 if w.dtype == "bf16" else B.SB_F32
        cfg.max_seqs = self.S
        cfg.page_size = 16
        cfg.max_pages = max_pages
        cfg.prefill_chunk = prefill_chunk
        cfg.draft_vocab = w.draft_vocab
        cfg.adapt_cap = adapt_cap
        self.cfg = cfg
        ctx = C.c_void_p()
        rc = self.lib.sb_create(C.byref(cfg), C.byref(ctx))
        if rc != B.SB_OK:
            raise B.SBError(rc, self.lib.sb_last_error(None).decode())
        self.ctx = ctx
        self.row_cap = self.lib.sb_row_capacity(C.byref(cfg))
        self.et = elem_dtype(w.dtype)
        # share_layers: every target layer's table entry points at layer 0's
        # device weights (full-depth tests whose oracle shares one layer)
        self.share_layers = share_layers
        self._weights(weights, seed)
        nbytes = self.lib.sb_workspace_bytes(C.byref(cfg))
        self.workspace = torch.empty(nbytes, dtype=torch.uint8,
                                     device=self.dev)
        B.check(self.lib, ctx, self.lib.sb_bind(
            ctx, C.byref(self.tw_c), C.byref(self.dw_c),
            _ptr(self.workspace), nbytes))
        self._buffers(page_seed)

    # ------------------------------------------------------------------
    def _weights(self, src, seed):
        w, s, dev = self.w, self.w.target, self.dev
        d, F = s.d_model, s.d_ff
        keep = []

        def get(name, shape, kind="normal", fp32=False):
            if src is not None:
                a = src[name]
                t = a if isinstance(a, torch.Tensor) else torch.from_numpy(
                    np.ascontiguousarray(a))
                t = t.to(dev)
                t = t.float() if (fp32 or kind != "normal") else t.to(self.et)
                return t.contiguous()
            if kind == "ones":
                return torch.ones(shape, dtype=torch.float32, device=dev)
            if kind == "zeros":
                return torch.zeros(shape, dtype=torch.float32, device=dev)
            t = device_normal(name, shape, seed, "f32" if fp32 else w.dtype,
                              dev)
            return t.float() if fp32 else t

        def pack(t, gate_up=False):
            """Projection matrix in the library's layout (bf16: fragment
            packed by sb_pack_weight; f32: unchanged)."""
            if self.et != torch.bfloat16:
                return t
            out = torch.empty_like(t)
            B.check(self.lib, None, self.lib.sb_pack_weight(
                _ptr(t), _ptr(out), t.shape[0], t.shape[1], B.SB_BF16,
                int(gate_up), C.c_void_p(
                    torch.cuda.current_stream(dev).cuda_stream)))
            return out

        def layer(prefix, drafter):
            qkv = torch.cat([get(prefix + "wq", (s.q_dim, d)),
                             get(prefix + "wk", (s.kv_dim, d)),
                             get(prefix + "wv", (s.kv_dim, d))]).contiguous()
            gu = torch.cat([get(prefix + "wg", (F, d)),
                            get(prefix + "wu", (F, d))]).contiguous()
            t = dict(attn_norm=get(prefix + "attn_norm", (d,), "ones"),
                     w_qkv=pack(qkv), w_o=pack(get(prefix + "wo", (d, s.q_dim))),
                     mlp_norm=get(prefix + "mlp_norm", (d,), "ones"),
                     w_gate_up=pack(gu, True),
                     w_down=pack(get(prefix + "wd", (d, F))),
                     w_shift=pack(get(prefix + "w_shift", (d, 2 * d)))
                     if drafter else None)
            del qkv, gu
            keep.append(t)
            return B.LayerWeights(*[_ptr(t[k]) for k in
                                    ("attn_norm", "w_qkv", "w_o", "mlp_norm",
                                     "w_gate_up", "w_down", "w_shift")])

        if self.share_layers:
            first = layer("layers.0.", False)
            tl = (B.LayerWeights * s.n_layers)(*([first] * s.n_layers))
        else:
            tl = (B.LayerWeights * s.n_layers)(*[layer(f"layers.{i}.", False)
                                                 for i in range(s.n_layers)])
        embed = get("embed", (s.vocab, d))
        tfin = get("final_norm", (d,), "ones")
        tlm = pack(get("lm_head", (s.vocab, d)))
        dl = (B.LayerWeights * w.drafter_layers)(
            *[layer(f"d.layers.{i}.", True) for i in range(w.drafter_layers)])
        dt = dict(w_cond=pack(get("d.w_cond", (d, 3 * d))),
                  norm_c=get("d.norm_c", (d,), "ones"),
                  norm_e=get("d.norm_e", (d,), "ones"),
                  norm_q=get("d.norm_q", (d,), "ones"),
                  pos_query=get("d.pos_query", (w.K, d)),
                  w_fuse=pack(get("d.w_fuse", (d, 3 * d))),
                  final_norm=get("d.final_norm", (d,), "ones"),
                  lm_head=pack(get("d.lm_head", (self.Vd, d))),
                  rank_w=get("d.rank_w", (4, d + 15), fp32=True),
                  rank_b=get("d.rank_b", (4,), "zeros"),
                  d2t=self._d2t(src, seed))
        self._keep = (keep, embed, tfin, tlm, dt, tl, dl)
        self.tw_c = B.TargetWeights(_ptr(embed), tl, _ptr(tfin), _ptr(tlm))
        self.dw_c = B.DrafterWeights(
            _ptr(dt["w_cond"]), _ptr(dt["norm_c"]), _ptr(dt["norm_e"]),
            _ptr(dt["norm_q"]), _ptr(dt["pos_query"]), _ptr(dt["w_fuse"]), dl,
            _ptr(dt["final_norm"]), _ptr(dt["lm_head"]), _ptr(dt["rank_w"]),
            _ptr(dt["rank_b"]), _ptr(dt["d2t"]))

    def _d2t(self, src, seed):
        """Drafter id -> target id map of a reduced drafter vocabulary (None
        for the full one): from the weights when given, else a seeded
        sorted random subset of the target vocabulary."""
        V, Vd = self.w.target.vocab, self.Vd
        if Vd == V:
            return None
        if src is not None:
            m = torch.as_tensor(np.asarray(src["d.d2t"], np.int32))
        else:
            g = torch.Generator().manual_seed(seed + 7)
            m = torch.randperm(V, generator=g)[:Vd].sort().values.to(
                torch.int32)
        return m.to(self.dev).contiguous()

    def _buffers(self, page_seed):
        w, s, dev, S = self.w, self.w.target, self.dev, self.S
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        d, V = s.d_model, s.vocab
        n_pages = S * self.max_pages
        rng = np.random.default_rng(page_seed)

        def pool(n_layers):
            # K pages [Hkv][16][hd]; V pages transposed [Hkv][hd][16]
            k = torch.zeros((n_layers, n_pages, s.n_kv_heads, 16, s.head_dim),
                            dtype=self.et, device=dev)
            v = torch.zeros((n_layers, n_pages, s.n_kv_heads, s.head_dim, 16),
                            dtype=self.et, device=dev)
            pt = torch.from_numpy(rng.permutation(n_pages).astype(
                np.int32).reshape(S, self.max_pages)).to(dev)
            return k, v, pt

        self.tk, self.tv, self.tpt = pool(s.n_layers)
        self.dk, self.dv, self.dpt = pool(w.drafter_layers)
        self.tkv_c = B.KV(_ptr(self.tk), _ptr(self.tv), _ptr(self.tpt),
                          s.n_layers, n_pages)
        self.dkv_c = B.KV(_ptr(self.dk), _ptr(self.dv), _ptr(self.dpt),
                          w.drafter_layers, n_pages)
        self.root = torch.zeros(S, **i32)
        self.T = torch.zeros(S, **i32)
        self.cond_taps = torch.zeros(S, 3, d, **f32)
        self.seqs_c = B.Seqs(S, _ptr(self.root), _ptr(self.T),
                             _ptr(self.cond_taps))
        bud, rc = w.budget, self.row_cap
        bw, rw = (bud + 31) // 32, (rc + 31) // 32
        self.tree = dict(
            n_nodes=torch.zeros(S, **i32), token=torch.zeros(S, bud, **i32),
            parent=torch.zeros(S, bud, **i32), depth=torch.zeros(S, bud, **i32),
            row=torch.zeros(S, bud, **i32), rank=torch.zeros(S, bud, **i32),
            logp=torch.zeros(S, bud, **f32), cum_logp=torch.zeros(S, bud, **f32),
            anc=torch.zeros(S, bud, bw, **i32), n_rows=torch.zeros(S, **i32),
            row_block=torch.zeros(S, rc, **i32),
            row_start=torch.zeros(S, rc, **i32),
            row_k=torch.zeros(S, rc, **i32), row_pos=torch.zeros(S, rc, **i32),
            row_vis=torch.zeros(S, rc, rw, **i32),
            h_last=torch.zeros(S, rc, d, **f32),
            n_starts=torch.zeros(S, **i32),
            starts=torch.zeros(S, w.B_max, **i32))
        self.tree_c = B.Tree(*[_ptr(self.tree[f]) for f in B.TREE_FIELDS])
        call_cap = S * w.B_max * w.K
        self.call_cap = call_cap
        self.dout = dict(
            topk_id=torch.zeros(S, rc, B.TOPK, **i32),
            topk_logit=torch.zeros(S, rc, B.TOPK, **f32),
            lse=torch.zeros(S, rc, **f32), psi=torch.zeros(S, rc, B.PSI_DIM, **f32),
            bucket=torch.zeros(S, rc, **i32), branch=torch.zeros(S, rc, **i32),
            logits=None, call_seq=torch.zeros(call_cap, **i32),
            call_row=torch.zeros(call_cap, **i32), n_call=torch.zeros(1, **i32))
        self.vout = dict(argmax=torch.zeros(S, bud, **i32),
                         taps=torch.zeros(S, bud, 3, d, **f32), logits=None)
        self.aout = dict(path=torch.zeros(S, w.M * w.K, **i32),
                         n_accepted=torch.zeros(S, **i32),
                         bonus=torch.zeros(S, **i32),
                         r_reject=torch.zeros(S, **f32))
        self.aout_c = B.AcceptOut(*[_ptr(self.aout[f]) for f in
                                    ("path", "n_accepted", "bonus",
                                     "r_reject")])
        self.V = V

    # ------------------------------------------------------------------
    @property
    def stream(self):
        return C.c_void_p(torch.cuda.current_stream(self.dev).cuda_stream)

    def _check(self, rc):
        B.check(self.lib, self.ctx, rc)

    def prefill(self, prompts):
        lens = [len(p) for p in prompts]
        ld = max(lens)
        arr = np.zeros((self.S, ld), np.int32)
        for i, p in enumerate(prompts):
            arr[i, :len(p)] = p
        self.prompt_dev = torch.from_numpy(arr).to(self.dev)
        clens = (C.c_int32 * self.S)(*lens)
        self._check(self.lib.sb_prefill(
            self.ctx, C.byref(self.seqs_c), _ptr(self.prompt_dev), ld, clens,
            C.byref(self.tkv_c), C.byref(self.dkv_c), self.stream))

    def expand(self, m, want_logits=False):
        if want_logits:
            if self.dout["logits"] is None:
                self.dout["logits"] = torch.zeros(self.call_cap, self.Vd,
                                                  dtype=torch.float32,
                                                  device=self.dev)
            lg = self.dout["logits"]
        else:
            lg = None
        o = B.DraftOut(*[_ptr(self.dout[f] if f != "logits" else lg)
                         for f in B.DRAFT_OUT_FIELDS])
        self._check(self.lib.sb_draft_block_expand(
            self.ctx, m, self.w.K, C.byref(self.seqs_c), C.byref(self.dkv_c),
            C.byref(self.tree_c), C.byref(o), self.stream))

    def verify(self, want_logits=False):
        if want_logits and self.vout["logits"] is None:
            self.vout["logits"] = torch.zeros(self.S * self.w.budget, self.V,
                                              dtype=torch.float32,
                                              device=self.dev)
        lg = self.vout["logits"] if want_logits else None
        self.vout_c = B.VerifyOut(_ptr(self.vout["argmax"]),
                                  _ptr(self.vout["taps"]), _ptr(lg))
        self._check(self.lib.sb_tree_verify(
            self.ctx, C.byref(self.seqs_c), C.byref(self.tree_c),
            C.byref(self.tkv_c), C.byref(self.vout_c), self.stream))

    def accept(self):
        self._check(self.lib.sb_accept(
            self.ctx, self.S, C.byref(self.tree_c),
            _ptr(self.vout["argmax"]), C.byref(self.aout_c), self.stream))

    def accept_sample(self, temperature, u_accept, u_bonus, *,
                      noalloc=False, n_seqs=None):
        """Stochastic acceptance over the logits of the last
        verify(want_logits=True); u_accept, u_bonus: device float tensors
        [n_seqs][budget] of uniforms in [0, 1).  noalloc: the
        allocation-free entry point (static scratch); n_seqs: the first
        n_seqs sequences only (default all)."""
        if self.vout["logits"] is None:
            raise RuntimeError("accept_sample needs verify(want_logits=True)")
        for u in (u_accept, u_bonus):
            if (u.dtype != torch.float32 or not u.is_cuda
                    or tuple(u.shape) != (self.S, self.w.budget)
                    or not u.is_contiguous()):
                raise ValueError("uniforms must be contiguous float32 device "
                                 f"tensors of shape ({self.S}, "
                                 f"{self.w.budget})")
        fn = (self.lib.sb_accept_sample_noalloc if noalloc
              else self.lib.sb_accept_sample)
        self._check(fn(
            self.ctx, n_seqs or self.S, C.byref(self.tree_c),
            _ptr(self.vout["logits"]), float(temperature), _ptr(u_accept),
            _ptr(u_bonus), C.byref(self.aout_c), self.stream))

    def commit(self):
        vc = B.VerifyOut(_ptr(self.vout["argmax"]), _ptr(self.vout["taps"]),
                         C.c_void_p(0))
        self._check(self.lib.sb_commit(
            self.ctx, C.byref(self.seqs_c), C.byref(self.tree_c),
            C.byref(vc), C.byref(self.aout_c), C.byref(self.tkv_c),
            C.byref(self.dkv_c), self.stream))

    def iteration(self):
        for m in range(1, self.w.M + 1):
            self.expand(m)
        self.verify()
        self.accept()
        self.commit()

    def set_length_bound(self, max_T: int):
        """Bound of T over all sequences (0: unknown); needed after writing
        T or the caches directly."""
        self._check(self.lib.sb_set_length_bound(self.ctx, int(max_T)))

    def set_debug(self, on: bool):
        """Start (clearing the status word) or stop the device-side reports
        of clamped page-table entries and token ids."""
        self._check(self.lib.sb_set_debug(self.ctx, int(bool(on))))

    def device_check(self):
        """Raises SBError (SB_EDEVICE) if a kernel clamped an out-of-range
        page-table entry or token id since the last check."""
        self._check(self.lib.sb_device_check(self.ctx, self.stream))

    # ---- head-only adaptation ----------------------------------------
    def adapt_buffer(self):
        """Device buffer for sb_adapt_push / sb_head_update."""
        cap = self.cfg.adapt_cap
        b = dict(h=torch.zeros(cap, self.w.target.d_model, dtype=torch.float32,
                               device=self.dev),
                 target=torch.zeros(cap, dtype=torch.int32, device=self.dev),
                 count=torch.zeros(1, dtype=torch.int32, device=self.dev))
        b["c"] = B.AdaptBuffer(_ptr(b["h"]), _ptr(b["target"]),
                               _ptr(b["count"]), cap)
        return b

    def head_copy(self):
        """A training copy of the drafter's LM head and rank head."""
        dt = self._keep[4]
        return dict(lm_head=dt["lm_head"].clone(), rank_w=dt["rank_w"].clone(),
                    rank_b=dt["rank_b"].clone())

    def adapt_push(self, buf):
        self._check(self.lib.sb_adapt_push(
            self.ctx, self.S, C.byref(self.tree_c), C.byref(self.aout_c),
            C.byref(buf["c"]), self.stream))

    def head_update(self, buf, lm_head0, train, lr, kl_weight, loss=None,
                    stream=None):
        hw = B.HeadWeights(_ptr(train["lm_head"]), _ptr(train["rank_w"]),
                           _ptr(train["rank_b"]))
        st = self.stream if stream is None else C.c_void_p(stream.cuda_stream)
        self._check(self.lib.sb_head_update(
            self.ctx, C.byref(buf["c"]), _ptr(lm_head0), C.byref(hw),
            float(lr), float(kl_weight), _ptr(loss), st))

    def set_buckets(self, buckets):
        """Force the drafter rows' buckets from a device int32 tensor
        [n_seqs][row_cap] (read by every later expand; its contents may be
        rewritten between calls), or restore the rank-head argmax (None)."""
        if buckets is None:
            self._buckets = None
            self._check(self.lib.sb_set_bucket_override(self.ctx, None))
            return
        if (buckets.dtype != torch.int32 or not buckets.is_cuda
                or tuple(buckets.shape) != (self.S, self.row_cap)
                or not buckets.is_contiguous()):
            raise ValueError("buckets must be a contiguous int32 device "
                             f"tensor of shape ({self.S}, {self.row_cap})")
        self._buckets = buckets
        self._check(self.lib.sb_set_bucket_override(self.ctx, _ptr(buckets)))

    def profile(self, enable: bool):
        self._check(self.lib.sb_profile(self.ctx, 1 if enable else 0))

    def profile_read(self) -> dict:
        arr = (B.KernelStat * 3)()
        self._check(self.lib.sb_profile_read(self.ctx, arr))
        out = {name: dict(launches=arr[i].launches, ms=arr[i].total_ms,
                          bytes=arr[i].bytes, flops=arr[i].flops)
               for i, name in enumerate(B.PROF_CLASSES)}
        g = (B.GemmStat * len(B.GEMM_GROUPS))()
        self._check(self.lib.sb_profile_read_gemm(self.ctx, g))
        out["gemm_groups"] = {
            name: dict(launches=g[i].launches,
                       launches_with_rows=g[i].launches_with_rows,
                       ms=g[i].total_ms, bytes_read=g[i].bytes_read,
                       bytes_written=g[i].bytes_written, flops=g[i].flops)
            for i, name in enumerate(B.GEMM_GROUPS)}
        return out

    # ------------------------------------------------------------------
    # cache access for tests (host <-> device copies of single entries)
    def _pool(self, which):
        return ((self.tk, self.tv, self.tpt) if which == "target"
                else (self.dk, self.dv, self.dpt))

    def write_cache(self, which, seq, k, v, start=0):
        """k, v: [n_layers][n, Hkv, hd] arrays written to entries
        start..start+n-1 of sequence seq."""
        K_, V_, pt = self._pool(which)
        n = np.asarray(k[0]).shape[0]
        e = torch.arange(start, start + n, device=self.dev)
        pages = pt[seq].long()[e // 16]
        slots = e % 16
        for layer in range(len(k)):
            kk = torch.as_tensor(np.asarray(k[layer], np.float32)).to(self.dev)
            vv = torch.as_tensor(np.asarray(v[layer], np.float32)).to(self.dev)
            K_[layer][pages, :, slots, :] = kk.to(self.et)
            V_[layer][pages, :, :, slots] = vv.to(self.et)

    def read_cache(self, which, seq, n, start=0):
        """[n_layers, n, Hkv, hd] float32 copies of entries start..start+n-1."""
        K_, V_, pt = self._pool(which)
        e = torch.arange(start, start + n, device=self.dev)
        pages = pt[seq].long()[e // 16]
        slots = e % 16
        ks = torch.stack([K_[layer][pages, :, slots, :]
                          for layer in range(K_.shape[0])])
        vs = torch.stack([V_[layer][pages, :, :, slots]
                          for layer in range(V_.shape[0])])
        return ks.float().cpu().numpy(), vs.float().cpu().numpy()

    def __del__(self):
        try:
            if getattr(self, "ctx", None):
                self.lib.sb_destroy(self.ctx)
                self.ctx = None
        except Exception:
            pass
