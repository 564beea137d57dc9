"""Seeded synthetic inputs shared by the oracle-side tests and the GPU harness.

This module holds no arithmetic of the method: only model shapes, workload
descriptions, seeded random draws and bf16 bit packing of those draws.  The
oracle (``oracle/``) and the GPU path (``paper_2605_07243_amd``) both take
their weights, prompts and cache layouts from here, so that the two sides see
bit-identical inputs while sharing no compute code.

Random-init recipe (SpecBlock ships no trained weights): every matrix, the
embedding, the drafter's position queries and the rank-head matrix are drawn
i.i.d. N(0, 0.02); RMSNorm gains are 1 and the rank-head bias is 0.  Each
tensor has its own substream keyed by (seed, crc32(name)), so a tensor's values
do not depend on which other tensors are generated.
"""
from __future__ import annotations

import dataclasses
import zlib
from concurrent.futures import ThreadPoolExecutor

import numpy as np

INIT_STD = 0.02


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Llama-style decoder dimensions."""
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rope_theta: float = 500000.0
    norm_eps: float = 1e-5

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim


@dataclasses.dataclass(frozen=True)
class Workload:
    """One speculative-decoding workload: target, drafter and tree shape."""
    name: str
    dtype: str                 # "f32" or "bf16"
    target: ModelShape
    drafter_layers: int
    K: int                     # block depth (positions per drafter forward)
    M: int                     # block expansions per verifier iteration
    B_max: int                 # next-block starts per sequence
    budget: int                # tree nodes per sequence, root included
    n_seqs: int
    prompt_len: tuple          # (lo, hi) inclusive; lo == hi for fixed length
    page_size: int = 16
    branch_map: tuple = (2, 4, 6, 4)
    draft_vocab: int = 0       # drafter output vocabulary (0: the target's)

    @property
    def tap_layers(self) -> tuple:
        L = self.target.n_layers
        return (0, L // 2, L - 1)

    @property
    def rows_per_seq(self) -> int:
        """Drafter rows one sequence can produce in one iteration."""
        return self.K + (self.M - 1) * self.B_max * self.K


LLAMA3_8B = ModelShape(32, 4096, 32, 8, 128, 14336, 128256)
LLAMA3_70B = ModelShape(80, 8192, 64, 8, 128, 28672, 128256)
TINY = ModelShape(2, 256, 4, 4, 64, 1024, 1024)

WORKLOADS = {
    "tiny-fp32": Workload("tiny-fp32", "f32", TINY, 1, K=4, M=3, B_max=4,
                          budget=32, n_seqs=1, prompt_len=(128, 128)),
    "llama3-8b-k4": Workload("llama3-8b-k4", "bf16", LLAMA3_8B, 1, K=4, M=2,
                             B_max=8, budget=60, n_seqs=1,
                             prompt_len=(1024, 1024)),
    "llama3-8b-k8-long": Workload("llama3-8b-k8-long", "bf16", LLAMA3_8B, 1,
                                  K=8, M=2, B_max=16, budget=128, n_seqs=1,
                                  prompt_len=(4096, 4096)),
    "llama3-8b-batch16-paged": Workload("llama3-8b-batch16-paged", "bf16",
                                        LLAMA3_8B, 1, K=4, M=2, B_max=8,
                                        budget=64, n_seqs=16,
                                        prompt_len=(512, 2048)),
    # the paper's own drafter shape: two decoder layers, 32000-token
    # reduced output vocabulary, K 4, M 2, 60-node trees (Sec. 4, App. A)
    "llama3-8b-paper-drafter": Workload("llama3-8b-paper-drafter", "bf16",
                                        LLAMA3_8B, 2, K=4, M=2, B_max=8,
                                        budget=60, n_seqs=1,
                                        prompt_len=(1024, 1024),
                                        draft_vocab=32000),
    "llama3-70b-k6": Workload("llama3-70b-k6", "bf16", LLAMA3_70B, 1, K=6,
                              M=2, B_max=8, budget=96, n_seqs=4,
                              prompt_len=(2048, 2048)),
}


def with_layers(w: Workload, n_layers: int, name_suffix: str = "") -> Workload:
    """Same workload with a shallower target (same per-layer shapes)."""
    t = dataclasses.replace(w.target, n_layers=n_layers)
    return dataclasses.replace(w, target=t, name=w.name + name_suffix)


# ----------------------------------------------------------------------------
# bf16 packing of generated values (input preparation only)
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    return (r >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


# ----------------------------------------------------------------------------
# seeded draws
# ----------------------------------------------------------------------------

def _rng(seed: int, name: str, chunk: int = -1) -> np.random.Generator:
    key = [seed, zlib.crc32(name.encode())]
    return np.random.default_rng(key if chunk < 0 else key + [chunk])


# Large tensors are drawn in fixed chunks, each from its own stream keyed by
# (seed, name, chunk index), so the values do not depend on how many threads
# fill them.
CHUNK = 1 << 22


def _fill_chunk(seed, name, flat, c, std, dtype):
    part = flat[c * CHUNK:(c + 1) * CHUNK]
    _rng(seed, name, c).standard_normal(out=part, dtype=np.float32)
    part *= np.float32(std)
    if dtype == "bf16":
        part[...] = bf16_bits_to_f32(f32_to_bf16_bits(part))


def normal(seed: int, name: str, shape, std: float = INIT_STD,
           dtype: str = "f32", pool=None) -> np.ndarray:
    """N(0, std) float32 array; for dtype "bf16" the values are rounded to
    bf16 (returned as float32 holding bf16-representable values).  ``pool``
    (a concurrent.futures executor) fills the chunks in parallel."""
    n = int(np.prod(shape))
    flat = np.empty(n, np.float32)
    chunks = range((n + CHUNK - 1) // CHUNK)
    if pool is None:
        for c in chunks:
            _fill_chunk(seed, name, flat, c, std, dtype)
    else:
        list(pool.map(lambda c: _fill_chunk(seed, name, flat, c, std, dtype),
                      chunks))
    return flat.reshape(shape)


def _layer_specs(prefix: str, s: ModelShape):
    d, F = s.d_model, s.d_ff
    return [
        (prefix + "attn_norm", (d,), "ones"),
        (prefix + "wq", (s.q_dim, d), "normal"),
        (prefix + "wk", (s.kv_dim, d), "normal"),
        (prefix + "wv", (s.kv_dim, d), "normal"),
        (prefix + "wo", (d, s.q_dim), "normal"),
        (prefix + "mlp_norm", (d,), "ones"),
        (prefix + "wg", (F, d), "normal"),
        (prefix + "wu", (F, d), "normal"),
        (prefix + "wd", (d, F), "normal"),
    ]


def target_specs(s: ModelShape):
    specs = [("embed", (s.vocab, s.d_model), "normal")]
    for i in range(s.n_layers):
        specs += _layer_specs(f"layers.{i}.", s)
    specs += [("final_norm", (s.d_model,), "ones"),
              ("lm_head", (s.vocab, s.d_model), "normal")]
    return specs


def drafter_specs(s: ModelShape, n_layers: int, K: int, draft_vocab: int = 0):
    d = s.d_model
    specs = [("d.w_cond", (d, 3 * d), "normal"),
             ("d.norm_c", (d,), "ones"),
             ("d.norm_e", (d,), "ones"),
             ("d.norm_q", (d,), "ones"),
             ("d.pos_query", (K, d), "normal"),
             ("d.w_fuse", (d, 3 * d), "normal")]
    for i in range(n_layers):
        specs.append((f"d.layers.{i}.w_shift", (d, 2 * d), "normal"))
        specs += _layer_specs(f"d.layers.{i}.", s)
    specs += [("d.final_norm", (d,), "ones"),
              ("d.lm_head", (draft_vocab or s.vocab, d), "normal"),
              ("d.rank_w", (4, d + 15), "normal"),
              ("d.rank_b", (4,), "zeros")]
    return specs


def make_weights(specs, seed: int = 0, dtype: str = "f32",
                 threads: int = 8, jitter: float = 0.0) -> dict:
    """Generate every tensor in ``specs``.  Rank-head parameters stay fp32
    (the rank head is a tiny fp32 classifier in every configuration).

    ``jitter`` > 0 draws norm gains as 1 + N(0, jitter) and the rank-head
    bias as N(0, jitter) instead of the constant 1 / 0, so that tests can
    tell the gains and biases apart."""
    def one(spec, ex):
        name, shape, kind = spec
        if kind == "ones":
            if jitter:
                return (1.0 + normal(seed, name, shape, jitter)).astype(np.float32)
            return np.ones(shape, np.float32)
        if kind == "zeros":
            if jitter:
                return normal(seed, name, shape, jitter)
            return np.zeros(shape, np.float32)
        dt = "f32" if name.startswith("d.rank_") else dtype
        return normal(seed, name, shape, dtype=dt, pool=ex)
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return {spec[0]: one(spec, ex) for spec in specs}


def target_weights(w: Workload, seed: int = 0, jitter: float = 0.0) -> dict:
    return make_weights(target_specs(w.target), seed, w.dtype, jitter=jitter)


def draft_vocab_map(seed: int, vocab: int, draft_vocab: int) -> np.ndarray:
    """Target ids of a reduced drafter vocabulary, int32 [draft_vocab],
    strictly increasing: a seeded random subset standing in for the most
    frequent target tokens (no token statistics exist for random weights)."""
    ids = _rng(seed, "d2t").choice(vocab, size=draft_vocab, replace=False)
    return np.sort(ids).astype(np.int32)


def drafter_weights(w: Workload, seed: int = 0, jitter: float = 0.0) -> dict:
    out = make_weights(drafter_specs(w.target, w.drafter_layers, w.K,
                                     w.draft_vocab), seed, w.dtype,
                       jitter=jitter)
    if w.draft_vocab and w.draft_vocab != w.target.vocab:
        out["d.d2t"] = draft_vocab_map(seed, w.target.vocab, w.draft_vocab)
    return out


def prompt_lengths(w: Workload, seed: int = 2) -> np.ndarray:
    lo, hi = w.prompt_len
    if lo == hi:
        return np.full(w.n_seqs, lo, np.int64)
    return _rng(seed, "prompt_lengths").integers(lo, hi + 1, size=w.n_seqs)


def prompts(w: Workload, seed: int = 1, lengths=None) -> list:
    """Uniform random token ids in [0, vocab), one array per sequence."""
    if lengths is None:
        lengths = prompt_lengths(w)
    rng = _rng(seed, "prompts")
    return [rng.integers(0, w.target.vocab, size=int(n)).astype(np.int64)
            for n in lengths]


# Class frequencies of the rank-head buckets b0..b3 of a trained 8B-class
# drafter (App. B, rank-head quality table), in tenths of a percent.
PAPER_BUCKET_PERMILLE = (752, 150, 41, 57)


def paper_buckets(seed: int, iteration: int, n_seqs: int,
                  row_cap: int) -> np.ndarray:
    """Forced drafter-row buckets of one iteration, int32 [n_seqs][row_cap]:
    i.i.d. draws with the frequencies PAPER_BUCKET_PERMILLE, from a stream
    keyed by (seed, iteration, sequence), so that a sequence's draws do not
    depend on the batch it runs in."""
    edges = np.cumsum(PAPER_BUCKET_PERMILLE)[:-1]
    out = np.empty((n_seqs, row_cap), np.int32)
    for s in range(n_seqs):
        u = np.random.default_rng(
            [seed, zlib.crc32(b"paper_buckets"), iteration, s]).integers(
                0, 1000, size=row_cap)
        out[s] = np.searchsorted(edges, u, side="right")
    return out


def uniform_tree(w: Workload, k: int) -> Workload:
    """The "uniform fixed-k tree" ablation of rank-guided branching at the
    same node budget (Sec. 4, ablations): every drafter row is forced into
    bucket b1 (uniform_buckets) and every bucket branches k, so each row
    contributes its top-k tokens and every sibling is a next-block start
    candidate."""
    return dataclasses.replace(w, name=f"{w.name}-uniform{k}",
                               branch_map=(k, k, k, k))


def uniform_buckets(n_seqs: int, row_cap: int) -> np.ndarray:
    """Forced buckets of the uniform tree: b1 for every row."""
    return np.ones((n_seqs, row_cap), np.int32)


def random_kv(seed: int, name: str, n_tokens: int, s: ModelShape,
              dtype: str, std: float = 1.0):
    """Synthetic K and V of one layer, [n_tokens, n_kv_heads, head_dim]."""
    shp = (n_tokens, s.n_kv_heads, s.head_dim)
    return (normal(seed, name + ".k", shp, std, dtype),
            normal(seed, name + ".v", shp, std, dtype))
