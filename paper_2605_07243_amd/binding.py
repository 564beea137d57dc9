"""ctypes view of the C ABI in include/specblock.h (argument marshalling only).

The shared library is built in-tree by ``paper_2605_07243_amd.build``; loading
fails loudly when it is missing.  Every struct mirrors the header field by
field.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# SPECBLOCK_LIB selects another build of the same library (the host
# AddressSanitizer build of the ABI checks); the default is the in-tree one
LIB_PATH = os.environ.get("SPECBLOCK_LIB") or os.path.join(HERE,
                                                            "libspecblock.so")

(SB_OK, SB_EINVAL, SB_ESHAPE, SB_EBUDGET, SB_EDTYPE, SB_EHIP, SB_ESTATE,
 SB_EDEVICE) = range(8)
SB_F32, SB_BF16 = 0, 1
TOPK, PSI_DIM = 10, 15

vp = C.c_void_p
i32 = C.c_int32


class ModelDims(C.Structure):
    _fields_ = [("n_layers", i32), ("d_model", i32), ("n_heads", i32),
                ("n_kv_heads", i32), ("head_dim", i32), ("d_ff", i32),
                ("vocab", i32), ("rope_theta", C.c_float),
                ("norm_eps", C.c_float)]


class Config(C.Structure):
    _fields_ = [("target", ModelDims), ("drafter_layers", i32),
                ("tap_layers", i32 * 3), ("K", i32), ("M", i32),
                ("B_max", i32), ("budget", i32), ("branch_map", i32 * 4),
                ("dtype", i32), ("max_seqs", i32), ("page_size", i32),
                ("max_pages", i32), ("prefill_chunk", i32),
                ("draft_vocab", i32), ("adapt_cap", i32)]


class LayerWeights(C.Structure):
    _fields_ = [("attn_norm", vp), ("w_qkv", vp), ("w_o", vp),
                ("mlp_norm", vp), ("w_gate_up", vp), ("w_down", vp),
                ("w_shift", vp)]


class TargetWeights(C.Structure):
    _fields_ = [("embed", vp), ("layers", C.POINTER(LayerWeights)),
                ("final_norm", vp), ("lm_head", vp)]


class DrafterWeights(C.Structure):
    _fields_ = [("w_cond", vp), ("norm_c", vp), ("norm_e", vp),
                ("norm_q", vp), ("pos_query", vp), ("w_fuse", vp),
                ("layers", C.POINTER(LayerWeights)), ("final_norm", vp),
                ("lm_head", vp), ("rank_w", vp), ("rank_b", vp),
                ("d2t", vp)]


class AdaptBuffer(C.Structure):
    _fields_ = [("h", vp), ("target", vp), ("count", vp), ("cap", i32)]


class HeadWeights(C.Structure):
    _fields_ = [("lm_head", vp), ("rank_w", vp), ("rank_b", vp)]


class KV(C.Structure):
    _fields_ = [("k", vp), ("v", vp), ("page_table", vp), ("n_layers", i32),
                ("n_pages", i32)]


class Seqs(C.Structure):
    _fields_ = [("n_seqs", i32), ("root", vp), ("T", vp), ("cond_taps", vp)]


TREE_FIELDS = ["n_nodes", "token", "parent", "depth", "row", "rank", "logp",
               "cum_logp", "anc", "n_rows", "row_block", "row_start", "row_k",
               "row_pos", "row_vis", "h_last", "n_starts", "starts"]


class Tree(C.Structure):
    _fields_ = [(f, vp) for f in TREE_FIELDS]


DRAFT_OUT_FIELDS = ["topk_id", "topk_logit", "lse", "psi", "bucket", "branch",
                    "logits", "call_seq", "call_row", "n_call"]


class DraftOut(C.Structure):
    _fields_ = [(f, vp) for f in DRAFT_OUT_FIELDS]


class VerifyOut(C.Structure):
    _fields_ = [("argmax", vp), ("taps", vp), ("logits", vp)]


class AcceptOut(C.Structure):
    _fields_ = [("path", vp), ("n_accepted", vp), ("bonus", vp),
                ("r_reject", vp)]


class KernelStat(C.Structure):
    _fields_ = [("launches", C.c_int64), ("total_ms", C.c_double),
                ("bytes", C.c_double), ("flops", C.c_double)]


class GemmStat(C.Structure):
    _fields_ = [("launches", C.c_int64), ("launches_with_rows", C.c_int64),
                ("total_ms", C.c_double), ("bytes_read", C.c_double),
                ("bytes_written", C.c_double), ("flops", C.c_double)]


PROF_CLASSES = ("gemm", "tree_attn", "vocab")
GEMM_GROUPS = ("target", "drafter", "swiglu", "lm_head")

EXPORTS = ["sb_row_capacity", "sb_workspace_bytes", "sb_create", "sb_destroy",
           "sb_last_error", "sb_bind", "sb_prefill", "sb_draft_block_expand",
           "sb_tree_verify", "sb_accept", "sb_commit", "sb_set_length_bound",
           "sb_profile", "sb_profile_read", "sb_profile_read_gemm",
           "sb_pack_weight",
           "sb_set_bucket_override", "sb_accept_sample", "sb_adapt_push",
           "sb_head_update", "sb_accept_sample_noalloc", "sb_set_debug",
           "sb_device_check"]

_lib = None


def load(path: str = LIB_PATH):
    """Load libspecblock.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with "
            "`python -m paper_2605_07243_amd.build` (there is no fallback)")
    lib = C.CDLL(path)
    P = C.POINTER
    lib.sb_row_capacity.argtypes = [P(Config)]
    lib.sb_row_capacity.restype = i32
    lib.sb_workspace_bytes.argtypes = [P(Config)]
    lib.sb_workspace_bytes.restype = C.c_size_t
    lib.sb_create.argtypes = [P(Config), P(vp)]
    lib.sb_create.restype = C.c_int
    lib.sb_destroy.argtypes = [vp]
    lib.sb_destroy.restype = None
    lib.sb_last_error.argtypes = [vp]
    lib.sb_last_error.restype = C.c_char_p
    lib.sb_bind.argtypes = [vp, P(TargetWeights), P(DrafterWeights), vp,
                            C.c_size_t]
    lib.sb_bind.restype = C.c_int
    lib.sb_pack_weight.argtypes = [vp, vp, i32, i32, i32, i32, vp]
    lib.sb_pack_weight.restype = C.c_int
    lib.sb_prefill.argtypes = [vp, P(Seqs), vp, i32, P(i32), P(KV), P(KV), vp]
    lib.sb_prefill.restype = C.c_int
    lib.sb_draft_block_expand.argtypes = [vp, i32, i32, P(Seqs), P(KV),
                                          P(Tree), P(DraftOut), vp]
    lib.sb_draft_block_expand.restype = C.c_int
    lib.sb_tree_verify.argtypes = [vp, P(Seqs), P(Tree), P(KV), P(VerifyOut),
                                   vp]
    lib.sb_tree_verify.restype = C.c_int
    lib.sb_accept.argtypes = [vp, i32, P(Tree), vp, P(AcceptOut), vp]
    lib.sb_accept.restype = C.c_int
    lib.sb_commit.argtypes = [vp, P(Seqs), P(Tree), P(VerifyOut),
                              P(AcceptOut), P(KV), P(KV), vp]
    lib.sb_commit.restype = C.c_int
    lib.sb_set_length_bound.argtypes = [vp, i32]
    lib.sb_set_length_bound.restype = C.c_int
    lib.sb_set_debug.argtypes = [vp, i32]
    lib.sb_set_debug.restype = C.c_int
    lib.sb_device_check.argtypes = [vp, vp]
    lib.sb_device_check.restype = C.c_int
    lib.sb_accept_sample.argtypes = [vp, i32, vp, vp, C.c_float, vp, vp,
                                     vp, vp]
    lib.sb_accept_sample.restype = C.c_int
    lib.sb_accept_sample_noalloc.argtypes = [vp, i32, vp, vp, C.c_float, vp,
                                             vp, vp, vp]
    lib.sb_accept_sample_noalloc.restype = C.c_int
    lib.sb_adapt_push.argtypes = [vp, i32, vp, vp, vp, vp]
    lib.sb_adapt_push.restype = C.c_int
    lib.sb_head_update.argtypes = [vp, vp, vp, vp, C.c_float, C.c_float, vp,
                                   vp]
    lib.sb_head_update.restype = C.c_int
    lib.sb_set_bucket_override.argtypes = [vp, vp]
    lib.sb_set_bucket_override.restype = C.c_int
    lib.sb_profile.argtypes = [vp, i32]
    lib.sb_profile.restype = C.c_int
    lib.sb_profile_read.argtypes = [vp, P(KernelStat)]
    lib.sb_profile_read.restype = C.c_int
    lib.sb_profile_read_gemm.argtypes = [vp, P(GemmStat)]
    lib.sb_profile_read_gemm.restype = C.c_int
    _lib = lib
    return lib


class SBError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"specblock error {code}: {msg}")
        self.code = code


def check(lib, ctx, rc):
    if rc != SB_OK:
        raise SBError(rc, lib.sb_last_error(ctx).decode())
