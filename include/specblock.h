/*
 * specblock.h - C ABI of the SpecBlock block-expansion hot path on MI355X.
 *
 * SpecBlock (Block-Iterative Speculative Decoding with Dynamic Tree
 * Drafting) alternates drafting and verification.  One verifier iteration
 * (Alg. 2 of the paper) is:
 *
 *   for m = 1..M:  sb_draft_block_expand   one batched drafter forward over
 *                                          every start x K block positions,
 *                                          then psi, rank head, branching and
 *                                          sibling attachment (Sec. 3.1-3.2)
 *   sb_tree_verify                         one target forward over the tree
 *   sb_accept                              greedy acceptance walk
 *   sb_commit                              keep the accepted K/V, advance
 *
 * Conventions
 * - Every pointer inside the structs below is a DEVICE pointer unless its
 *   comment says "host".  The caller allocates and owns all memory: the
 *   library never allocates or frees device memory.  Its scratch lives in one
 *   caller-provided workspace of sb_workspace_bytes() bytes.
 * - Floating-point storage type "elem" is float32 when cfg.dtype == SB_F32
 *   and bfloat16 (uint16_t bits, round-to-nearest-even) when SB_BF16.
 *   Accumulation, norms, softmax, residual stream, logits, h^(L) and all
 *   outputs typed float are float32.
 * - Matrices are row-major [out_features][in_features] (y = W x), except
 *   that with SB_BF16 the projection matrices passed to sb_bind (w_qkv, w_o,
 *   w_gate_up, w_down, w_shift, w_cond, w_fuse and both lm_head) are in the
 *   fragment-packed layout written by sb_pack_weight.  embed and pos_query
 *   stay row-major.
 * - Calls are asynchronous: they enqueue work on `stream` (a hipStream_t;
 *   NULL = the default stream) and return.  Outputs are valid once the
 *   stream has reached that point.  No call synchronises with the host.
 * - Every call returns SB_OK (0) or an error code; arguments are validated on
 *   the host before anything is enqueued, so an error leaves device state
 *   untouched.  sb_last_error() describes the last failure of a context.
 * - One context may be used by one host thread / stream at a time.
 */
#ifndef SPECBLOCK_H
#define SPECBLOCK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum sb_status {
  SB_OK = 0,
  SB_EINVAL = 1,   /* NULL or misaligned pointer, bad argument value        */
  SB_ESHAPE = 2,   /* dimensions inconsistent with the configuration       */
  SB_EBUDGET = 3,  /* tree, row, page or workspace capacity exceeded        */
  SB_EDTYPE = 4,   /* unknown storage type                                  */
  SB_EHIP = 5,     /* a HIP runtime call failed (message in sb_last_error)  */
  SB_ESTATE = 6,   /* call out of order (e.g. before sb_bind)               */
  SB_EDEVICE = 7   /* sb_device_check: kernels clamped an out-of-range input */
};

enum sb_dtype { SB_F32 = 0, SB_BF16 = 1 };

#define SB_TOPK 10     /* top-k kept per drafter row (psi uses the top 10) */
#define SB_PSI_DIM 15  /* distribution summary psi (App. B)                */
#define SB_N_BUCKETS 4 /* rank-head buckets b0..b3 (Sec. 3.2)              */

/* Llama-style decoder dimensions (the drafter layers match the target's
 * per-layer architecture, Sec. 3.1). */
typedef struct sb_model_dims {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab;
  float rope_theta, norm_eps;
} sb_model_dims;

typedef struct sb_config {
  sb_model_dims target;     /* drafter width/heads/vocab equal the target's  */
  int32_t drafter_layers;   /* L of the drafter                               */
  int32_t tap_layers[3];    /* target layers giving h_low, h_mid, h_top (Eq.1)*/
  int32_t K;                /* block depth: positions per drafter forward     */
  int32_t M;                /* block expansions per verifier iteration        */
  int32_t B_max;            /* next-block starts per sequence                 */
  int32_t budget;           /* tree nodes per sequence, root included (<=512) */
  int32_t branch_map[4];    /* bucket -> branching b(.) (App. A.5), 0..10     */
  int32_t dtype;            /* enum sb_dtype                                  */
  int32_t max_seqs;         /* sequences per call                             */
  int32_t page_size;        /* K/V page size in tokens; must be 16            */
  int32_t max_pages;        /* page-table row length (pages per sequence),
                               1..16384                                       */
  int32_t prefill_chunk;    /* rows per prefill step (multiple of 16)         */
  int32_t draft_vocab;      /* drafter output vocabulary: 0 = the target's;
                               else a multiple of 16 in 10..vocab, the
                               drafter's reduced vocabulary (App. A: the most
                               frequent target tokens), mapped to target ids
                               by sb_drafter_weights.d2t                      */
  int32_t adapt_cap;        /* positions per head-only update, 0..64 (0: no
                               sb_adapt_push / sb_head_update)               */
} sb_config;

/* One decoder layer.  elem matrices; float gains. */
typedef struct sb_layer_weights {
  const void* attn_norm;  /* float [d]                                        */
  const void* w_qkv;      /* elem [(H + 2 Hkv) hd][d]: Q heads, K heads, V heads */
  const void* w_o;        /* elem [d][H hd]                                   */
  const void* mlp_norm;   /* float [d]                                        */
  const void* w_gate_up;  /* elem [2F][d]: gate rows 0..F-1, then up rows     */
  const void* w_down;     /* elem [d][F]                                      */
  const void* w_shift;    /* drafter: elem [d][2d] layer-wise shift (Eq. 3),
                             applied to [h_k, h_{k-1}]; target: NULL          */
} sb_layer_weights;

typedef struct sb_target_weights {
  const void* embed;                /* elem [V][d] (shared with the drafter)  */
  const sb_layer_weights* layers;   /* host array [n_layers]                  */
  const void* final_norm;           /* float [d]                              */
  const void* lm_head;              /* elem [V][d]                            */
} sb_target_weights;

typedef struct sb_drafter_weights {
  const void* w_cond;      /* elem [d][3d]: c = W_cond [h_low,h_mid,h_top] (Eq.1)*/
  const void* norm_c;      /* float [d] RMSNorm gain of c       (Eq. 2)       */
  const void* norm_e;      /* float [d] RMSNorm gain of embed(x)              */
  const void* norm_q;      /* float [d] RMSNorm gain of q_k                   */
  const void* pos_query;   /* elem [K][d] learnable position queries q_1..q_K */
  const void* w_fuse;      /* elem [d][3d]: W_fuse [norm c, norm e, norm q]   */
  const sb_layer_weights* layers;   /* host array [drafter_layers]            */
  const void* final_norm;  /* float [d]                                       */
  const void* lm_head;     /* elem [Vd][d], Vd = draft_vocab or V             */
  const void* rank_w;      /* float [4][d + 15]: rank head over [h^(L), psi]  */
  const void* rank_b;      /* float [4]                                       */
  const int32_t* d2t;      /* device int32 [Vd]: target id of drafter id i,
                              strictly increasing in [0, V) (checked by
                              sb_bind); NULL only when Vd == V (identity)    */
} sb_drafter_weights;

/* Paged K/V cache of one model.  Entry i of sequence s lives in page
 * page_table[s][i / 16] at slot i % 16.  Per layer and page:
 *   k: [n_kv_heads][16][head_dim]   elem
 *   v: [n_kv_heads][head_dim][16]   elem (transposed within the page)
 * i.e. k is [n_layers][n_pages][n_kv_heads][16][head_dim].
 * The target cache holds positions 0..T-1 (entry i = position i); the
 * drafter cache holds positions 1..T (entry i = position i + 1). */
typedef struct sb_kv {
  void* k;
  void* v;
  const int32_t* page_table;   /* [max_seqs][max_pages]                      */
  int32_t n_layers;            /* host value                                 */
  int32_t n_pages;             /* host value: pages in the pool              */
} sb_kv;

/* Per-sequence decoding state. */
typedef struct sb_seqs {
  int32_t n_seqs;      /* host value, <= cfg.max_seqs                        */
  int32_t* root;       /* [S] root token x_T (last verified, not yet run)    */
  int32_t* T;          /* [S] root position = committed entries per cache    */
  float* cond_taps;    /* [S][3][d] target taps at position T-1 (Eq. 1 input)*/
} sb_seqs;

/* Draft tree of the current iteration plus the drafter rows that built it.
 * Node 0 is the root.  Nodes are topologically ordered (parent < child).
 * Row r of sequence s is the r-th drafter row produced in this iteration;
 * the rows of one start are consecutive, k = 1..K. */
typedef struct sb_tree {
  int32_t* n_nodes;     /* [S]                                               */
  int32_t* token;       /* [S][budget]                                       */
  int32_t* parent;      /* [S][budget] (-1 for the root)                     */
  int32_t* depth;       /* [S][budget]                                       */
  int32_t* row;         /* [S][budget] row that proposed the node (-1 root)  */
  int32_t* rank;        /* [S][budget] 1-based rank in that row (0 root)     */
  float* logp;          /* [S][budget] log p of the token in its row         */
  float* cum_logp;      /* [S][budget] sum of logp along the root path       */
  uint32_t* anc;        /* [S][budget][ceil(budget/32)] ancestor-or-self bits*/
  int32_t* n_rows;      /* [S]                                               */
  int32_t* row_block;   /* [S][row_cap] expansion index m (1-based)          */
  int32_t* row_start;   /* [S][row_cap] start node of the row's block        */
  int32_t* row_k;       /* [S][row_cap] block position k (1-based)           */
  int32_t* row_pos;     /* [S][row_cap] RoPE position                        */
  uint32_t* row_vis;    /* [S][row_cap][ceil(row_cap/32)] visible rows       */
  float* h_last;        /* [S][row_cap][d] cached h^(L) (pre final norm)     */
  int32_t* n_starts;    /* [S] starts of the next block                      */
  int32_t* starts;      /* [S][B_max] their node ids                         */
} sb_tree;
/* row_cap = K + (M - 1) * B_max * K, see sb_row_capacity(). */

/* Per-row results of one block expansion, indexed [S][row_cap]. */
typedef struct sb_draft_out {
  int32_t* topk_id;     /* [S][row_cap][10] target ids (drafter ids through
                           d2t), larger logit first, ties to the smaller id  */
  float* topk_logit;    /* [S][row_cap][10]                                  */
  float* lse;           /* [S][row_cap] log-sum-exp of the row's Vd logits   */
  float* psi;           /* [S][row_cap][15] App. B summary                   */
  int32_t* bucket;      /* [S][row_cap] rank-head bucket 0..3 (Eq. 4)        */
  int32_t* branch;      /* [S][row_cap] b(bucket)                            */
  float* logits;        /* optional (NULL = not written): [call_cap][Vd] in
                           call-row order, drafter ids                       */
  int32_t* call_seq;    /* [call_cap] sequence of call row i                 */
  int32_t* call_row;    /* [call_cap] its row id within the sequence         */
  int32_t* n_call;      /* [1] rows in this call                             */
} sb_draft_out;
/* call_cap = max_seqs * B_max * K (block 1: max_seqs * K). */

typedef struct sb_verify_out {
  int32_t* argmax;      /* [S][budget] target greedy token per node          */
  float* taps;          /* [S][budget][3][d] target taps per node            */
  float* logits;        /* optional: [max_seqs * budget][V] in call-row order
                           (sequence-major, node order)                      */
} sb_verify_out;

typedef struct sb_accept_out {
  int32_t* path;        /* [S][M K] accepted node ids, root excluded         */
  int32_t* n_accepted;  /* [S] a: accepted draft tokens                      */
  int32_t* bonus;       /* [S] target token after the last accepted node     */
  float* r_reject;      /* optional (NULL = not written): [S] the verifier-
                           derived signal's r (Sec. 3.4, Eq. 8): the
                           drafter's probability of the bonus token at the
                           rejected position, from the drafter row that
                           predicted the position after the last accepted
                           node (its cached h^(L) through the final norm
                           and LM head, over its log-sum-exp); 0 when the
                           bonus is outside a reduced drafter vocabulary,
                           -1 when no drafter row predicts that position.
                           A query's signal is s = sum of (1 - r) over its
                           iterations with r >= 0.                          */
} sb_accept_out;

typedef struct sb_ctx sb_ctx;

/* Capacities derived from a configuration. */
int32_t sb_row_capacity(const sb_config* cfg);
/* Workspace bytes sb_bind needs for this configuration (0 if invalid). */
size_t sb_workspace_bytes(const sb_config* cfg);

/* Validate cfg (SB_EINVAL / SB_ESHAPE / SB_EDTYPE) and create a context.
 * The configuration carries the inputs of one verifier iteration (Alg. 2:
 * block depth K, block budget M, the bucket-to-branching map b(.) of the
 * inference procedure, App. A.5), the drafter block's shape (Sec. 3.1: a
 * Llama-style decoder of the target's width, App. A.1: L layers and an
 * optional reduced vocabulary) and the target's, plus capacities.  Host
 * only: nothing is allocated on the device.  *out is NULL on error. */
int sb_create(const sb_config* cfg, sb_ctx** out);
void sb_destroy(sb_ctx* ctx);
/* Thread-unsafe description of the last error of ctx (or of the last failed
 * sb_create when ctx is NULL). */
const char* sb_last_error(const sb_ctx* ctx);

/* Attach weights and workspace.  The target tables hold the verifier
 * (Alg. 2, M) and the drafter tables the drafter D_theta of Sec. 3.1:
 * W_cond (Eq. 1), the three input norms, position queries and W_fuse
 * (Eq. 2), per layer W_shift (Eq. 3) and the decoder weights, the LM head
 * and the rank head g_phi (Eq. 4).  Tables are copied (host arrays may be
 * freed); the device memory they point to must outlive the context.
 * workspace: device, 256-byte aligned, >= sb_workspace_bytes(cfg) bytes,
 * owned by the caller and used as the library's scratch until the context
 * is destroyed or bound again.  Errors: SB_EINVAL (NULL or misaligned
 * pointers, a d2t that is not strictly increasing in [0, vocab)),
 * SB_EBUDGET (workspace too small), SB_EHIP (reading d2t failed).
 * SB_BF16: the projection matrices must have been packed by sb_pack_weight
 * (w_gate_up with gate_up = 1, the others with 0).  With SB_BF16 the first
 * drafter forward after sb_bind caches W_fuse's q_k part (the last d columns
 * of W_fuse applied to norm_q(q_k), k = 1..K; Eq. 2) in the workspace; bind
 * again after changing w_fuse, norm_q or pos_query. */
int sb_bind(sb_ctx* ctx, const sb_target_weights* target,
            const sb_drafter_weights* drafter, void* workspace,
            size_t workspace_bytes);

/* Weight layout conversion (setup, not the hot path).  The projections
 * are the dense contractions of the drafter and the target (Sec. 3.1, Eq.
 * 1-3); their bf16 weights are stored in the order the MFMA kernels consume
 * them, so that every weight load of a wavefront is 1 KiB contiguous.
 *
 * src: device, row-major elem [rows][cols] (for gate_up: gate rows
 * 0..rows/2-1, then up rows).  dst: device, rows * cols elem, must not
 * overlap src; the caller owns both.
 *   SB_F32:  dst is a plain copy (f32 weights stay row-major).
 *   SB_BF16: needs rows % 32 == 0 and cols % 64 == 0 (src, dst 16-byte
 *     aligned).  Logical row r' of block rb = r' / 32 is source row r' when
 *     gate_up == 0; with gate_up != 0, logical row 32 rb + j is gate row
 *     16 rb + j (j < 16) or up row rows/2 + 16 rb + j - 16.  Element
 *       dst[((kb * (rows / 32) + rb) * 4 + i) * 512 + l * 8 + e]
 *         = logical[32 rb + l % 32][64 kb + 32 (l / 32) + 8 i + e]
 *     for l = 0..63, i = 0..3, e = 0..7.
 * Enqueued on `stream`; errors: SB_EINVAL (NULL / misaligned / overlapping
 * pointers, rows or cols < 1), SB_ESHAPE (bf16 sizes), SB_EDTYPE, SB_EHIP;
 * the message is in sb_last_error(NULL). */
int sb_pack_weight(const void* src, void* dst, int32_t rows, int32_t cols,
                   int32_t dtype, int32_t gate_up, void* stream);

/* Prefill (setup, not the hot path).  It produces what one verifier
 * iteration requires (Alg. 2): the last verified token, the target's
 * multi-layer features of the preceding position, and the committed
 * prefix's K/V for both models; the drafter's entries are the K/V each
 * committed position produced in its own draft forward (App. A.2), here a
 * one-position block per prompt position.  Causal target forward over each prompt
 * x_0..x_{n_s-1}, writing target K/V entries 0..n_s-1, the root x_{n_s}
 * (greedy), T = n_s and cond_taps; then drafter catch-up rows for positions
 * 1..n_s (a K = 1 block started at position p-1 conditioned on the target
 * taps of position p-2, zero for p = 1), written to the drafter cache.
 * prompt: device [n_seqs][ld_prompt]; lens: HOST [n_seqs], 1..max_pages*16-1.
 * The caller fills both page tables. */
int sb_prefill(sb_ctx* ctx, const sb_seqs* seqs, const int32_t* prompt,
               int32_t ld_prompt, const int32_t* lens, sb_kv* target_kv,
               sb_kv* draft_kv, void* stream);

/* One block expansion (Sec. 3.1-3.2; Alg. 2 inner loop).
 * block_index 1 starts a new iteration: it resets `tree` to the root
 * (seqs->root at seqs->T) and conditions the single start on
 * c = W_cond [cond_taps] (Eq. 1).  block_index m > 1 expands the starts the
 * previous call left in tree->starts, each conditioned on the cached h^(L)
 * of the row that proposed it (bypassing W_cond).  Each start runs K rows:
 * h0_k = W_fuse [norm c, norm embed(token), norm q_k] (Eq. 2), then per
 * drafter layer the shift W_shift [h_k, h_{k-1}] (Eq. 3, h_0 := h_1) and the
 * decoder layer, attending to the drafter prefix (entries 1..T), the rows of
 * earlier blocks on the start's path and its own rows <= k.  Then the final
 * norm, the LM head over the drafter vocabulary, top-10 (mapped to target
 * ids through d2t) / log-sum-exp / entropy, psi, the rank head (argmax,
 * ties to the lower bucket, unless sb_set_bucket_override forces the
 * buckets), b = branch_map[bucket], sibling
 * attachment in (k, start, rank) order within the budget, and the next
 * starts (chain ends first, then rank>=2 siblings of b1/b2 rows by cum_logp,
 * at most B_max, none when the tree is full).
 * K must equal cfg.K; block_index 1..cfg.M. */
int sb_draft_block_expand(sb_ctx* ctx, int32_t block_index, int32_t K,
                          const sb_seqs* seqs, const sb_kv* draft_kv,
                          sb_tree* tree, sb_draft_out* out, void* stream);

/* Tree verification (Alg. 2): one target forward over every tree node, node
 * n at position T + depth(n), attending to target entries 0..T-1 and its
 * ancestors-or-self.  Writes the node K/V to the library's tree scratch
 * (kept for sb_commit), argmax (ties to the smaller id) and taps. */
int sb_tree_verify(sb_ctx* ctx, const sb_seqs* seqs, const sb_tree* tree,
                   const sb_kv* target_kv, sb_verify_out* out, void* stream);

/* Greedy acceptance: from the root follow the child whose token equals the
 * target's argmax at the current node (lowest node id on duplicates); the
 * argmax at the last accepted node is the bonus.  tau = n_accepted + 1. */
int sb_accept(sb_ctx* ctx, int32_t n_seqs, const sb_tree* tree,
              const int32_t* argmax, sb_accept_out* out, void* stream);

/* Stochastic acceptance at temperature T > 0, the paper's sampling setting
 * (T = 1.0, Sec. 4), which it verifies by rejection sampling without
 * giving the algorithm; this is the lossless multi-candidate scheme.  At
 * node n, with p_n = softmax(z_n / T) over the target vocabulary, the
 * children are tested in node-id order, each as a point-mass draft against
 * the residual r (p_n without the tokens rejected so far, renormalised):
 * child c with token x is accepted when u_accept[s][c] < r(x) and the walk
 * moves to c; otherwise x leaves the residual (a child whose token was
 * already rejected is skipped).  When no child is accepted, the bonus is the
 * smallest token id whose cumulative residual mass exceeds u_bonus[s][n]
 * times the residual total.  Every emitted token is then distributed as the
 * target's own sample at that position.
 * logits: device float [sum of n_nodes][V], the target logits of
 *   sb_tree_verify (verify_out.logits) in call-row order (sequence-major,
 *   node order) for the same n_seqs and tree;
 * u_accept, u_bonus: device float [n_seqs][budget], uniforms in [0, 1)
 *   indexed by node id (the caller draws them; the library draws nothing);
 * out: as sb_accept (path, n_accepted, bonus; tau = n_accepted + 1), for
 *   sb_commit.
 * Errors: SB_EINVAL (temperature not positive and finite, NULL or
 * misaligned pointers), SB_ESHAPE (n_seqs), SB_ESTATE (not bound). */
int sb_accept_sample(sb_ctx* ctx, int32_t n_seqs, const sb_tree* tree,
                     const float* logits, float temperature,
                     const float* u_accept, const float* u_bonus,
                     sb_accept_out* out, void* stream);

/* Allocation-free variant of sb_accept_sample, for callers that cannot
 * allocate (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation): same arguments, same results, but the per-node
 * softmax tile statistics live in a static device array of the library
 * (65536 float2 entries, 512 KiB, one copy per GPU, held until the process
 * ends) instead of the bound workspace, and the call allocates nothing.
 * The context need not be bound unless out->r_reject is requested (the
 * signal reads the drafter weights and the workspace); only its
 * configuration (budget, vocab, K, M, B_max) is used otherwise.
 * Requires n_seqs * budget * ceil(vocab / 16384) <= 65536 (else
 * SB_EBUDGET).  Every call on a GPU shares that GPU's array, which keeps
 * the last call's contents (each call writes every entry it reads, so
 * nothing needs clearing): calls that overlap in time on one GPU, on any
 * stream or context, race and must be ordered by the caller.
 * Errors: as sb_accept_sample, plus SB_EBUDGET, SB_ESTATE (r_reject on an
 * unbound context), SB_EHIP (the array's address could not be resolved). */
int sb_accept_sample_noalloc(sb_ctx* ctx, int32_t n_seqs, const sb_tree* tree,
                             const float* logits, float temperature,
                             const float* u_accept, const float* u_bonus,
                             sb_accept_out* out, void* stream);

/* Commit (Alg. 2: the accepted prefix and the bonus are committed before
 * the next iteration, App. A.5; committed positions keep the K/V of their
 * own draft forward, App. A.2).  Target K/V of the root and accepted nodes (from the last
 * sb_tree_verify) become entries T..T+a; drafter entries for positions
 * T+1..T+a reuse the K/V of the rows that proposed the accepted nodes, and
 * position T+a+1 reuses the row continuing the last accepted node, or, when
 * the tree has none, a catch-up row (K = 1 block started at the last
 * accepted node, conditioned on the taps of its parent).  Then root = bonus,
 * T += a + 1, cond_taps = taps of the last accepted node. */
/* Errors: SB_EINVAL (NULL or misaligned pointers), SB_ESHAPE (n_seqs,
 * cache layer counts), SB_ESTATE (not bound).  Pages for the new entries
 * must already be in both page tables. */
int sb_commit(sb_ctx* ctx, sb_seqs* seqs, const sb_tree* tree,
              const sb_verify_out* verify, const sb_accept_out* acc,
              sb_kv* target_kv, sb_kv* draft_kv, void* stream);

/* Upper bound of T over all sequences, used to size the tree-attention
 * split of the committed prefix.  sb_prefill sets it to the longest prompt
 * + 1 and every sb_commit raises it by M K + 1; a caller that writes T or
 * the caches itself must call this with a valid bound, or with 0 (unknown:
 * the page-table capacity max_pages * 16 is assumed).  A bound below the
 * true T makes attention skip the entries beyond it. */
int sb_set_length_bound(sb_ctx* ctx, int32_t max_T);

/* Device-side range checks (a debugging aid, not part of the method).  Two
 * kinds of caller-supplied index are read by kernels only: the entries of
 * the KV page tables (sb_kv.page_table) and the token ids of the prompt and
 * of sb_seqs.root.  Every such read is clamped into range (page to
 * 0 .. n_pages - 1, token to 0 .. vocab - 1), so a bad value never reads or
 * writes outside the pools or the embedding table; it silently computes on
 * the clamped index instead.  sb_set_debug(ctx, 1) waits for the device,
 * clears the context's status word and makes the kernels of later calls
 * set a bit in it for every clamp (one atomic per clamped read; nothing
 * when inputs are in range); sb_set_debug(ctx, 0) stops reporting.  sb_device_check returns
 * SB_OK at once if sb_set_debug has not been called since sb_bind (the
 * word is not cleared at bind, which touches no device memory); otherwise
 * it waits for `stream`, reads the word and, if it is not zero, clears it
 * and returns SB_EDEVICE with sb_last_error() naming the kinds of input
 * that were out of range (page-table entry, token id) since the last
 * check.  The word is per context and shared by all its streams.
 * Errors: SB_EINVAL (NULL), SB_ESTATE (not bound), SB_EHIP. */
int sb_set_debug(sb_ctx* ctx, int32_t on);
int sb_device_check(sb_ctx* ctx, void* stream);

/* Serving-time adaptation, head-only action (Sec. 3.4; the per-query
 * adaptation procedure of App. A.3; the bandit that picks the action is the
 * caller's).  Rejected positions are buffered on the device; a head update
 * steps a training copy of the drafter's LM head and rank head (the decoder
 * trunk and the final norm stay frozen) and empties the buffer. */
typedef struct sb_adapt_buffer {
  float* h;           /* device [cap][d]: h^(L) of the drafter row that
                         predicted each buffered position                   */
  int32_t* target;    /* device [cap]: the token the target chose there     */
  int32_t* count;     /* device [1]: positions held (caller zeroes it once) */
  int32_t cap;        /* host: must equal cfg.adapt_cap                     */
} sb_adapt_buffer;

typedef struct sb_head_weights {
  void* lm_head;      /* device elem [Vd][d], laid out like the bound
                         drafter LM head (bf16: packed by sb_pack_weight)   */
  float* rank_w;      /* device [4][d + 15]                                 */
  float* rank_b;      /* device [4]                                         */
} sb_head_weights;

/* Append, for each of the n_seqs sequences whose rejected position (the one
 * after the last accepted node of `acc`) has a predicting drafter row, that
 * row's cached h^(L) and the bonus token, in sequence order, while the
 * buffer has room (the rest are dropped).  Call after sb_accept /
 * sb_accept_sample and before the next sb_draft_block_expand reuses the
 * tree's rows.  Errors: SB_ESTATE (adapt_cap 0 or not bound), SB_EINVAL,
 * SB_ESHAPE (n_seqs, buf->cap). */
int sb_adapt_push(sb_ctx* ctx, int32_t n_seqs, const sb_tree* tree,
                  const sb_accept_out* acc, sb_adapt_buffer* buf,
                  void* stream);

/* One head-only step on the buffered positions i (n = min(count, cap)):
 * a_i = final_norm(h_i) (stored like the LM head's operand),
 * p_i = softmax(W_train a_i) over the drafter vocabulary, p0_i the same
 * with lm_head0 (the pre-deployment head, frozen); loss = mean over i of
 *   -log p_i(y_i)                 (y_i = target[i] as a drafter id; no term
 *                                  when it is outside a reduced vocabulary)
 *   + kl_weight KL(p_i || p0_i)
 *   - log softmax(W_r [h_i, psi_i] + b_r)(bucket of y_i's rank in p_i; b3
 *                                  past rank 10 or outside the vocabulary)
 * with psi_i and the rank labels taken before the step and held fixed; then
 * train.lm_head, rank_w, rank_b -= lr * gradient (plain SGD; the LM head is
 * rounded back to its element type), the mean loss (before the step) goes
 * to loss_out (device float, optional) and count is reset to 0.  The update
 * uses its own workspace, so it may run on another stream than inference
 * (order it after the pushes it consumes); train.lm_head must be a copy
 * distinct from the bound inference head and from lm_head0.  Errors:
 * SB_ESTATE, SB_EINVAL (pointers, lr or kl_weight negative or not finite),
 * SB_ESHAPE (buf->cap). */
int sb_head_update(sb_ctx* ctx, sb_adapt_buffer* buf, const void* lm_head0,
                   sb_head_weights* train, float lr, float kl_weight,
                   float* loss_out, void* stream);

/* Forced rank-head buckets, a synthetic workload knob for random-init
 * weights: with buckets != NULL, every later sb_draft_block_expand takes
 * the bucket of row r of sequence s from buckets[s * row_cap + r] instead of
 * the argmax of the rank-head scores (Sec. 3.2, Eq. 4; psi and the scores
 * are still computed), so that a caller can shape trees with given bucket
 * frequencies (e.g. the class frequencies of the rank-head quality table,
 * App. B).  buckets: device int32 [max_seqs][row_cap], owned by the caller,
 * read on the call's stream by each sb_draft_block_expand (its contents may
 * change between calls); values outside 0..3 are clamped to that range.
 * NULL restores the argmax.  Errors: SB_EINVAL (NULL ctx, misaligned). */
int sb_set_bucket_override(sb_ctx* ctx, const int32_t* buckets);

/* Kernel timing (the per-kernel measurements the hot path is judged by;
 * not part of the method).  While enabled, the library brackets every
 * launch of the projection GEMM, the tree attention (split kernel + merge)
 * and the vocabulary reduction with HIP events on the call's stream and
 * accumulates per class: launches, event-measured milliseconds and, for
 * the GEMM, the algorithmic bytes and flops of the rows each launch
 * actually processed (after every profiled GEMM launch a one-thread kernel
 * copies its live row count into the workspace; a launch with no rows is
 * credited no bytes, its duration still counts).  Algorithmic bytes of a
 * launch with m > 0 rows: the N x K weights and the m x K activations read,
 * m x N fp32 outputs written (the SwiGLU projection: m x N/2 bf16).
 * sb_profile(ctx, 1) resets and starts, sb_profile(ctx, 0) stops;
 * sb_profile_read waits for the recorded events and fills out[SB_PROF_N];
 * sb_profile_read_gemm fills out[SB_GEMM_N] per group of projections.
 * At most 32768 GEMM launches are recorded with their row counts per
 * sb_profile(ctx, 1); later ones are credited at their row capacity.
 * Errors: SB_EINVAL (NULL), SB_EHIP. */
enum sb_prof_class { SB_PROF_GEMM = 0, SB_PROF_ATTN = 1, SB_PROF_VOCAB = 2,
                     SB_PROF_N = 3 };
typedef struct sb_kernel_stat {
  int64_t launches;
  double total_ms;
  double bytes;
  double flops;
} sb_kernel_stat;
/* GEMM groups: target projections (QKV, O, down of sb_tree_verify and
 * sb_prefill), drafter projections (W_cond, W_fuse, W_shift and the
 * drafter's QKV, O, down), the fused gate/up + SwiGLU projections of both
 * models, and the two LM heads. */
enum sb_gemm_group { SB_GEMM_TARGET = 0, SB_GEMM_DRAFTER = 1,
                     SB_GEMM_SWIGLU = 2, SB_GEMM_LM_HEAD = 3, SB_GEMM_N = 4 };
typedef struct sb_gemm_stat {
  int64_t launches;
  int64_t launches_with_rows;
  double total_ms;
  double bytes_read;       /* algorithmic: weights + activation rows        */
  double bytes_written;    /* algorithmic: output rows                      */
  double flops;            /* 2 per multiply-add over the processed rows    */
} sb_gemm_stat;
int sb_profile(sb_ctx* ctx, int32_t enable);
int sb_profile_read(sb_ctx* ctx, sb_kernel_stat* out);
int sb_profile_read_gemm(sb_ctx* ctx, sb_gemm_stat* out);

#ifdef __cplusplus
}
#endif
#endif /* SPECBLOCK_H */
