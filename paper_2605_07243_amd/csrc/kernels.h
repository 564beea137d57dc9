// Internal launch interface between the C-ABI engine and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "specblock.h"

#define SB_MAX_SEQS 64

namespace sb {

typedef uint16_t bf16_t;

// Rows of one forward call, compacted sequence-major.  Device arrays of
// capacity `cap` rows; the active count is read on the device from *n.
struct CallPlan {
  int* n;            // [1]
  int* seq;          // [cap] sequence of the row
  int* slot;         // [cap] the row's slot in its sequence's segment
  int* pos;          // [cap] RoPE position
  int* token;        // [cap] input token (target) / start token (drafter)
  uint32_t* vis;     // [cap][vis_words] segment slots the row attends to
  int* k;            // [cap] drafter block position, 1-based
  int* pred;         // [cap] call index of the shift partner (k-1, or self)
  int* cond;         // [cap] row of the condition matrix (-1: zero vector)
  int* seq_off;      // [max_seqs + 1] first call row of each sequence
  int* prefix_len;   // [max_seqs] committed entries visible to the sequence
  int* seg_len;      // [max_seqs] valid segment slots of the sequence
  int* out_row;      // [cap] destination index of per-row outputs (or -1)
  int* kv_dst;       // [cap] cache entry the row's K/V is committed to (-1)
  int cap;
  int vis_words;
  int n_seqs;        // host value: sequences with valid seq_off entries
};

// K/V addressing: paged prefix + per-sequence segment, both in the
// [kvh][16][hd] (K) / [kvh][hd][16] (V) page layout, one layer at a time.
struct KVView {
  const void* k;            // layer base of the page pool
  const void* v;
  const int* page_table;    // [S][max_pages]
  int max_pages;
  int n_pages;              // pages in the pool (indices are clamped to it)
  const void* seg_k;        // layer base of the segment pool [S][seg_pages]
  const void* seg_v;
  int seg_pages;            // pages per sequence in the segment pool
  int* err = nullptr;       // debug status word (out-of-range pages), or null
};

// Projection GEMM plan.  bf16: 32-row activation tiles per workgroup (mf),
// 32-row weight fragments per wave (nf), weight stages in flight (pf);
// f32: mf 16-row tiles.  ks: K-chunks (partial sums).
struct GemmPlan {
  int mf, nf, pf, ks;
};
// Shapes the GEMMs take: bf16 N % 32 == 0 and K % 128 == 0 (fragment-packed
// weights); f32 N % 16 == 0 and K % 32 == 0.
bool gemm_shape_ok(int N, int K, int elem_bytes);
// retile: the call sums K-split partials in its consumer (plain
// projections); the many-row planner may then pick other tile shapes.
GemmPlan gemm_plan(int N, int K, int m_cap, int elem_bytes,
                   bool retile = false);
// Largest K-split any call of this shape may use (partial-buffer sizing).
// Kernel-attached timing of the next projection-GEMM launch (profiling).
void gemm_time_next_launch(hipEvent_t start, hipEvent_t stop);
bool gemm_time_pending();
// Kernel-attached timing of the next tree-attention call (kernel + merge).
void attn_time_next_launch(hipEvent_t start, hipEvent_t stop);
bool attn_time_pending();
int gemm_ksplit(int N, int K, int elem_bytes);
// P[ks][m][n] = X[m] . W[n] over K-chunk ks for the first *m_count rows.
// bf16 W is fragment-packed, f32 W row-major.  ksplit <= 0: the plan's
// split; otherwise at most ksplit K-chunks.  Returns the K-chunks written.
template <typename T>
int launch_gemm_xwt(const T* X, int ldx, const T* W, int N, int K, float* P,
                    size_t part_stride, const int* m_count, int m_cap,
                    int ksplit, hipStream_t st);
// Gate/up projection with SwiGLU in the epilogue (bf16; W packed with the
// gate_up interleave, [2F][K] logical): act[m][j] = silu(gate_j) * up_j for
// the first *m_count rows, act row stride F.
void launch_gemm_swiglu(const bf16_t* X, int ldx, const bf16_t* W, int F,
                        int K, bf16_t* act, const int* m_count, int m_cap,
                        hipStream_t st);
// LM head (bf16, fragment-packed W [N][K], one K-chunk) with the vocabulary
// reduction in the epilogue: for each of the first *m_count rows and each
// column tile of the launch, the record (top-1 value and id, m, s, u) the
// separate reduction would write, at rec[(row * n_chunks + tile) * 5]; the
// fp32 logits [row][N] are written too unless logits is NULL.  topk must be
// 1 (nothing is launched otherwise).  Returns n_chunks, the column tiles
// per row (gemm_vocab_chunks).
int launch_gemm_vocab(const bf16_t* X, int ldx, const bf16_t* W, int N,
                      int K, float* logits, const int* m_count, int m_cap,
                      int topk, float* rec, hipStream_t st);
int gemm_vocab_chunks(int N, int K, int m_cap);
// Row-major bf16 [rows][cols] -> fragment-packed (rows % 32, cols % 64).
int launch_pack_weight(const bf16_t* src, bf16_t* dst, int rows, int cols,
                       bool gate_up, hipStream_t st);

template <typename T>
void launch_embed(const CallPlan& p, const T* embed, int d, float* x,
                  hipStream_t st);
template <typename T>
void launch_rmsnorm(const float* x, const int* n, int cap, int d,
                    const float* g, float eps, T* out, int ldo,
                    hipStream_t st);
// x = (accumulate ? x : 0) + sum_ks P[ks]; then optionally out = rmsnorm(x)*g
// and taps[out_row][j] = x for every bit j of tap_mask.
// add_rows (optional, fp32 [.][d]): row add_rows[add_idx[i] - 1] is added
// to row i's partial sum before the residual.
template <typename T>
void launch_residual(float* x, const float* P, int ks, size_t part_stride,
                     const int* n, int cap, int d, bool accumulate,
                     const float* g, float eps, T* out, int ldo, float* taps,
                     int tap_mask, const int* out_row, hipStream_t st,
                     const float* add_rows = nullptr,
                     const int* add_idx = nullptr);
// out[k] = rmsnorm(src[k]) * g for rows k < n_rows (T rows of width d).
template <typename T>
void launch_norm_rows(const T* src, int n_rows, int d, const float* g,
                      float eps, T* out, hipStream_t st);
template <typename T>
void launch_qkv_post(const float* P, int ks, size_t part_stride,
                     const CallPlan& p, int H, int Hkv, int hd, float theta,
                     T* q, void* seg_k, void* seg_v, int seg_pages,
                     hipStream_t st);
template <typename T>
void launch_swiglu(const float* P, int ks, size_t part_stride, const int* n,
                   int cap, int F, T* out, hipStream_t st);
template <typename T>
void launch_shift_prep(const float* h, const CallPlan& p, int d, T* out,
                       hipStream_t st);
// Eq. 2 operand rows [norm_c(c), norm_e(embed(x)), norm_q(q_k)] (parts 3,
// row stride 3d) or without the q_k third (parts 2, row stride 2d).
template <typename T>
void launch_fuse_prep(const float* cond, const CallPlan& p, const T* embed,
                      const T* pos_query, const float* gc, const float* ge,
                      const float* gq, float eps, int d, T* out, int parts,
                      hipStream_t st);
// out[i] = T(src[idx[i]]) rows of width w (idx == nullptr: identity).
template <typename T>
void launch_rows_to_elem(const float* src, const int* idx, const int* n,
                         int cap, int w, T* out, hipStream_t st);

// Tree attention over paged prefix + masked segment.
// o_part / ml: split partials [max_split][cap][H][hd] / [max_split][cap][H][2]
// (used when there is more than one split, then merged by a second launch).
// n_split: splits of the fixed plan (split length max_prefix / n_split);
// the bf16 32x32 kernel may instead size the splits on the device from the
// prefix lengths (at most max_split per sequence) and then writes each
// row's split count to split_rows [cap] for the merge.
template <typename T>
void launch_tree_attn(const T* q, const CallPlan& p, const KVView& kv,
                      int rows_per_seq_cap, int H, int Hkv, int hd,
                      int n_split, int max_prefix, float* o_part, float* ml,
                      T* out, int max_split, int* split_rows, hipStream_t st);
// Query groups (workgroups) per (sequence, KV head) of a launch (seq_heads
// = the launch's sequences x KV heads, es = element bytes).
int attn_qgroups(int rows_per_seq_cap, int G, int seq_heads, int es);
// Workgroups a launch of that shape should reach for one full round of the
// chip (the split count is chosen to reach it).
int attn_workgroup_target(int rows_per_seq_cap, int G, int seq_heads, int es);

// Vocabulary reductions over fp32 logits [cap][V], in chunks of at most
// kVocabChunkMax logits (a chunk is staged in LDS); a row needs at least
// ceil(V / kVocabChunkMax) record slots.
constexpr int kVocabChunkMax = 12288;
// Returns the number of chunk records written per row (<= max_chunks).
int launch_vocab_partial(const float* logits, const int* n, int cap, int V,
                         int max_chunks, int topk, float* part,
                         hipStream_t st);
struct DraftRowOut {
  int* topk_id;
  float* topk_logit;
  float* lse;
  float* psi;
  int* bucket;
  int* branch;
  float* h_last;        // tree h_last [S][row_cap][d] (also the rank-head input)
  const int* bucket_in; // optional forced buckets [S][row_cap] (else argmax)
  const int* d2t;       // drafter id -> target id [n_vocab] (NULL: identity)
  float* lse_copy;      // the library's own copy of lse [S][row_cap]
  int n_vocab;          // drafter vocabulary (ids of the partial records)
  int row_cap;
};
void launch_draft_finalize(const float* part, int n_chunks, const CallPlan& p,
                           const float* x, const float* rank_w,
                           const float* rank_b, int d, int4 bmap,
                           DraftRowOut o, hipStream_t st);
void launch_verify_finalize(const float* part, int n_chunks, const int* n,
                            int cap, const int* out_row, int* argmax,
                            hipStream_t st);

// Tree kernels.
// Launches of a forward whose rows are usually all past the live count
// (the catch-up rows of a commit): while set (per host thread), the
// few-row GEMM, residual and RoPE launches test the count before loading
// anything, so that an empty launch exits at once.
void set_rows_likely_empty(bool v);
bool rows_likely_empty();

// Debug status bits (sb_device_check): a caller-supplied page-table entry
// or token id was outside its range and was clamped into it.
constexpr int kDevPage = 1, kDevToken = 2;

struct TreeDims {
  int S, K, M, B_max, budget;
  int bw;        // ancestor words per node
  int row_cap;   // drafter rows per sequence per iteration
  int rw;        // visibility words per drafter row
  int d;
  int V;         // target vocabulary (caller-supplied tokens are clamped to it)
  int* err;      // debug status word, or null
};
struct CommitInfo {
  int* T_old;
  int* a;
  int* cur;
  int* cont;
};
// Whole cache pools (all layers): pages [L][n_pages][Hkv][16][hd] and the
// per-sequence segment scratch [L][S][seg_pages][Hkv][16][hd].
struct KVPools {
  void* k;
  void* v;
  const int* page_table;
  int max_pages;
  int n_pages;
  void* seg_k;
  void* seg_v;
  int seg_pages;
  int* err;      // debug status word (out-of-range pages), or null
};
void launch_block1_reset(const TreeDims& td, const sb_tree& t, const int* root,
                         int* n_aux, hipStream_t st);
// Rows of one block expansion; also exports them (call_seq / call_row
// [out_cap], -1 past the call's rows, n_call).
void launch_plan_block(const TreeDims& td, int m, const sb_tree& t,
                       const int* T, const CallPlan& p, int* blk_row0,
                       int* blk_nst, int out_cap, int* call_seq,
                       int* call_row, int* n_call, hipStream_t st);
void launch_attach(const TreeDims& td, const sb_tree& t, const sb_draft_out& o,
                   const int* blk_row0, const int* blk_nst, hipStream_t st);
void launch_plan_verify(const TreeDims& td, const sb_tree& t, const int* T,
                        const CallPlan& p, hipStream_t st);
// Verifier-derived signal at the rejected position (tree.hip).
template <typename T>
void launch_reject_signal(const TreeDims& td, const sb_tree& t,
                          const sb_accept_out& acc, const float* row_lse,
                          const T* lm_head, const float* gain, float eps,
                          const int* d2t, int Vd, float* r_out,
                          hipStream_t st);
// Head-only drafter update (tree.hip push, vocab.hip rows, adapt.hip).
void launch_adapt_push(const TreeDims& td, const sb_tree& t,
                       const sb_accept_out& acc, float* buf_h, int* buf_y,
                       int* count, int cap, hipStream_t st);
void launch_adapt_rows(float* Z, const float* Z0, int Vd, const float* part,
                       const float* part0, int n_chunks, const int* n_eff,
                       int cap, const float* h, int d, const int* targets,
                       const int* d2t, const float* rank_w,
                       const float* rank_b, float kl_w, float* psi_out,
                       float* ds_out, float* loss_out, hipStream_t st);
template <typename T>
void launch_adapt_prep(const float* h, const int* count, int cap,
                       const float* g, float eps, int d, T* A, int* n_eff,
                       hipStream_t st);
template <typename T>
void launch_lm_update(T* W, int Vd, int d, const float* G, const T* A,
                      const int* n_eff, float lr, hipStream_t st);
void launch_rank_update(float* rank_w, float* rank_b, const float* ds,
                        const float* h, const float* psi, int d,
                        const int* n_eff, float lr, const float* loss,
                        float* loss_out, int* count, hipStream_t st);
int adapt_column_width(int elem_bytes);
int adapt_stripe_rows();
// Stochastic acceptance (sampling.hip).
int sample_tiles(int V);       // statistics tiles per node row
int sample_max_vocab();
void launch_node_stats(const float* logits, int V, float inv_t,
                       const int* n_nodes, int n_seqs, int budget,
                       float2* stats, hipStream_t st);
void launch_accept_sample(const TreeDims& td, const sb_tree& t,
                          const float* logits, int V, float inv_t,
                          const float2* stats, const float* u_acc,
                          const float* u_bonus, const sb_accept_out& o,
                          hipStream_t st);
void launch_accept(const TreeDims& td, const sb_tree& t, const int* argmax,
                   const sb_accept_out& o, hipStream_t st);
void launch_commit_plan(const TreeDims& td, const sb_tree& t,
                        const sb_accept_out& acc, const int* T,
                        const CommitInfo& ci, const CallPlan& fb,
                        int* taps_idx, int* n_aux, hipStream_t st);
template <typename T>
void launch_commit_copy(const TreeDims& td, const sb_tree& t,
                        const sb_accept_out& acc, const CommitInfo& ci,
                        bool drafter, const KVPools& kv, int pool_seqs,
                        int n_layers, int Hkv, int hd, hipStream_t st);
template <typename T>
void launch_seg_to_cache(const CallPlan& p, const KVPools& kv, int S,
                         int n_layers, int Hkv, int hd, hipStream_t st);
void launch_commit_state(const TreeDims& td, const sb_seqs& sq,
                         const sb_accept_out& acc, const CommitInfo& ci,
                         const float* taps, hipStream_t st);
// Prompt tokens outside 0 .. V - 1 are clamped into it (and recorded in the
// debug status word err when it is not null).
void launch_plan_prefill_target(int S, int s, int a, int n, const int* prompt,
                                int ld, const CallPlan& p, int V, int* err,
                                hipStream_t st);
void launch_plan_prefill_draft(int S, int s, int a, int n, const int* prompt,
                               int ld, const CallPlan& p, int* n_aux, int V,
                               int* err, hipStream_t st);
void launch_prefill_finish(const sb_seqs& sq, int s, int len, int d,
                           const float* taps_pf, int n_last,
                           const int* root_arg, hipStream_t st);
void launch_copy_f32(float* dst, const float* src, int n, hipStream_t st);
void launch_set_int(int* p, int v, hipStream_t st);
// *dst = *src (one thread; e.g. a row count captured for the profiler)
void launch_copy_int(int* dst, const int* src, hipStream_t st);

}  // namespace sb
