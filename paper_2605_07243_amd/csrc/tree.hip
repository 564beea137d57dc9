// Tree bookkeeping on the device: row plans for each forward call, rank-
// guided sibling attachment and next-block starts (Sec. 3.2, Alg. 2), the
// greedy acceptance walk and the commit copies.  Small single-workgroup or
// one-wave-per-sequence kernels; nothing here synchronises with the host.
#include <float.h>

#include "bounds.h"
#include "common.h"
#include "kernels.h"
#include "specblock.h"

namespace sb {

// ---------------------------------------------------------------------------
// Block 1: reset the tree to the root (node 0, one start) and count the
// W_cond rows (one per sequence).
__global__ void block1_reset_kernel(TreeDims td, sb_tree t,
                                    const int* __restrict__ root,
                                    int* __restrict__ n_aux) {
  for (int s = threadIdx.x; s < td.S; s += blockDim.x) {
    const size_t b = (size_t)s * td.budget;
    t.n_nodes[s] = 1;
    t.token[b] = checked_index(root[s], td.V, td.err, kDevToken);
    t.parent[b] = -1;
    t.depth[b] = 0;
    t.row[b] = -1;
    t.rank[b] = 0;
    t.logp[b] = 0.f;
    t.cum_logp[b] = 0.f;
    for (int w = 0; w < td.bw; ++w) t.anc[b * td.bw + w] = (w == 0) ? 1u : 0u;
    t.n_rows[s] = 0;
    t.n_starts[s] = 1;
    t.starts[(size_t)s * td.B_max] = 0;
  }
  if (threadIdx.x == 0) *n_aux = td.S;
}

// Rows of one block expansion: start b of sequence s gets rows k = 1..K at
// positions pos(start) + k; they see the rows visible to the row that
// proposed the start plus their own block's rows <= k.
// The call rows are also exported (call_seq / call_row [out_cap], -1 past
// the rows, n_call).
__global__ void plan_block_kernel(TreeDims td, int m, sb_tree t,
                                  const int* __restrict__ T, CallPlan p,
                                  int* __restrict__ blk_row0,
                                  int* __restrict__ blk_nst, int out_cap,
                                  int* __restrict__ call_seq,
                                  int* __restrict__ call_row,
                                  int* __restrict__ n_call) {
  __shared__ int cnt[SB_MAX_SEQS], old[SB_MAX_SEQS], off[SB_MAX_SEQS + 1];
  __shared__ int Ts[SB_MAX_SEQS];
  const int K = td.K, rw = td.rw;
  const int tid = threadIdx.x;
  // every sequence's counts loaded at once (one thread each), offsets by a
  // scan in LDS, then one pass over all rows: no chain of dependent global
  // round trips per sequence
  if (tid < td.S) {
    const int s = tid;
    const int n_old = t.n_rows[s];
    int nst = min(t.n_starts[s], td.B_max);
    nst = max(0, min(nst, (td.row_cap - n_old) / K));
    cnt[s] = nst * K;
    old[s] = n_old;
    Ts[s] = T[s];
    p.prefix_len[s] = Ts[s];
    p.seg_len[s] = n_old + nst * K;
    blk_row0[s] = n_old;
    blk_nst[s] = nst;
  }
  __syncthreads();
  if (tid == 0) {
    int o = 0;
    for (int s = 0; s < td.S; ++s) {
      off[s] = o;
      o += cnt[s];
    }
    off[td.S] = o;
  }
  __syncthreads();
  const int total = off[td.S];
  if (tid <= td.S) p.seq_off[tid] = off[tid];
  if (tid == 0) {
    *p.n = total;
    *n_call = total;
  }
  for (int i = total + tid; i < out_cap; i += blockDim.x) {
    call_seq[i] = -1;
    call_row[i] = -1;
  }
  for (int i = tid; i < total; i += blockDim.x) {
    int s = 0;
    while (off[s + 1] <= i) ++s;
    const int j = i - off[s];
    const int b = j / K, k = j % K + 1;
    const int lr = old[s] + j;
    call_seq[i] = s;
    call_row[i] = lr;
    const int sn = t.starts[(size_t)s * td.B_max + b];
    const size_t nidx = (size_t)s * td.budget + sn;
    const int srow = t.row[nidx];
    const int pos = Ts[s] + t.depth[nidx] + k;
    p.seq[i] = s;
    p.slot[i] = lr;
    p.pos[i] = pos;
    p.token[i] = t.token[nidx];
    p.k[i] = k;
    p.pred[i] = k > 1 ? i - 1 : i;
    p.cond[i] = (m == 1 || srow < 0) ? s : s * td.row_cap + srow;
    p.out_row[i] = s * td.row_cap + lr;
    p.kv_dst[i] = -1;
    const size_t rbase = (size_t)s * td.row_cap;
    for (int w = 0; w < rw; ++w) {
      uint32_t bits = (m > 1 && srow >= 0) ? t.row_vis[(rbase + srow) * rw + w] : 0u;
      // own block rows lr-k+1 .. lr
      for (int q = lr - k + 1; q <= lr; ++q)
        if ((q >> 5) == w) bits |= 1u << (q & 31);
      t.row_vis[(rbase + lr) * rw + w] = bits;
      p.vis[(size_t)i * p.vis_words + w] = bits;
    }
    t.row_block[rbase + lr] = m;
    t.row_start[rbase + lr] = sn;
    t.row_k[rbase + lr] = k;
    t.row_pos[rbase + lr] = pos;
  }
  __syncthreads();
  if (tid < td.S) t.n_rows[tid] = old[tid] + cnt[tid];
}

// Sibling attachment of one block in (k, start, rank) order within the
// budget, then the next block's starts.  One wave per sequence; lane b owns
// start b of the block.  The block's row results (branch, bucket, lse,
// top-10 ids and logits: rows row0 .. row0 + nst K - 1, at most 512) are
// staged in LDS with coalesced loads before the attachment loop, and the
// cumulative log-probability of every new node that qualifies as a next
// start is kept in LDS, so that the loop and the start selection read no
// global memory.
constexpr int kAttachRows = 512;
__global__ __launch_bounds__(64) void attach_kernel(
    TreeDims td, sb_tree t, const int* __restrict__ topk_id,
    const float* __restrict__ topk_logit, const float* __restrict__ lse,
    const int* __restrict__ bucket, const int* __restrict__ branch,
    const int* __restrict__ blk_row0, const int* __restrict__ blk_nst) {
  __shared__ int ids_s[kAttachRows * SB_TOPK_K];
  __shared__ float lg_s[kAttachRows * SB_TOPK_K];
  __shared__ float lse_s[kAttachRows];
  __shared__ int br_s[kAttachRows];
  __shared__ int bk_s[kAttachRows];
  __shared__ float cand_s[kAttachRows];   // new node id - first_new
  const int s = blockIdx.x;
  const int lane = threadIdx.x;
  const int K = td.K, budget = td.budget, bw = td.bw;
  const int nst = blk_nst[s];
  const int row0 = blk_row0[s];
  const size_t nb = (size_t)s * budget;
  const size_t rb = (size_t)s * td.row_cap;
  const int nrows = min(nst * K, kAttachRows);
  const bool mine = lane < nst;
  // independent loads first: the block's rows, the start nodes
  for (int e = lane; e < nrows * SB_TOPK_K; e += 64) {
    ids_s[e] = topk_id[(rb + row0) * SB_TOPK_K + e];
    lg_s[e] = topk_logit[(rb + row0) * SB_TOPK_K + e];
  }
  for (int j = lane; j < nrows; j += 64) {
    lse_s[j] = lse[rb + row0 + j];
    br_s[j] = branch[rb + row0 + j];
    bk_s[j] = bucket[rb + row0 + j];
  }
  for (int j = lane; j < budget; j += 64) cand_s[j] = -FLT_MAX;
  int chain = mine ? t.starts[(size_t)s * td.B_max + lane] : 0;
  bool alive = mine;
  int chain_depth = 0;
  float chain_cum = 0.f;
  uint32_t chain_anc[SB_MAX_ANC_WORDS];
#pragma unroll
  for (int w = 0; w < SB_MAX_ANC_WORDS; ++w) chain_anc[w] = 0u;
  if (mine) {
    chain_depth = t.depth[nb + chain];
    chain_cum = t.cum_logp[nb + chain];
#pragma unroll
    for (int w = 0; w < SB_MAX_ANC_WORDS; ++w)
      if (w < bw) chain_anc[w] = t.anc[(nb + chain) * bw + w];
  }
  int nn = t.n_nodes[s];
  const int first_new = nn;
  __syncthreads();
  for (int k = 1; k <= K; ++k) {
    const int j = lane * K + (k - 1);          // block-local row
    const int r = row0 + j;
    const bool live = mine && alive && j < nrows;
    const int want = live ? br_s[j] : 0;   // 0..10
    int total;
    const int excl = wave_excl_scan_small<4>(want, total);
    const int id0 = nn + excl;
    if (live) {
      const float l0 = lse_s[j];
      const int bk = bk_s[j];
      const bool cand_row = bk == 1 || bk == 2;
      for (int rank = 1; rank <= want; ++rank) {
        const int id = id0 + rank - 1;
        if (id >= budget) break;
        const int q = j * SB_TOPK_K + (rank - 1);
        const float lp = lg_s[q] - l0;
        t.token[nb + id] = ids_s[q];
        t.parent[nb + id] = chain;
        t.depth[nb + id] = chain_depth + 1;
        t.row[nb + id] = r;
        t.rank[nb + id] = rank;
        t.logp[nb + id] = lp;
        t.cum_logp[nb + id] = chain_cum + lp;
        if (rank >= 2 && cand_row) cand_s[id - first_new] = chain_cum + lp;
#pragma unroll
        for (int w = 0; w < SB_MAX_ANC_WORDS; ++w)
          if (w < bw)
            t.anc[(nb + id) * bw + w] =
                chain_anc[w] | ((id >> 5) == w ? (1u << (id & 31)) : 0u);
      }
      if (want >= 1 && id0 < budget) {
        chain = id0;
        chain_depth += 1;
        chain_cum += lg_s[j * SB_TOPK_K] - l0;
#pragma unroll
        for (int w = 0; w < SB_MAX_ANC_WORDS; ++w)
          if ((id0 >> 5) == w) chain_anc[w] |= 1u << (id0 & 31);
      } else {
        alive = false;
      }
    }
    nn = min(budget, nn + total);
  }
  if (lane == 0) t.n_nodes[s] = nn;
  __syncthreads();   // candidate values of all lanes visible below
  // next-block starts: chain ends first, then rank >= 2 siblings of b1/b2
  // rows by cumulative log-probability (ties: lower node id)
  int* out = t.starts + (size_t)s * td.B_max;
  if (nn >= budget) {
    if (lane == 0) t.n_starts[s] = 0;
    return;
  }
  int n_ends;
  const int is_end = (mine && alive) ? 1 : 0;
  const int e_excl = wave_excl_scan_small<1>(is_end, n_ends);
  if (is_end && e_excl < td.B_max) out[e_excl] = chain;
  int taken = min(n_ends, td.B_max);
  // candidate mask per lane: node first_new + lane + 64 q
  uint32_t cand = 0u;
  for (int q = 0; q < 8; ++q) {
    const int id = first_new + lane + 64 * q;
    if (id < nn && cand_s[id - first_new] > -FLT_MAX) cand |= 1u << q;
  }
  while (taken < td.B_max) {
    float bv = -FLT_MAX;
    int bi = 0x7FFFFFFF;
    for (int q = 0; q < 8; ++q) {
      if (cand & (1u << q)) {
        const int id = first_new + lane + 64 * q;
        const float v = cand_s[id - first_new];
        if (better(v, id, bv, bi)) {
          bv = v;
          bi = id;
        }
      }
    }
    float v = bv;
    int id = bi;
    wave_best_pair(v, id);
    if (id == 0x7FFFFFFF) break;
    if (lane == 0) out[taken] = id;
    if (((id - first_new) & 63) == lane) cand &= ~(1u << ((id - first_new) >> 6));
    ++taken;
  }
  if (lane == 0) t.n_starts[s] = taken;
}

// Verification rows: every node of every tree at T + depth, seeing its
// ancestors-or-self.
__global__ void plan_verify_kernel(TreeDims td, sb_tree t,
                                   const int* __restrict__ T, CallPlan p) {
  __shared__ int off[SB_MAX_SEQS + 1];
  __shared__ int Ts[SB_MAX_SEQS];
  const int tid = threadIdx.x;
  // counts loaded at once, offsets by a scan in LDS, one pass over all rows
  if (tid < td.S) {
    off[tid + 1] = min(t.n_nodes[tid], td.budget);
    Ts[tid] = T[tid];
  }
  __syncthreads();
  if (tid == 0) {
    off[0] = 0;
    for (int s = 0; s < td.S; ++s) off[s + 1] += off[s];
  }
  __syncthreads();
  const int total = off[td.S];
  if (tid < td.S) {
    p.prefix_len[tid] = Ts[tid];
    p.seg_len[tid] = off[tid + 1] - off[tid];
  }
  if (tid <= td.S) p.seq_off[tid] = off[tid];
  if (tid == 0) *p.n = total;
  for (int i = tid; i < total; i += blockDim.x) {
    int s = 0;
    while (off[s + 1] <= i) ++s;
    const int j = i - off[s];
    const size_t nidx = (size_t)s * td.budget + j;
    p.seq[i] = s;
    p.slot[i] = j;
    p.pos[i] = Ts[s] + t.depth[nidx];
    p.token[i] = t.token[nidx];
    p.k[i] = 1;
    p.pred[i] = i;
    p.cond[i] = -1;
    p.out_row[i] = s * td.budget + j;
    p.kv_dst[i] = -1;
    for (int w = 0; w < p.vis_words; ++w)
      p.vis[(size_t)i * p.vis_words + w] = w < td.bw ? t.anc[nidx * td.bw + w] : 0u;
  }
}

// Greedy acceptance walk, one wave per sequence.
__global__ __launch_bounds__(64) void accept_kernel(TreeDims td, sb_tree t,
                                                    const int* __restrict__ argmax,
                                                    sb_accept_out out) {
  const int s = blockIdx.x;
  const int lane = threadIdx.x;
  const size_t nb = (size_t)s * td.budget;
  const int nn = min(t.n_nodes[s], td.budget);
  const int path_cap = td.M * td.K;
  int cur = 0, a = 0;
  while (a < path_cap) {
    const int g = argmax[nb + cur];
    int best = 0x7FFFFFFF;
    for (int j = 1 + lane; j < nn; j += 64)
      if (t.parent[nb + j] == cur && t.token[nb + j] == g) best = min(best, j);
    best = wave_min_i(best);
    if (best == 0x7FFFFFFF) break;
    if (lane == 0) out.path[(size_t)s * path_cap + a] = best;
    cur = best;
    ++a;
  }
  if (lane == 0) {
    out.n_accepted[s] = a;
    out.bonus[s] = argmax[nb + cur];
  }
}

// The drafter row at position pos(cur) + 1 on a path through node cur: the
// next row of cur's block when cur is a chain node short of K, else row 1 of
// a block started at cur; -1 when the tree has none.
__device__ int continuing_row(const TreeDims& td, const sb_tree& t, int s,
                              int cur) {
  const size_t nb = (size_t)s * td.budget;
  const size_t rb = (size_t)s * td.row_cap;
  const int nrows = t.n_rows[s];
  if (cur == 0) return nrows > 0 ? 0 : -1;
  const int r = t.row[nb + cur];
  if (t.rank[nb + cur] == 1 && t.row_k[rb + r] < td.K && r + 1 < nrows)
    return r + 1;
  for (int j = 0; j < nrows; ++j)
    if (t.row_start[rb + j] == cur && t.row_k[rb + j] == 1) return j;
  return -1;
}

// Commit planning: last accepted node, the drafter row continuing it (or a
// catch-up row when the tree has none) and the catch-up call plan.
__global__ void commit_plan_kernel(TreeDims td, sb_tree t, sb_accept_out acc,
                                   const int* __restrict__ T, CommitInfo ci,
                                   CallPlan fb, int* __restrict__ taps_idx,
                                   int* __restrict__ n_aux) {
  const int path_cap = td.M * td.K;
  for (int s = threadIdx.x; s < td.S; s += blockDim.x) {
    const size_t nb = (size_t)s * td.budget;
    const size_t rb = (size_t)s * td.row_cap;
    const int a = acc.n_accepted[s];
    const int cur = a > 0 ? acc.path[(size_t)s * path_cap + a - 1] : 0;
    const int cont = continuing_row(td, t, s, cur);
    ci.T_old[s] = T[s];
    ci.a[s] = a;
    ci.cur[s] = cur;
    ci.cont[s] = cont;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int o = 0;
    for (int s = 0; s < td.S; ++s) {
      fb.seq_off[s] = o;
      const int a = ci.a[s];
      fb.prefix_len[s] = ci.T_old[s] + a;   // drafter entries 1..T+a
      if (ci.cont[s] < 0) {
        const int cur = ci.cur[s];
        const size_t nb = (size_t)s * td.budget;
        fb.seq[o] = s;
        fb.slot[o] = 0;
        fb.pos[o] = ci.T_old[s] + a + 1;
        fb.token[o] = t.token[nb + cur];
        fb.k[o] = 1;
        fb.pred[o] = o;
        fb.cond[o] = o;
        fb.out_row[o] = -1;
        fb.kv_dst[o] = ci.T_old[s] + a;
        for (int w = 0; w < fb.vis_words; ++w)
          fb.vis[(size_t)o * fb.vis_words + w] = (w == 0) ? 1u : 0u;
        fb.seg_len[s] = 1;
        taps_idx[o] = s * td.budget + max(t.parent[nb + cur], 0);
        ++o;
      } else {
        fb.seg_len[s] = 0;
      }
    }
    fb.seq_off[td.S] = o;
    *fb.n = o;
    *n_aux = o;
  }
}

// Copy committed K/V entries.  Target: the root and accepted nodes (verify
// scratch slot = node id) to entries T .. T+a.  Drafter: the rows that
// proposed the accepted nodes to entries T .. T+a-1 (positions T+1 ..
// T+a), and the continuing row, if any, to entry T+a.
template <typename T>
__global__ void commit_copy_kernel(TreeDims td, sb_tree t, sb_accept_out acc,
                                   CommitInfo ci, int drafter, KVPools kv,
                                   int pool_seqs, int Hkv, int hd) {
  const int s = blockIdx.x;
  const int j = blockIdx.y;               // 0 .. M K
  const int l = blockIdx.z / Hkv, kh = blockIdx.z % Hkv;
  const int a = ci.a[s];
  const int T0 = ci.T_old[s];
  const int path_cap = td.M * td.K;
  int src_slot, dst;
  if (!drafter) {
    if (j > a) return;
    src_slot = j == 0 ? 0 : acc.path[(size_t)s * path_cap + j - 1];
    dst = T0 + j;
  } else {
    if (j < a) {
      const int node = acc.path[(size_t)s * path_cap + j];
      src_slot = t.row[(size_t)s * td.budget + node];
      dst = T0 + j;
    } else if (j == a && ci.cont[s] >= 0) {
      src_slot = ci.cont[s];
      dst = T0 + a;
    } else {
      return;
    }
  }
  // entries outside the page table (a negative T included) are not written
  if (dst < 0 || (dst >> 4) >= kv.max_pages) return;
  const int page_i = dst >> 4;
  const int page = checked_index(kv.page_table[(size_t)s * kv.max_pages + page_i],
                                 kv.n_pages, kv.err, kDevPage);
  const int sl = dst & 15;
  const int sp = src_slot >> 4, ss = src_slot & 15;
  if (sp >= kv.seg_pages) return;
  const size_t lay = (size_t)l;
  const size_t src_page = ((lay * pool_seqs + s) * kv.seg_pages + sp) * Hkv + kh;
  const size_t dst_page = (lay * kv.n_pages + page) * Hkv + kh;
  const T* sk = static_cast<const T*>(kv.seg_k) + src_page * 16 * hd;
  const T* sv = static_cast<const T*>(kv.seg_v) + src_page * 16 * hd;
  T* dk = static_cast<T*>(kv.k) + dst_page * 16 * hd;
  T* dv = static_cast<T*>(kv.v) + dst_page * 16 * hd;
  for (int e = threadIdx.x; e < hd; e += blockDim.x) {
    dk[sl * hd + e] = sk[ss * hd + e];
    dv[e * 16 + sl] = sv[e * 16 + ss];
  }
}

// Rows of a plan whose kv_dst >= 0: segment slot -> cache entry kv_dst.
template <typename T>
__global__ void seg_to_cache_kernel(CallPlan p, KVPools kv, int S, int Hkv,
                                    int hd) {
  const int i = blockIdx.x;
  if (i >= *p.n) return;
  const int dst = p.kv_dst[i];
  if (dst < 0) return;
  const int l = blockIdx.y / Hkv, kh = blockIdx.y % Hkv;
  const int s = p.seq[i], slot = p.slot[i];
  const int page_i = dst >> 4;
  if (page_i >= kv.max_pages) return;
  const int page = checked_index(kv.page_table[(size_t)s * kv.max_pages + page_i],
                                 kv.n_pages, kv.err, kDevPage);
  const int sl = dst & 15;
  const int sp = slot >> 4, ss = slot & 15;
  if (sp >= kv.seg_pages) return;
  const size_t src_page = (((size_t)l * S + s) * kv.seg_pages + sp) * Hkv + kh;
  const size_t dst_page = ((size_t)l * kv.n_pages + page) * Hkv + kh;
  const T* sk = static_cast<const T*>(kv.seg_k) + src_page * 16 * hd;
  const T* sv = static_cast<const T*>(kv.seg_v) + src_page * 16 * hd;
  T* dk = static_cast<T*>(kv.k) + dst_page * 16 * hd;
  T* dv = static_cast<T*>(kv.v) + dst_page * 16 * hd;
  for (int e = threadIdx.x; e < hd; e += blockDim.x) {
    dk[sl * hd + e] = sk[ss * hd + e];
    dv[e * 16 + sl] = sv[e * 16 + ss];
  }
}

__global__ void commit_state_kernel(TreeDims td, sb_seqs sq, sb_accept_out acc,
                                    CommitInfo ci, const float* __restrict__ taps) {
  const int s = blockIdx.x;
  const int cur = ci.cur[s];
  // 3 d floats (d % 32 == 0): float4 copy, every load issued before the
  // stores (the destination cannot alias the taps)
  const float4* __restrict__ src = reinterpret_cast<const float4*>(
      taps + ((size_t)s * td.budget + cur) * 3 * td.d);
  float4* __restrict__ dst =
      reinterpret_cast<float4*>(sq.cond_taps + (size_t)s * 3 * td.d);
  const int n4 = 3 * td.d / 4;
  for (int e = threadIdx.x; e < n4; e += blockDim.x) dst[e] = src[e];
  if (threadIdx.x == 0) {
    sq.T[s] = ci.T_old[s] + ci.a[s] + 1;
    sq.root[s] = acc.bonus[s];
  }
}

// Prefill of sequence s, chunk [a, a + n): target rows (causal chain).
__global__ void plan_prefill_target_kernel(int S, int s, int a, int n,
                                           const int* __restrict__ prompt,
                                           int ld, CallPlan p, int V,
                                           int* __restrict__ err) {
  if (threadIdx.x == 0) {
    for (int q = 0; q <= S; ++q) p.seq_off[q] = q <= s ? 0 : n;
    for (int q = 0; q < S; ++q) {
      p.prefix_len[q] = q == s ? a : 0;
      p.seg_len[q] = q == s ? n : 0;
    }
    *p.n = n;
  }
  for (int j = threadIdx.x; j < n; j += blockDim.x) {
    p.seq[j] = s;
    p.slot[j] = j;
    p.pos[j] = a + j;
    p.token[j] = checked_index(prompt[(size_t)s * ld + a + j], V, err, kDevToken);
    p.k[j] = 1;
    p.pred[j] = j;
    p.cond[j] = -1;
    p.out_row[j] = 1 + j;          // taps slot in the prefill tap buffer
    p.kv_dst[j] = a + j;
    for (int w = 0; w < p.vis_words; ++w) {
      uint32_t bits = 0u;
      for (int q = 32 * w; q < 32 * w + 32 && q <= j; ++q) bits |= 1u << (q & 31);
      p.vis[(size_t)j * p.vis_words + w] = bits;
    }
  }
}

// Prefill drafter catch-up rows for positions a+1 .. a+n: row r is a K = 1
// block started at position a + r with token x_{a+r}, conditioned on the
// target taps of position a + r - 1 (tap buffer slot r; none for position 1).
__global__ void plan_prefill_draft_kernel(int S, int s, int a, int n,
                                          const int* __restrict__ prompt,
                                          int ld, CallPlan p,
                                          int* __restrict__ n_aux, int V,
                                          int* __restrict__ err) {
  if (threadIdx.x == 0) {
    for (int q = 0; q <= S; ++q) p.seq_off[q] = q <= s ? 0 : n;
    for (int q = 0; q < S; ++q) {
      p.prefix_len[q] = q == s ? a : 0;
      p.seg_len[q] = q == s ? n : 0;
    }
    *p.n = n;
    *n_aux = n;
  }
  for (int r = threadIdx.x; r < n; r += blockDim.x) {
    p.seq[r] = s;
    p.slot[r] = r;
    p.pos[r] = a + 1 + r;
    p.token[r] = checked_index(prompt[(size_t)s * ld + a + r], V, err, kDevToken);
    p.k[r] = 1;
    p.pred[r] = r;
    p.cond[r] = (a + r >= 1) ? r : -1;
    p.out_row[r] = -1;
    p.kv_dst[r] = a + r;
    for (int w = 0; w < p.vis_words; ++w) {
      uint32_t bits = 0u;
      for (int q = 32 * w; q < 32 * w + 32 && q <= r; ++q) bits |= 1u << (q & 31);
      p.vis[(size_t)r * p.vis_words + w] = bits;
    }
  }
}

// Prefill end of sequence s: T = len, root = argmax of the last row,
// cond_taps = taps of position len - 1 (tap buffer slot n_last).
__global__ void prefill_finish_kernel(sb_seqs sq, int s, int len, int d,
                                      const float* __restrict__ taps_pf,
                                      int n_last, const int* __restrict__ root_arg) {
  float* dst = sq.cond_taps + (size_t)s * 3 * d;
  const float* src = taps_pf + (size_t)n_last * 3 * d;
  for (int e = threadIdx.x; e < 3 * d; e += blockDim.x) dst[e] = src[e];
  if (threadIdx.x == 0) {
    sq.T[s] = len;
    sq.root[s] = root_arg[0];
  }
}

__global__ void copy_f32_kernel(float* __restrict__ dst, const float* __restrict__ src,
                                int n) {
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < n; e += gridDim.x * blockDim.x)
    dst[e] = src[e];
}

__global__ void set_int_kernel(int* __restrict__ p, int v) { *p = v; }

__global__ void copy_int_kernel(int* __restrict__ dst,
                                const int* __restrict__ src) {
  *dst = *src;
}

// ---------------------------------------------------------------------------
// launchers

void launch_block1_reset(const TreeDims& td, const sb_tree& t, const int* root,
                         int* n_aux, hipStream_t st) {
  block1_reset_kernel<<<1, 64, 0, st>>>(td, t, root, n_aux);
}
void launch_plan_block(const TreeDims& td, int m, const sb_tree& t,
                       const int* T, const CallPlan& p, int* blk_row0,
                       int* blk_nst, int out_cap, int* call_seq,
                       int* call_row, int* n_call, hipStream_t st) {
  plan_block_kernel<<<1, 256, 0, st>>>(td, m, t, T, p, blk_row0, blk_nst,
                                       out_cap, call_seq, call_row, n_call);
}
void launch_attach(const TreeDims& td, const sb_tree& t, const sb_draft_out& o,
                   const int* blk_row0, const int* blk_nst, hipStream_t st) {
  attach_kernel<<<td.S, 64, 0, st>>>(td, t, o.topk_id, o.topk_logit, o.lse,
                                     o.bucket, o.branch, blk_row0, blk_nst);
}
void launch_plan_verify(const TreeDims& td, const sb_tree& t, const int* T,
                        const CallPlan& p, hipStream_t st) {
  plan_verify_kernel<<<1, 256, 0, st>>>(td, t, T, p);
}
// Verifier-derived update signal (Sec. 3.4, Eq. 8): at the rejected position
// (the one after the last accepted node, where the bonus token stands), the
// drafter's probability r of the target's token, from the row that predicted
// that position: r = exp(z[bonus] - lse) with z[bonus] = W_lm[bonus] .
// norm(h^(L)) recomputed from the row's cached h^(L) (the final RMSNorm and
// the LM-head operand rounding of the drafter forward), lse the row's
// log-sum-exp.  -1 when no drafter row predicts that position; 0 when the
// bonus token is outside a reduced drafter vocabulary.
template <typename T>
__global__ __launch_bounds__(256) void reject_signal_kernel(
    TreeDims td, sb_tree t, sb_accept_out acc, const float* __restrict__ row_lse,
    const T* __restrict__ lm_head, const float* __restrict__ gain, float eps,
    const int* __restrict__ d2t, int Vd, float* __restrict__ r_out) {
  __shared__ float red[4];
  __shared__ int sh_id;
  const int s = blockIdx.x, tid = threadIdx.x;
  const int path_cap = td.M * td.K;
  const int a = acc.n_accepted[s];
  const int cur = a > 0 ? acc.path[(size_t)s * path_cap + a - 1] : 0;
  const int cont = continuing_row(td, t, s, cur);
  if (cont < 0) {
    if (tid == 0) r_out[s] = -1.f;
    return;
  }
  const int bonus = acc.bonus[s];
  if (tid == 0) {
    int id = -1;
    if (d2t == nullptr) {
      id = (bonus >= 0 && bonus < Vd) ? bonus : -1;
    } else {   // d2t is strictly increasing: binary search
      int lo = 0, hi = Vd - 1;
      while (lo <= hi) {
        const int mid = (lo + hi) >> 1;
        const int v = d2t[mid];
        if (v == bonus) {
          id = mid;
          break;
        }
        if (v < bonus) lo = mid + 1;
        else hi = mid - 1;
      }
    }
    sh_id = id;
  }
  __syncthreads();
  const int id = sh_id;
  if (id < 0) {
    if (tid == 0) r_out[s] = 0.f;
    return;
  }
  const int d = td.d;
  const size_t o = (size_t)s * td.row_cap + cont;
  const float* h = t.h_last + o * d;
  const int lane = tid & 63, w = tid >> 6;
  float ss = 0.f;
  for (int k = tid; k < d; k += 256) ss += h[k] * h[k];
  ss = wave_sum(ss);
  if (lane == 0) red[w] = ss;
  __syncthreads();
  const float rs = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
  __syncthreads();
  // eight consecutive columns per step: one 16-byte run of the packed
  // (or row-major) LM-head row, all loads independent
  float z = 0.f;
  for (int k0 = 8 * tid; k0 < d; k0 += 8 * 256) {
    size_t wi;
    if constexpr (sizeof(T) == 2) {
      // fragment-packed LM head (32-row x 64-column blocks)
      const int c = k0 & 63;
      const int l = (id & 31) + 32 * (c >> 5);
      wi = ((((size_t)(k0 >> 6) * (Vd >> 5) + (id >> 5)) * 4 + ((c & 31) >> 3)) *
            512) + (size_t)l * 8;
    } else {
      wi = (size_t)id * d + k0;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = Elem<T>::to_f32(
          Elem<T>::from_f32(h[k0 + e] * rs * gain[k0 + e]));
      z += Elem<T>::to_f32(lm_head[wi + e]) * x;
    }
  }
  z = wave_sum(z);
  if (lane == 0) red[w] = z;
  __syncthreads();
  if (tid == 0)
    r_out[s] = __expf((red[0] + red[1] + red[2] + red[3]) - row_lse[o]);
}

void launch_accept(const TreeDims& td, const sb_tree& t, const int* argmax,
                   const sb_accept_out& o, hipStream_t st) {
  accept_kernel<<<td.S, 64, 0, st>>>(td, t, argmax, o);
}
// Adaptation buffer push (Sec. 3.4): each sequence's rejected position
// (the one after its last accepted node) whose drafter row exists appends
// (that row's cached h^(L), the bonus token) to the buffer, in sequence
// order, while room is left.  One workgroup.
__global__ __launch_bounds__(256) void adapt_push_kernel(
    TreeDims td, sb_tree t, sb_accept_out acc, float* __restrict__ buf_h,
    int* __restrict__ buf_y, int* __restrict__ count, int cap) {
  __shared__ int slot[SB_MAX_SEQS], src[SB_MAX_SEQS];
  const int path_cap = td.M * td.K;
  if (threadIdx.x < td.S) {
    const int s = threadIdx.x;
    const int a = acc.n_accepted[s];
    const int cur = a > 0 ? acc.path[(size_t)s * path_cap + a - 1] : 0;
    src[s] = continuing_row(td, t, s, cur);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int c = *count;
    for (int s = 0; s < td.S; ++s) {
      slot[s] = (src[s] >= 0 && c < cap) ? c : -1;
      if (slot[s] >= 0) {
        buf_y[slot[s]] = acc.bonus[s];
        ++c;
      }
    }
    *count = c;
  }
  __syncthreads();
  const int d = td.d;
  for (int s = 0; s < td.S; ++s) {
    if (slot[s] < 0) continue;
    const float* hs = t.h_last + ((size_t)s * td.row_cap + src[s]) * d;
    float* hd = buf_h + (size_t)slot[s] * d;
    for (int k = threadIdx.x; k < d; k += 256) hd[k] = hs[k];
  }
}

void launch_adapt_push(const TreeDims& td, const sb_tree& t,
                       const sb_accept_out& acc, float* buf_h, int* buf_y,
                       int* count, int cap, hipStream_t st) {
  adapt_push_kernel<<<1, 256, 0, st>>>(td, t, acc, buf_h, buf_y, count, cap);
}

template <typename T>
void launch_reject_signal(const TreeDims& td, const sb_tree& t,
                          const sb_accept_out& acc, const float* row_lse,
                          const T* lm_head, const float* gain, float eps,
                          const int* d2t, int Vd, float* r_out,
                          hipStream_t st) {
  reject_signal_kernel<T><<<td.S, 256, 0, st>>>(td, t, acc, row_lse, lm_head,
                                                gain, eps, d2t, Vd, r_out);
}
template void launch_reject_signal<float>(const TreeDims&, const sb_tree&,
                                          const sb_accept_out&, const float*,
                                          const float*, const float*, float,
                                          const int*, int, float*,
                                          hipStream_t);
template void launch_reject_signal<bf16_t>(const TreeDims&, const sb_tree&,
                                           const sb_accept_out&, const float*,
                                           const bf16_t*, const float*, float,
                                           const int*, int, float*,
                                           hipStream_t);
void launch_commit_plan(const TreeDims& td, const sb_tree& t,
                        const sb_accept_out& acc, const int* T,
                        const CommitInfo& ci, const CallPlan& fb,
                        int* taps_idx, int* n_aux, hipStream_t st) {
  commit_plan_kernel<<<1, 64, 0, st>>>(td, t, acc, T, ci, fb, taps_idx, n_aux);
}
template <typename T>
void launch_commit_copy(const TreeDims& td, const sb_tree& t,
                        const sb_accept_out& acc, const CommitInfo& ci,
                        bool drafter, const KVPools& kv, int pool_seqs,
                        int n_layers, int Hkv, int hd, hipStream_t st) {
  dim3 grid(td.S, td.M * td.K + 1, n_layers * Hkv);
  commit_copy_kernel<T><<<grid, 128, 0, st>>>(td, t, acc, ci, drafter ? 1 : 0,
                                              kv, pool_seqs, Hkv, hd);
}
template <typename T>
void launch_seg_to_cache(const CallPlan& p, const KVPools& kv, int S,
                         int n_layers, int Hkv, int hd, hipStream_t st) {
  dim3 grid(p.cap, n_layers * Hkv);
  seg_to_cache_kernel<T><<<grid, 128, 0, st>>>(p, kv, S, Hkv, hd);
}
void launch_commit_state(const TreeDims& td, const sb_seqs& sq,
                         const sb_accept_out& acc, const CommitInfo& ci,
                         const float* taps, hipStream_t st) {
  commit_state_kernel<<<td.S, 1024, 0, st>>>(td, sq, acc, ci, taps);
}
void launch_plan_prefill_target(int S, int s, int a, int n, const int* prompt,
                                int ld, const CallPlan& p, int V, int* err,
                                hipStream_t st) {
  plan_prefill_target_kernel<<<1, 256, 0, st>>>(S, s, a, n, prompt, ld, p, V,
                                                err);
}
void launch_plan_prefill_draft(int S, int s, int a, int n, const int* prompt,
                               int ld, const CallPlan& p, int* n_aux, int V,
                               int* err, hipStream_t st) {
  plan_prefill_draft_kernel<<<1, 256, 0, st>>>(S, s, a, n, prompt, ld, p,
                                               n_aux, V, err);
}
void launch_prefill_finish(const sb_seqs& sq, int s, int len, int d,
                           const float* taps_pf, int n_last,
                           const int* root_arg, hipStream_t st) {
  prefill_finish_kernel<<<1, 256, 0, st>>>(sq, s, len, d, taps_pf, n_last,
                                           root_arg);
}
void launch_copy_f32(float* dst, const float* src, int n, hipStream_t st) {
  copy_f32_kernel<<<(n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024, 256, 0,
                    st>>>(dst, src, n);
}
void launch_set_int(int* p, int v, hipStream_t st) {
  set_int_kernel<<<1, 1, 0, st>>>(p, v);
}
void launch_copy_int(int* dst, const int* src, hipStream_t st) {
  copy_int_kernel<<<1, 1, 0, st>>>(dst, src);
}

template void launch_commit_copy<float>(const TreeDims&, const sb_tree&,
                                        const sb_accept_out&, const CommitInfo&,
                                        bool, const KVPools&, int, int, int,
                                        int, hipStream_t);
template void launch_commit_copy<bf16_t>(const TreeDims&, const sb_tree&,
                                         const sb_accept_out&,
                                         const CommitInfo&, bool,
                                         const KVPools&, int, int, int, int,
                                         hipStream_t);
template void launch_seg_to_cache<float>(const CallPlan&, const KVPools&, int,
                                         int, int, int, hipStream_t);
template void launch_seg_to_cache<bf16_t>(const CallPlan&, const KVPools&, int,
                                          int, int, int, hipStream_t);

}  // namespace sb
