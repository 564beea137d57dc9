// Vocabulary-wide reductions over fp32 logits: top-k with ties to the
// smaller id, max, sum exp(z - max) and sum exp(z - max) z, merged exactly
// across chunks; then psi (App. B), the rank head (Eq. 4) and branching for
// drafter rows, or the greedy argmax for verified nodes.
#include <float.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace sb {

// Partial record per (row, chunk): KT values, KT ids (int bits), m, s, u.
template <int KT>
__device__ __forceinline__ void topk_insert(float (&tv)[KT], int (&ti)[KT],
                                            float v, int id) {
  if (!better(v, id, tv[KT - 1], ti[KT - 1])) return;
  tv[KT - 1] = v;
  ti[KT - 1] = id;
#pragma unroll
  for (int j = KT - 1; j > 0; --j) {
    if (better(tv[j], ti[j], tv[j - 1], ti[j - 1])) {
      const float a = tv[j];
      tv[j] = tv[j - 1];
      tv[j - 1] = a;
      const int b = ti[j];
      ti[j] = ti[j - 1];
      ti[j - 1] = b;
    }
  }
}

__device__ __forceinline__ void stats_merge(float& m, float& s, float& u,
                                            float m2, float s2, float u2) {
  const float M = fmaxf(m, m2);
  const float a = (s > 0.f) ? __expf(m - M) : 0.f;
  const float b = (s2 > 0.f) ? __expf(m2 - M) : 0.f;
  s = s * a + s2 * b;
  u = u * a + u2 * b;
  m = M;
}

// Wave-wide best (value, smaller id); every lane gets the winner.
__device__ __forceinline__ void wave_best(float& v, int& id) {
  wave_best_pair(v, id);
}

// Wave-wide merge of (m, s, u) statistics; every lane gets the result (the
// pairwise merge is symmetric, so DPP / permlane partners agree).
__device__ __forceinline__ void wave_stats(float& m, float& s, float& u) {
#define SB_STATS_DPP(C)                                                       \
  {                                                                           \
    const float m2 = dpp_f<C>(m), s2 = dpp_f<C>(s), u2 = dpp_f<C>(u);        \
    stats_merge(m, s, u, m2, s2, u2);                                         \
  }
  SB_STATS_DPP(0xB1) SB_STATS_DPP(0x4E) SB_STATS_DPP(0x141) SB_STATS_DPP(0x140)
#undef SB_STATS_DPP
  {
    const float2 a = swap16(m), b = swap16(s), c = swap16(u);
    m = a.x;
    s = b.x;
    u = c.x;
    stats_merge(m, s, u, a.y, b.y, c.y);
  }
  {
    const float2 a = swap32(m), b = swap32(s), c = swap32(u);
    m = a.x;
    s = b.x;
    u = c.x;
    stats_merge(m, s, u, a.y, b.y, c.y);
  }
}

// Pops the wave-wide top KT of per-lane sorted lists into (bv, bi).
template <int KT>
__device__ __forceinline__ void wave_topk(float (&tv)[KT], int (&ti)[KT],
                                          float (&bv)[KT], int (&bi)[KT]) {
#pragma unroll
  for (int k = 0; k < KT; ++k) {
    float v = tv[0];
    int id = ti[0];
    wave_best(v, id);
    bv[k] = v;
    bi[k] = id;
    if (ti[0] == id && tv[0] == v) {      // the owner pops its head
#pragma unroll
      for (int j = 0; j < KT - 1; ++j) {
        tv[j] = tv[j + 1];
        ti[j] = ti[j + 1];
      }
      tv[KT - 1] = -FLT_MAX;
      ti[KT - 1] = 0x7FFFFFFF;
    }
  }
}

// Candidate list of the threshold filter (values, ids) per workgroup.
constexpr int kCandCap = 256;

// Partial record of one (row, chunk).  The chunk is staged in LDS with
// coalesced 16-byte loads; a thread owns elements v0 + tid, v0 + tid + 256,
// ... .  Pass 1 takes each thread's maximum (and, for KT = 1, its first
// arg-max); pass 2 sums exp(z - max) and exp(z - max) z against that maximum
// and, for KT > 1, collects the candidates z >= T, where T is a lower bound
// of the chunk's KT-th largest logit: in each wave, the KT-th largest
// distinct value among the 64 thread maxima (KT of the wave's logits are at
// least that large), the largest over the waves.  The candidates, usually a
// dozen or two, are ordered by rank (value, then smaller id); a chunk with
// more than kCandCap candidates (many equal logits) falls back to per-thread
// sorted lists merged wave by wave.
template <int KT>
__global__ __launch_bounds__(256) void vocab_partial_kernel(
    const float* __restrict__ logits, const int* __restrict__ n, int V,
    int chunk, float* __restrict__ part) {
  const int i = blockIdx.y;
  if (i >= *n) return;
  const int c = blockIdx.x;
  const int v0 = c * chunk, v1 = min(V, v0 + chunk);
  const float* z = logits + (size_t)i * V;
  extern __shared__ float zs[];
  __shared__ float sm[4], ss[4], su[4], thr[4];
  __shared__ float cv[kCandCap], ov[4][KT];
  __shared__ int ci[kCandCap], oi[4][KT];
  __shared__ int n_cand;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (threadIdx.x == 0) n_cand = 0;
  const int nvec = v1 > v0 ? (v1 - v0) >> 2 : 0;
#pragma unroll 8
  for (int e = threadIdx.x; e < nvec; e += 256)
    reinterpret_cast<float4*>(zs)[e] =
        *reinterpret_cast<const float4*>(z + v0 + 4 * e);
  __syncthreads();
  float mx = -FLT_MAX;
  int mi = 0x7FFFFFFF;
  for (int j = v0 + threadIdx.x; j < v1; j += 256) {
    const float x = zs[j - v0];
    if (x > mx) {
      mx = x;
      mi = j;
    }
  }
  float tb = -FLT_MAX;
  if constexpr (KT > 1) {
    // KT-th distinct value among the wave's thread maxima
    float v = mx, t = -FLT_MAX;
#pragma unroll
    for (int k = 0; k < KT; ++k) {
      const float b = wave_max(v);
      t = b;
      if (v == b) v = -INFINITY;
    }
    if (lane == 0) thr[w] = t;
    __syncthreads();
    tb = fmaxf(fmaxf(fmaxf(thr[0], thr[1]), fmaxf(thr[2], thr[3])), -FLT_MAX);
  }
  float s = 0.f, u = 0.f;
  for (int j = v0 + threadIdx.x; j < v1; j += 256) {
    const float x = zs[j - v0];
    const float e = __expf(x - mx);
    s += e;
    u = fmaf(e, x, u);
    if constexpr (KT > 1) {
      if (x >= tb) {
        const int q = atomicAdd(&n_cand, 1);
        if (q < kCandCap) {
          cv[q] = x;
          ci[q] = j;
        }
      }
    }
  }
  const float m = mx;
  float M = m, S = s, U = u;
  wave_stats(M, S, U);
  if (lane == 0) {
    sm[w] = M;
    ss[w] = S;
    su[w] = U;
  }
  float* rec = part + ((size_t)i * gridDim.x + c) * (2 * KT + 3);
  if constexpr (KT == 1) {
    float bv[1] = {mx};
    int bi[1] = {mi};
    wave_best(bv[0], bi[0]);
    if (lane == 0) {
      ov[w][0] = bv[0];
      oi[w][0] = bi[0];
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      for (int q = 1; q < 4; ++q)
        if (better(ov[q][0], oi[q][0], bv[0], bi[0])) {
          bv[0] = ov[q][0];
          bi[0] = oi[q][0];
        }
      rec[0] = bv[0];
      rec[1] = __int_as_float(bi[0]);
    }
  } else {
    __syncthreads();
    const int nc = n_cand;
    if (nc <= kCandCap) {
      // rank of candidate t among the candidates; ranks < KT are the top KT
      if (threadIdx.x < nc) {
        const float x = cv[threadIdx.x];
        const int id = ci[threadIdx.x];
        int r = 0;
        for (int q = 0; q < nc; ++q) r += better(cv[q], ci[q], x, id) ? 1 : 0;
        if (r < KT) {
          rec[r] = x;
          rec[KT + r] = __int_as_float(id);
        }
      }
      if (threadIdx.x >= nc && threadIdx.x < KT) {
        rec[threadIdx.x] = -FLT_MAX;
        rec[KT + threadIdx.x] = __int_as_float(0x7FFFFFFF);
      }
    } else {
      float tv[KT];
      int ti[KT];
#pragma unroll
      for (int k = 0; k < KT; ++k) {
        tv[k] = -FLT_MAX;
        ti[k] = 0x7FFFFFFF;
      }
      for (int j = v0 + threadIdx.x; j < v1; j += 256) {
        const float x = zs[j - v0];
        if (x >= tb) topk_insert<KT>(tv, ti, x, j);
      }
      float bv[KT];
      int bi[KT];
      wave_topk<KT>(tv, ti, bv, bi);
      if (lane == 0) {
#pragma unroll
        for (int k = 0; k < KT; ++k) {
          ov[w][k] = bv[k];
          oi[w][k] = bi[k];
        }
      }
      __syncthreads();
      if (w == 0) {
        float lv[KT];
        int li[KT];
#pragma unroll
        for (int k = 0; k < KT; ++k) {
          lv[k] = lane < 4 ? ov[lane][k] : -FLT_MAX;
          li[k] = lane < 4 ? oi[lane][k] : 0x7FFFFFFF;
        }
        wave_topk<KT>(lv, li, bv, bi);
        if (lane == 0) {
#pragma unroll
          for (int k = 0; k < KT; ++k) {
            rec[k] = bv[k];
            rec[KT + k] = __int_as_float(bi[k]);
          }
        }
      }
    }
  }
  if (threadIdx.x == 0) {
    float Mb = sm[0], Sb = ss[0], Ub = su[0];
    for (int q = 1; q < 4; ++q) stats_merge(Mb, Sb, Ub, sm[q], ss[q], su[q]);
    rec[2 * KT] = Mb;
    rec[2 * KT + 1] = Sb;
    rec[2 * KT + 2] = Ub;
  }
}

int launch_vocab_partial(const float* logits, const int* n, int cap, int V,
                         int max_chunks, int topk, float* part,
                         hipStream_t st) {
  // chunks of at most kVocabChunkMax logits (48 KiB LDS stage), about 2048
  // workgroups when the row capacity allows, at most max_chunks (the record
  // buffer, sized for at least ceil(V / kVocabChunkMax))
  int n_chunks = std::max(1, std::min(max_chunks, (2048 + cap - 1) / cap));
  n_chunks = std::max(n_chunks, (V + kVocabChunkMax - 1) / kVocabChunkMax);
  const int chunk = (((V + n_chunks - 1) / n_chunks) + 3) & ~3;
  const dim3 grid(n_chunks, cap);
  const size_t lds = (size_t)chunk * sizeof(float);
  if (topk == 1)
    vocab_partial_kernel<1><<<grid, 256, lds, st>>>(logits, n, V, chunk, part);
  else
    vocab_partial_kernel<SB_TOPK_K><<<grid, 256, lds, st>>>(logits, n, V, chunk,
                                                            part);
  return n_chunks;
}

// Merge the chunk records of row i inside wave 0: top KT, m, s, u.
template <int KT>
__device__ __forceinline__ void merge_row(const float* __restrict__ part,
                                          int n_chunks, float (&bv)[KT],
                                          int (&bi)[KT], float& M, float& S,
                                          float& U) {
  const int lane = threadIdx.x & 63;
  float tv[KT];
  int ti[KT];
#pragma unroll
  for (int k = 0; k < KT; ++k) {
    tv[k] = -FLT_MAX;
    ti[k] = 0x7FFFFFFF;
  }
  float m = -FLT_MAX, s = 0.f, u = 0.f;
  for (int c = lane; c < n_chunks; c += SB_WAVE) {
    const float* o = part + (size_t)c * (2 * KT + 3);
#pragma unroll
    for (int k = 0; k < KT; ++k) topk_insert<KT>(tv, ti, o[k], __float_as_int(o[KT + k]));
    stats_merge(m, s, u, o[2 * KT], o[2 * KT + 1], o[2 * KT + 2]);
  }
  wave_stats(m, s, u);
  wave_topk<KT>(tv, ti, bv, bi);
  M = m;
  S = s;
  U = u;
}

// Merge the chunk records of row i over the whole workgroup (for the ~1000
// records per row of the LM head's fused reduction): every thread
// folds records threadIdx.x, + blockDim.x, ..., each wave reduces its
// threads' lists and statistics, and wave 0 merges the waves' (lds: one
// record per wave, at most 16 waves).  Call with every thread; the result
// is valid in wave 0.
template <int KT>
__device__ __forceinline__ void merge_row_block(const float* __restrict__ part,
                                                int n_chunks, float (&bv)[KT],
                                                int (&bi)[KT], float& M,
                                                float& S, float& U,
                                                float (*lds)[2 * KT + 3]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  float tv[KT];
  int ti[KT];
#pragma unroll
  for (int k = 0; k < KT; ++k) {
    tv[k] = -FLT_MAX;
    ti[k] = 0x7FFFFFFF;
  }
  float m = -FLT_MAX, s = 0.f, u = 0.f;
  for (int c = threadIdx.x; c < n_chunks; c += blockDim.x) {
    const float* o = part + (size_t)c * (2 * KT + 3);
#pragma unroll
    for (int k = 0; k < KT; ++k) topk_insert<KT>(tv, ti, o[k], __float_as_int(o[KT + k]));
    stats_merge(m, s, u, o[2 * KT], o[2 * KT + 1], o[2 * KT + 2]);
  }
  wave_stats(m, s, u);
  wave_topk<KT>(tv, ti, bv, bi);
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < KT; ++k) {
      lds[w][k] = bv[k];
      lds[w][KT + k] = __int_as_float(bi[k]);
    }
    lds[w][2 * KT] = m;
    lds[w][2 * KT + 1] = s;
    lds[w][2 * KT + 2] = u;
  }
  __syncthreads();
  if (w == 0) {
#pragma unroll
    for (int k = 0; k < KT; ++k) {
      tv[k] = lane < nw ? lds[lane][k] : -FLT_MAX;
      ti[k] = lane < nw ? __float_as_int(lds[lane][KT + k]) : 0x7FFFFFFF;
    }
    m = lane < nw ? lds[lane][2 * KT] : -FLT_MAX;
    s = lane < nw ? lds[lane][2 * KT + 1] : 0.f;
    u = lane < nw ? lds[lane][2 * KT + 2] : 0.f;
    wave_stats(m, s, u);
    wave_topk<KT>(tv, ti, bv, bi);
  }
  M = m;
  S = s;
  U = u;
}

// Drafter rows: top-10 ids (drafter ids mapped to target ids when the
// drafter has a reduced vocabulary), log-sum-exp,
// psi = [log p of top-10, z1-z2, z1-z3, z1-z5, p1, entropy],
// rank-head scores W_r [h^(L), psi] + b_r, bucket = argmax (ties low) or,
// when forced buckets are given, the forced one; branch = map[bucket].
// Also stores h^(L) into the tree's row cache.
__global__ __launch_bounds__(1024) void draft_finalize_kernel(
    const float* __restrict__ part, int n_chunks, CallPlan p,
    const float* __restrict__ x, const float* __restrict__ rank_w,
    const float* __restrict__ rank_b, int d, int4 bmap, DraftRowOut out) {
  __shared__ float psi_s[SB_PSI];
  __shared__ float red[16][4];
  const int i = blockIdx.x;
  if (i >= *p.n) return;
  const int o = p.out_row[i];
  // h^(L) part of the rank head: the row and four rank-head rows (d <=
  // 8192) are loaded before the record merge (they do not depend on it)
  constexpr int kMaxQ = 8;
  const float* xr = x + (size_t)i * d;
  float* hl = out.h_last + (size_t)o * d;
  const int ld = d + SB_PSI;
  float xv[kMaxQ];
  float wv[4][kMaxQ];
#pragma unroll
  for (int q = 0; q < kMaxQ; ++q) {
    const int j = threadIdx.x + 1024 * q;
    const bool in = j < d;
    xv[q] = in ? xr[j] : 0.f;
#pragma unroll
    for (int b = 0; b < 4; ++b) wv[b][q] = in ? rank_w[(size_t)b * ld + j] : 0.f;
  }
  float wp[4] = {0.f, 0.f, 0.f, 0.f};
  if (threadIdx.x < SB_PSI) {
#pragma unroll
    for (int b = 0; b < 4; ++b) wp[b] = rank_w[(size_t)b * ld + d + threadIdx.x];
  }
  if (threadIdx.x < 64) {
    float bv[SB_TOPK_K];
    int bi[SB_TOPK_K];
    float M, S, U;
    merge_row<SB_TOPK_K>(part + (size_t)i * n_chunks * (2 * SB_TOPK_K + 3),
                         n_chunks, bv, bi, M, S, U);
    if (threadIdx.x == 0) {
      const float lse = M + logf(S);
      const float ent = lse - U / S;
      for (int k = 0; k < SB_TOPK_K; ++k) {
        const int id = bi[k];
        out.topk_id[(size_t)o * SB_TOPK_K + k] =
            (out.d2t != nullptr && id >= 0 && id < out.n_vocab) ? out.d2t[id] : id;
        out.topk_logit[(size_t)o * SB_TOPK_K + k] = bv[k];
        psi_s[k] = bv[k] - lse;
      }
      psi_s[10] = bv[0] - bv[1];
      psi_s[11] = bv[0] - bv[2];
      psi_s[12] = bv[0] - bv[4];
      psi_s[13] = __expf(bv[0] - lse);
      psi_s[14] = ent;
      out.lse[o] = lse;
      out.lse_copy[o] = lse;
      for (int k = 0; k < SB_PSI; ++k) out.psi[(size_t)o * SB_PSI + k] = psi_s[k];
    }
  }
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int q = 0; q < kMaxQ; ++q)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[b] += wv[b][q] * xv[q];
#pragma unroll
  for (int q = 0; q < kMaxQ; ++q) {
    const int j = threadIdx.x + 1024 * q;
    if (j < d) hl[j] = xv[q];
  }
  __syncthreads();   // psi_s
  if (threadIdx.x < SB_PSI) {
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[b] += wp[b] * psi_s[threadIdx.x];
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const float t = wave_sum(acc[b]);
    if (lane == 0) red[w][b] = t;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int best = 0;
    float bs = 0.f;
    for (int b = 0; b < 4; ++b) {
      float sc = rank_b[b];
      for (int q = 0; q < 16; ++q) sc += red[q][b];
      if (b == 0 || sc > bs) {
        bs = sc;
        best = b;
      }
    }
    if (out.bucket_in) best = min(max(out.bucket_in[o], 0), 3);
    const int map[4] = {bmap.x, bmap.y, bmap.z, bmap.w};
    out.bucket[o] = best;
    out.branch[o] = map[best];
  }
}

void launch_draft_finalize(const float* part, int n_chunks, const CallPlan& p,
                           const float* x, const float* rank_w,
                           const float* rank_b, int d, int4 bmap,
                           DraftRowOut o, hipStream_t st) {
  draft_finalize_kernel<<<p.cap, 1024, 0, st>>>(part, n_chunks, p, x, rank_w,
                                               rank_b, d, bmap, o);
}

__global__ __launch_bounds__(256) void verify_finalize_kernel(
    const float* __restrict__ part, int n_chunks, const int* __restrict__ n,
    const int* __restrict__ out_row, int* __restrict__ argmax) {
  __shared__ float mrec[4][5];
  const int i = blockIdx.x;
  if (i >= *n) return;
  float bv[1];
  int bi[1];
  float M, S, U;
  merge_row_block<1>(part + (size_t)i * n_chunks * 5, n_chunks, bv, bi, M, S,
                     U, mrec);
  if (threadIdx.x == 0 && out_row[i] >= 0) argmax[out_row[i]] = bi[0];
}

void launch_verify_finalize(const float* part, int n_chunks, const int* n,
                            int cap, const int* out_row, int* argmax,
                            hipStream_t st) {
  verify_finalize_kernel<<<cap, 256, 0, st>>>(part, n_chunks, n, out_row,
                                              argmax);
}

// Head-only drafter update (Sec. 3.4), one workgroup per buffered position
// i: the drafter distribution p = softmax(z), z = W_train a (chunk records
// part), and p0 = softmax(z0), z0 = W_0 a (records part0); psi of p; the
// target's drafter id and rank in p, whose bucket is the rank-head label
// (past rank 10, or outside the drafter vocabulary: b3); KL(p || p0); the
// LM-logit gradient (1/n) [(p - e_y) + kl_w p (log p - log p0 - KL)]
// written over z; the rank-head score gradient
// ds = (1/n) (softmax(W_r [h, psi] + b_r) - e_label); the position's loss.
__global__ __launch_bounds__(256) void adapt_row_kernel(
    float* __restrict__ Z, const float* __restrict__ Z0, int Vd,
    const float* __restrict__ part, const float* __restrict__ part0,
    int n_chunks, const int* __restrict__ n_eff, const float* __restrict__ h,
    int d, const int* __restrict__ targets, const int* __restrict__ d2t,
    const float* __restrict__ rank_w, const float* __restrict__ rank_b,
    float kl_w, float* __restrict__ psi_out, float* __restrict__ ds_out,
    float* __restrict__ loss_out) {
  __shared__ float psi_s[SB_PSI];
  __shared__ float red[4];
  __shared__ float sh_lse, sh_lse0, sh_zy;
  __shared__ int sh_y;
  const int i = blockIdx.x;
  const int n = *n_eff;
  if (i >= n) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  float* z = Z + (size_t)i * Vd;
  const float* z0 = Z0 + (size_t)i * Vd;
  if (tid < 64) {
    float bv[SB_TOPK_K];
    int bi[SB_TOPK_K];
    float M, S, U;
    merge_row<SB_TOPK_K>(part + (size_t)i * n_chunks * (2 * SB_TOPK_K + 3),
                         n_chunks, bv, bi, M, S, U);
    float bv0[1];
    int bi0[1];
    float M0, S0, U0;
    merge_row<1>(part0 + (size_t)i * n_chunks * 5, n_chunks, bv0, bi0, M0, S0,
                 U0);
    if (tid == 0) {
      const float lse = M + logf(S);
      for (int k = 0; k < SB_TOPK_K; ++k) psi_s[k] = bv[k] - lse;
      psi_s[10] = bv[0] - bv[1];
      psi_s[11] = bv[0] - bv[2];
      psi_s[12] = bv[0] - bv[4];
      psi_s[13] = __expf(bv[0] - lse);
      psi_s[14] = lse - U / S;
      sh_lse = lse;
      sh_lse0 = M0 + logf(S0);
      // the target's drafter id (d2t strictly increasing), -1 if absent
      const int t = targets[i];
      int y = -1;
      if (d2t == nullptr) {
        y = (t >= 0 && t < Vd) ? t : -1;
      } else {
        int lo = 0, hi = Vd - 1;
        while (lo <= hi) {
          const int mid = (lo + hi) >> 1;
          const int v = d2t[mid];
          if (v == t) {
            y = mid;
            break;
          }
          if (v < t) lo = mid + 1;
          else hi = mid - 1;
        }
      }
      sh_y = y;
      sh_zy = y >= 0 ? z[y] : 0.f;
    }
  }
  __syncthreads();
  const float lse = sh_lse, lse0 = sh_lse0, zy = sh_zy;
  const int y = sh_y;
  // pass 1: KL(p || p0) and the target's rank
  float kl = 0.f, above = 0.f;
  for (int v = tid; v < Vd; v += 256) {
    const float zv = z[v];
    const float lp = zv - lse, lp0 = z0[v] - lse0;
    kl += __expf(lp) * (lp - lp0);
    if (y >= 0 && (zv > zy || (zv == zy && v < y))) above += 1.f;
  }
  kl = block_sum(kl, red);
  above = block_sum(above, red);
  const float inv_n = 1.0f / (float)n;
  // pass 2: the LM-logit gradient over z
  for (int v = tid; v < Vd; v += 256) {
    const float lp = z[v] - lse, lp0 = z0[v] - lse0;
    const float p = __expf(lp);
    // no cross-entropy term (and so no p term) for a target outside the
    // drafter vocabulary
    float g = y >= 0 ? p - (v == y ? 1.f : 0.f) : 0.f;
    g += kl_w * p * (lp - lp0 - kl);
    z[v] = g * inv_n;
  }
  // rank head over [h, psi]
  const float* hr = h + (size_t)i * d;
  const int ld = d + SB_PSI;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int j = tid; j < ld; j += 256) {
    const float x = j < d ? hr[j] : psi_s[j - d];
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[b] += rank_w[(size_t)b * ld + j] * x;
  }
  float sc[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) sc[b] = block_sum(acc[b], red) + rank_b[b];
  if (tid == 0) {
    const int r = (int)above + 1;
    const int label = y < 0 ? 3 : (r == 1 ? 0 : r <= 4 ? 1 : r <= 10 ? 2 : 3);
    const float mx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
    float se = 0.f;
    for (int b = 0; b < 4; ++b) se += __expf(sc[b] - mx);
    const float lsr = mx + logf(se);
    for (int b = 0; b < 4; ++b)
      ds_out[(size_t)i * 4 + b] =
          (__expf(sc[b] - lsr) - (b == label ? 1.f : 0.f)) * inv_n;
    for (int k = 0; k < SB_PSI; ++k) psi_out[(size_t)i * SB_PSI + k] = psi_s[k];
    float loss = kl_w * kl - (sc[label] - lsr);
    if (y >= 0) loss -= zy - lse;
    loss_out[i] = loss;
  }
}

void launch_adapt_rows(float* Z, const float* Z0, int Vd, const float* part,
                       const float* part0, int n_chunks, const int* n_eff,
                       int cap, const float* h, int d, const int* targets,
                       const int* d2t, const float* rank_w,
                       const float* rank_b, float kl_w, float* psi_out,
                       float* ds_out, float* loss_out, hipStream_t st) {
  adapt_row_kernel<<<cap, 256, 0, st>>>(Z, Z0, Vd, part, part0, n_chunks,
                                        n_eff, h, d, targets, d2t, rank_w,
                                        rank_b, kl_w, psi_out, ds_out,
                                        loss_out);
}

}  // namespace sb
