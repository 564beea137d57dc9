// Stochastic tree verification at temperature T > 0 (the paper's T = 1.0
// decoding setting, Sec. 4).  At node n with target distribution
// p_n = softmax(z_n / T) the children are tested in node-id order as
// point-mass drafts against the residual distribution (p_n with the tokens
// rejected so far removed and renormalised): child c with token x is taken
// when u_acc[c] < r(x), else x leaves the residual.  A child whose token was
// already rejected has residual probability zero and is skipped.  When no
// child is taken, the bonus token is drawn from the residual by inverse
// transform over increasing token ids with u_bonus[n].  Every emitted token
// is then distributed as the target's (speculative sampling applied
// recursively over a node's candidates).
//
// Two launches: the log-sum-exp of z / T of every verified node row (one
// workgroup per row), then the walk (one workgroup per sequence: wave 0
// walks the tree, the whole workgroup does the residual draw).
#include <float.h>

#include "common.h"
#include "kernels.h"
#include "specblock.h"

namespace sb {

namespace {

constexpr int kLseThreads = 512;
constexpr int kWalkThreads = 256;
constexpr int kMaxKids = 64;     // children tested per node (a node has at
                                 // most 2 * SB_TOPK: its continuing row and
                                 // the first row of a block started at it)

// Rows of sequences before s in call-row order (sequence-major, node order).
__device__ __forceinline__ int row_offset(const int* __restrict__ n_nodes,
                                          int s, int budget) {
  int off = 0;
  for (int j = 0; j < s; ++j) off += min(n_nodes[j], budget);
  return off;
}

__device__ __forceinline__ void lse_merge(float& m, float& s, float m2,
                                          float s2) {
  const float M = fmaxf(m, m2);
  const float a = s > 0.f ? __expf(m - M) : 0.f;
  const float b = s2 > 0.f ? __expf(m2 - M) : 0.f;
  s = s * a + s2 * b;
  m = M;
}

}  // namespace

// lse[s * budget + n] = log sum_x exp(z[row(s, n)][x] * inv_t).
__global__ __launch_bounds__(kLseThreads) void node_lse_kernel(
    const float* __restrict__ logits, int V, float inv_t,
    const int* __restrict__ n_nodes, int n_seqs, int budget,
    float* __restrict__ lse) {
  const int s = blockIdx.y, n = blockIdx.x;
  if (n >= min(n_nodes[s], budget)) return;
  const float* z = logits + (size_t)(row_offset(n_nodes, s, budget) + n) * V;
  float m = -FLT_MAX, sum = 0.f;
  for (int j = threadIdx.x; j < V; j += kLseThreads) {
    const float x = z[j] * inv_t;
    if (x > m) {
      sum = sum * __expf(m - x) + 1.f;
      m = x;
    } else {
      sum += __expf(x - m);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1)
    lse_merge(m, sum, __shfl_xor(m, o, SB_WAVE), __shfl_xor(sum, o, SB_WAVE));
  __shared__ float wm[kLseThreads / 64], ws[kLseThreads / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) {
    wm[w] = m;
    ws[w] = sum;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < kLseThreads / 64; ++i) lse_merge(m, sum, wm[i], ws[i]);
    lse[(size_t)s * budget + n] = m + logf(sum);
  }
}

__global__ __launch_bounds__(kWalkThreads) void accept_sample_kernel(
    TreeDims td, sb_tree t, const float* __restrict__ logits, int V,
    float inv_t, const float* __restrict__ lse,
    const float* __restrict__ u_acc, const float* __restrict__ u_bonus,
    sb_accept_out out) {
  __shared__ int par[512], tok[512];
  __shared__ int kid[kMaxKids];
  __shared__ float kp[kMaxKids], ku[kMaxKids];
  __shared__ int rej[kMaxKids];
  __shared__ int sh_cur, sh_nrej, sh_bonus;
  __shared__ double csum[kWalkThreads];
  const int s = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const size_t nb = (size_t)s * td.budget;
  const int nn = min(t.n_nodes[s], td.budget);
  const int off = row_offset(t.n_nodes, s, td.budget);
  const int path_cap = td.M * td.K;
  for (int j = tid; j < nn; j += kWalkThreads) {
    par[j] = t.parent[nb + j];
    tok[j] = t.token[nb + j];
  }
  __syncthreads();
  if (tid < 64) {
    // ---- the walk, wave 0 ----
    int cur = 0, a = 0, nrej = 0;
    while (true) {
      // children of cur in node-id order (ballot compaction)
      int nk = 0;
      for (int j0 = 1; j0 < nn; j0 += 64) {
        const int j = j0 + lane;
        const bool f = j < nn && par[j] == cur;
        const uint64_t mk = __ballot(f);
        const int pos = nk + __popcll(mk & ((1ull << lane) - 1ull));
        if (f && pos < kMaxKids) kid[pos] = j;
        nk += __popcll(mk);
      }
      nk = min(nk, kMaxKids);
      const size_t zrow = (size_t)(off + cur) * V;
      const float l = lse[nb + cur];
      if (lane < nk) {
        const int c = kid[lane];
        const int x = tok[c];
        // a token outside the vocabulary has no target mass
        kp[lane] = (x >= 0 && x < V) ? __expf(logits[zrow + x] * inv_t - l)
                                     : 0.f;
        ku[lane] = u_acc[nb + c];
      }
      // sequential tests (lane 0), result broadcast through LDS
      if (lane == 0) {
        int next = -1;
        float mass = 1.f;
        nrej = 0;
        for (int i = 0; i < nk; ++i) {
          const int x = tok[kid[i]];
          bool seen = false;
          for (int r = 0; r < nrej; ++r) seen |= rej[r] == x;
          if (seen) continue;
          if (ku[i] < kp[i] / mass) {
            next = kid[i];
            break;
          }
          rej[nrej++] = x;
          mass -= kp[i];
        }
        sh_cur = next;
        sh_nrej = nrej;
      }
      __builtin_amdgcn_wave_barrier();
      const int next = sh_cur;
      nrej = sh_nrej;
      if (next < 0 || a >= path_cap) break;
      if (lane == 0) out.path[(size_t)s * path_cap + a] = next;
      cur = next;
      ++a;
    }
    if (lane == 0) {
      out.n_accepted[s] = a;
      sh_cur = cur;
      sh_nrej = nrej;
    }
  }
  __syncthreads();
  // ---- residual draw at the last node, whole workgroup ----
  const int cur = sh_cur, nrej = sh_nrej;
  const float* z = logits + (size_t)(off + cur) * V;
  const float l = lse[nb + cur];
  const int chunk = (V + kWalkThreads - 1) / kWalkThreads;
  const int v0 = min(V, tid * chunk), v1 = min(V, v0 + chunk);
  // cumulative masses in float64: the draw's boundaries then carry only the
  // float32 error of the individual probabilities, not of a long sum
  double part = 0.0;
  for (int x = v0; x < v1; ++x) {
    bool r = false;
    for (int i = 0; i < nrej; ++i) r |= rej[i] == x;
    if (!r) part += (double)__expf(z[x] * inv_t - l);
  }
  csum[tid] = part;
  if (tid == 0) sh_bonus = -1;
  __syncthreads();
  // inclusive scan of the chunk masses (Hillis-Steele over LDS)
  for (int o = 1; o < kWalkThreads; o <<= 1) {
    const double v = tid >= o ? csum[tid - o] : 0.0;
    __syncthreads();
    csum[tid] += v;
    __syncthreads();
  }
  const double total = csum[kWalkThreads - 1];
  const double target = (double)u_bonus[nb + cur] * total;
  const double lo = tid > 0 ? csum[tid - 1] : 0.0;
  if (lo <= target && target < csum[tid] && part > 0.0) {
    double acc = lo;
    int pick = -1, last = -1;
    for (int x = v0; x < v1 && pick < 0; ++x) {
      bool r = false;
      for (int i = 0; i < nrej; ++i) r |= rej[i] == x;
      if (r) continue;
      const float p = __expf(z[x] * inv_t - l);
      if (p > 0.f) last = x;
      acc += (double)p;
      if (acc > target) pick = x;
    }
    // rounding can leave the chunk's own running sum short of its scanned
    // end; the chunk's last positive token is then the draw
    atomicMax(&sh_bonus, pick >= 0 ? pick : last);
  }
  __syncthreads();
  if (tid == 0) {
    int b = sh_bonus;
    if (b < 0) {
      // target at or past the total (rounding): the last token with mass
      for (int x = V - 1; x >= 0 && b < 0; --x) {
        bool r = false;
        for (int i = 0; i < nrej; ++i) r |= rej[i] == x;
        if (!r && __expf(z[x] * inv_t - l) > 0.f) b = x;
      }
      if (b < 0) b = 0;
    }
    out.bonus[s] = b;
  }
}

void launch_node_lse(const float* logits, int V, float inv_t,
                     const int* n_nodes, int n_seqs, int budget, float* lse,
                     hipStream_t st) {
  dim3 grid(budget, n_seqs);
  node_lse_kernel<<<grid, kLseThreads, 0, st>>>(logits, V, inv_t, n_nodes,
                                                n_seqs, budget, lse);
}

void launch_accept_sample(const TreeDims& td, const sb_tree& t,
                          const float* logits, int V, float inv_t,
                          const float* lse, const float* u_acc,
                          const float* u_bonus, const sb_accept_out& o,
                          hipStream_t st) {
  accept_sample_kernel<<<td.S, kWalkThreads, 0, st>>>(td, t, logits, V, inv_t,
                                                      lse, u_acc, u_bonus, o);
}

}  // namespace sb
