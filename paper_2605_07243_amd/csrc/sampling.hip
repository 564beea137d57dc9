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
// Two launches.  First the softmax statistics (max, sum of exp) of z / T
// for every verified node row, one workgroup per 16384-token tile of a row
// so that a row is read by many CUs at once.  Then the walk, one workgroup
// per sequence: wave 0 merges the tile statistics of the nodes it visits and
// runs the tests; the whole workgroup does the residual draw, streaming the
// last node's row tile by tile through LDS (coalesced loads) with each
// thread owning 64 consecutive tokens of a tile, so that the cumulative
// masses in token order are a scan over (tile, thread) in float64.
#include <float.h>

#include "common.h"
#include "kernels.h"
#include "specblock.h"

namespace sb {

namespace {

constexpr int kThreads = 256;
constexpr int kTile = 16384;          // tokens per tile (64 per thread)
constexpr int kMaxTiles = 16;         // V <= 262144
constexpr int kMaxKids = 64;          // children tested per node (a node has
                                      // at most 2 * SB_TOPK: its continuing
                                      // row and the first row of a block
                                      // started at it)

// Rows of sequences before s in call-row order (sequence-major, node order).
__device__ __forceinline__ int row_offset(const int* __restrict__ n_nodes,
                                          int s, int budget) {
  int off = 0;
  for (int j = 0; j < s; ++j) off += min(n_nodes[j], budget);
  return off;
}

__device__ __forceinline__ void stat_merge(float& m, float& s, float m2,
                                           float s2) {
  const float M = fmaxf(m, m2);
  const float a = s > 0.f ? __expf(m - M) : 0.f;
  const float b = s2 > 0.f ? __expf(m2 - M) : 0.f;
  s = s * a + s2 * b;
  m = M;
}

}  // namespace

// stats[(s * budget + n) * n_tiles + j] = (max, sum exp(x - max)) over the
// tokens of tile j of node n's row, x = z * inv_t.
__global__ __launch_bounds__(kThreads) void node_stats_kernel(
    const float* __restrict__ logits, int V, float inv_t,
    const int* __restrict__ n_nodes, int budget, int n_tiles,
    float2* __restrict__ stats) {
  const int j = blockIdx.x, n = blockIdx.y, s = blockIdx.z;
  if (n >= min(n_nodes[s], budget)) return;
  const float* z = logits + (size_t)(row_offset(n_nodes, s, budget) + n) * V;
  const int base = j * kTile;
  float4 v[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int e = base + 4 * (threadIdx.x + kThreads * q);
    v[q] = e < V ? *reinterpret_cast<const float4*>(z + e)
                 : make_float4(-FLT_MAX, -FLT_MAX, -FLT_MAX, -FLT_MAX);
  }
  float m = -FLT_MAX;
#pragma unroll
  for (int q = 0; q < 16; ++q)
    m = fmaxf(m, fmaxf(fmaxf(v[q].x, v[q].y), fmaxf(v[q].z, v[q].w)) * inv_t);
  float sum = 0.f;
  if (m > -FLT_MAX) {
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int e = base + 4 * (threadIdx.x + kThreads * q);
      if (e < V)
        sum += __expf(v[q].x * inv_t - m) + __expf(v[q].y * inv_t - m) +
               __expf(v[q].z * inv_t - m) + __expf(v[q].w * inv_t - m);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1)
    stat_merge(m, sum, __shfl_xor(m, o, SB_WAVE), __shfl_xor(sum, o, SB_WAVE));
  __shared__ float wm[kThreads / 64], ws[kThreads / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) {
    wm[w] = m;
    ws[w] = sum;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < kThreads / 64; ++i) stat_merge(m, sum, wm[i], ws[i]);
    stats[((size_t)s * budget + n) * n_tiles + j] = make_float2(m, sum);
  }
}

__global__ __launch_bounds__(kThreads) void accept_sample_kernel(
    TreeDims td, sb_tree t, const float* __restrict__ logits, int V,
    float inv_t, const float2* __restrict__ stats, int n_tiles,
    const float* __restrict__ u_acc, const float* __restrict__ u_bonus,
    sb_accept_out out) {
  __shared__ int par[512], tok[512];
  __shared__ int kid[kMaxKids];
  __shared__ float kp[kMaxKids], ku[kMaxKids];
  __shared__ int rej[kMaxKids];
  __shared__ int sh_cur, sh_nrej, sh_bonus;
  __shared__ float sh_lse;
  // a tile of probabilities, padded so that thread t's 64 tokens start at
  // 65 t (conflict-free reads), then the (thread, tile) scan of group masses
  __shared__ float tile[kThreads * 65];
  __shared__ double scan[kThreads][kMaxTiles + 1];   // padded rows
  __shared__ double wtot[kThreads / 64][kMaxTiles];
  const int s = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const size_t nb = (size_t)s * td.budget;
  const int nn = min(t.n_nodes[s], td.budget);
  const int off = row_offset(t.n_nodes, s, td.budget);
  const int path_cap = td.M * td.K;
  for (int j = tid; j < nn; j += kThreads) {
    par[j] = t.parent[nb + j];
    tok[j] = t.token[nb + j];
  }
  __syncthreads();
  if (tid < 64) {
    // ---- the walk, wave 0 ----
    int cur = 0, a = 0, nrej = 0;
    float l = 0.f;
    while (true) {
      // log-sum-exp of the node's row from its tile statistics
      {
        float m = -FLT_MAX, sm = 0.f;
        if (lane < n_tiles) {
          const float2 st = stats[(nb + cur) * n_tiles + lane];
          m = st.x;
          sm = st.y;
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1)
          stat_merge(m, sm, __shfl_xor(m, o, SB_WAVE),
                     __shfl_xor(sm, o, SB_WAVE));
        l = m + logf(sm);
      }
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
      sh_lse = l;
      sh_bonus = -1;
    }
  }
  __syncthreads();
  // ---- residual draw at the last node, whole workgroup ----
  // (runtime loops: this code runs once per launch, so its size, not its
  // trip counts, sets the instruction-fetch cost)
  const int cur = sh_cur, nrej = sh_nrej;
  const float l = sh_lse;
  const float* z = logits + (size_t)(off + cur) * V;
  const int w = tid >> 6;
  // tile j's logits in registers while tile j - 1 is summed
  float4 v[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int e = 4 * (tid + kThreads * q);
    v[q] = e < V ? *reinterpret_cast<const float4*>(z + e)
                 : make_float4(-FLT_MAX, -FLT_MAX, -FLT_MAX, -FLT_MAX);
  }
#pragma unroll 1
  for (int j = 0; j < n_tiles; ++j) {
    const int base = j * kTile;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int e = 4 * (tid + kThreads * q);
      float* d = tile + e + e / 64;
      // -FLT_MAX (past the vocabulary) gives exp = 0
      d[0] = __expf(v[q].x * inv_t - l);
      d[1] = __expf(v[q].y * inv_t - l);
      d[2] = __expf(v[q].z * inv_t - l);
      d[3] = __expf(v[q].w * inv_t - l);
    }
    if (j + 1 < n_tiles) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int e = base + kTile + 4 * (tid + kThreads * q);
        v[q] = e < V ? *reinterpret_cast<const float4*>(z + e)
                     : make_float4(-FLT_MAX, -FLT_MAX, -FLT_MAX, -FLT_MAX);
      }
    }
    __syncthreads();
    // rejected tokens leave the residual
    if (tid < nrej) {
      const int x = rej[tid] - base;
      if (x >= 0 && x < kTile) tile[x + x / 64] = 0.f;
    }
    __syncthreads();
    double g = 0.0;
#pragma unroll 8
    for (int i = 0; i < 64; ++i) g += (double)tile[65 * tid + i];
    // inclusive scan over the wave's threads
    double incl = g;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const double t = __shfl_up(incl, o, SB_WAVE);
      if (lane >= o) incl += t;
    }
    scan[tid][j] = incl;
    if (lane == 63) wtot[w][j] = incl;
    __syncthreads();
  }
  double total = 0.0;
#pragma unroll 1
  for (int j = 0; j < n_tiles; ++j)
    total += (wtot[0][j] + wtot[1][j]) + (wtot[2][j] + wtot[3][j]);
  const double target = (double)u_bonus[nb + cur] * total;
  double toff = 0.0;
#pragma unroll 1
  for (int j = 0; j < n_tiles; ++j) {
    double bw = toff;
    for (int i = 0; i < w; ++i) bw += wtot[i][j];
    const double lo = bw + (lane > 0 ? scan[tid - 1][j] : 0.0);
    const double hi = bw + scan[tid][j];
    toff += (wtot[0][j] + wtot[1][j]) + (wtot[2][j] + wtot[3][j]);
    if (hi > lo && lo <= target && target < hi) {
      // the group's residual probabilities, all loads in flight at once,
      // into this thread's own (no longer shared) slice of the tile buffer
      const int x0 = j * kTile + 64 * tid;
      float* my = tile + 65 * tid;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int x = x0 + 4 * q;
        const float4 u = x < V ? *reinterpret_cast<const float4*>(z + x)
                               : make_float4(-FLT_MAX, -FLT_MAX, -FLT_MAX,
                                             -FLT_MAX);
        my[4 * q] = __expf(u.x * inv_t - l);
        my[4 * q + 1] = __expf(u.y * inv_t - l);
        my[4 * q + 2] = __expf(u.z * inv_t - l);
        my[4 * q + 3] = __expf(u.w * inv_t - l);
      }
#pragma unroll 1
      for (int i = 0; i < nrej; ++i) {
        const int x = rej[i] - x0;
        if (x >= 0 && x < 64) my[x] = 0.f;
      }
      double acc = lo;
      int pick = -1, last = -1;
#pragma unroll 1
      for (int i = 0; i < 64 && pick < 0; ++i) {
        const float p = my[i];
        if (p > 0.f) last = x0 + i;
        acc += (double)p;
        if (acc > target) pick = x0 + i;
      }
      // rounding can leave the group's running sum short of its scanned
      // end; the group's last positive token is then the draw
      atomicMax(&sh_bonus, pick >= 0 ? pick : last);
    }
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

int sample_tiles(int V) { return (V + kTile - 1) / kTile; }
int sample_max_vocab() { return kTile * kMaxTiles; }

void launch_node_stats(const float* logits, int V, float inv_t,
                       const int* n_nodes, int n_seqs, int budget,
                       float2* stats, hipStream_t st) {
  dim3 grid(sample_tiles(V), budget, n_seqs);
  node_stats_kernel<<<grid, kThreads, 0, st>>>(logits, V, inv_t, n_nodes,
                                               budget, sample_tiles(V), stats);
}

void launch_accept_sample(const TreeDims& td, const sb_tree& t,
                          const float* logits, int V, float inv_t,
                          const float2* stats, const float* u_acc,
                          const float* u_bonus, const sb_accept_out& o,
                          hipStream_t st) {
  accept_sample_kernel<<<td.S, kThreads, 0, st>>>(
      td, t, logits, V, inv_t, stats, sample_tiles(V), u_acc, u_bonus, o);
}

}  // namespace sb
