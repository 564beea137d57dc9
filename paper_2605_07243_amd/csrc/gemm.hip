// Projection GEMMs on MFMA (gfx950).
//
//   P[ks][m][n] = sum_{k in K-chunk ks} X[m][k] * W[n][k]
//
// X holds the activation rows of a call (their count is read on the device),
// W is a [N][K] weight matrix.  K-chunks (the split of the contraction
// across workgroups) write separate partial sums that the consumer kernel
// adds, which keeps results independent of scheduling order.
//
// bf16 (gemm_tile_kernel).  Weights are stored fragment-packed (the layout
// sb_pack_weight writes): 32-row x 64-column blocks of 4 KiB, K-block-major,
// block (rb, kb) at element offset (kb * N/32 + rb) * 2048 (the waves that
// stream neighbouring row blocks at the same K-stage read neighbouring
// 4 KiB blocks), and inside a block
// four 1 KiB sub-steps i, lane l holding the 8 elements
//   W[32 rb + l % 32][64 kb + 32 (l / 32) + 8 i + e],  e = 0..7.
// That is the A operand of v_mfma_f32_32x32x16_bf16 for sub-step i when the
// contraction index of the 64-column block is permuted so that lane group
// l / 32 owns 32 consecutive columns; the activation operand is read with
// the same permutation, so the product is unchanged.  Every weight load of
// a wave is one contiguous 1 KiB, straight into registers (no LDS pass), a
// few K-stages ahead of the MFMAs.
//
// A workgroup (4 waves) owns 32 MF activation rows and 128 NF weight rows
// (32 NF per wave).  The activation K-slice is staged once per workgroup in
// LDS (double buffered, rows padded so the 16-byte MFMA operand reads are
// conflict-free) and read by all waves; activation rows are therefore the
// MFMA B operand and a lane's outputs are four consecutive features of one
// row (one 16-byte store).  Workgroup ids are remapped so that the
// workgroups resident on one XCD (ids congruent mod 8) take consecutive
// tiles: the activation row tiles of one weight tile run on the same XCD
// and share its weight lines in that XCD's L2.
//
// The SwiGLU variant reads a gate/up weight packed with 16 gate rows and the
// matching 16 up rows per 32-row block: a lane then holds gate and up of the
// same features and writes act = silu(gate) * up directly.
//
// f32 (gemm_xwt_kernel): row-major weights, fragments load straight into
// registers and eight v_mfma_f32_16x16x4_f32 per 32-wide step.
#include <float.h>
#include <hip/hip_ext.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace sb {

typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// acc[32x32] += A[32 x 16] * B[16 x 32]; lane l holds row l % 32 of A and
// column l % 32 of B, each with 8 contraction indices of lane group l / 32.
// Output register r of lane l: acc[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].
__device__ __forceinline__ f32x16_t mma_32x32x16(u32x4_t a, u32x4_t b,
                                                 f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(
      __builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c, 0,
      0, 0);
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

// Vocabulary records of the LM-head epilogue (the same record the separate
// reduction writes: KT values, KT ids as int bits, then m, s = sum exp(z - m)
// and u = sum exp(z - m) z).  Top-KT keeps the larger value first, equal
// values ordered by the smaller id.
template <int KT>
__device__ __forceinline__ void vr_insert(float (&tv)[KT], int (&ti)[KT],
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

__device__ __forceinline__ void vr_stats_merge(float& m, float& s, float& u,
                                               float m2, float s2, float u2) {
  const float M = fmaxf(m, m2);
  const float a = (s > 0.f) ? __expf(m - M) : 0.f;
  const float b = (s2 > 0.f) ? __expf(m2 - M) : 0.f;
  s = s * a + s2 * b;
  u = u * a + u2 * b;
  m = M;
}

// MF: 32-row activation tiles per workgroup; NF: 32-row weight fragments
// per wave; PF: K-stages (64 columns each) of weights in flight per wave.
// VR > 0 (LM heads, one K-chunk): besides (or, with P == nullptr, instead
// of) the fp32 outputs, each workgroup writes for every row the vocabulary
// record (top VR, m, s, u) of its 128 NF output columns to
// rec[(row * n_nt + column tile) * (2 VR + 3)].  n_first (a multiple of
// 32 NF; 0 with VR > 0): the launch covers weight rows n_first .. N - 1, in
// n_nt column tiles from there.
template <int MF, int NF, int PF, bool SWIGLU, int VR>
__global__ __launch_bounds__(256) void gemm_tile_kernel(
    const bf16_t* X, int ldx, const bf16_t* W, int K, float* __restrict__ P,
    int N, size_t part_stride, const int* __restrict__ m_count, int k_chunk,
    int n_mt, int n_nt, bf16_t* __restrict__ act, int F,
    float* __restrict__ rec, int n_first, int x_rows) {
  static_assert(PF == 2 || PF == 4, "weight ring depth");
  constexpr int BM = 32 * MF;
  constexpr int LD = 64 + 8;
  __shared__ __attribute__((aligned(16))) bf16_t xs[2][BM][LD];
  const int total = gridDim.x;
  int b = blockIdx.x;
  b = xcd_grouped(b, total);
  const int mt = b % n_mt;
  const int rest = b / n_mt;
  const int nt = rest % n_nt;
  const int kc = rest / n_nt;
  const int m_base = mt * BM;
  // live rows (a scalar load; it is waited for only at the exit test below)
  const int M = *m_count;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 31, h = lane >> 5;
  const int nb = n_first + nt * (128 * NF) + wave * (32 * NF);  // first row
  const bool wave_on = nb < N;                         // N % 32 == 0 tails
  const int kc0 = kc * k_chunk;
  const int nstage = k_chunk / 64;
  const size_t kstride = (size_t)(N / 32) * 2048;   // one K-block of all rows
  const bf16_t* wp[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int rb = min((nb >> 5) + f, N / 32 - 1);
    wp[f] = W + (size_t)(kc0 / 64) * kstride + (size_t)rb * 2048 + lane * 8;
  }
  u32x4_t wq[PF][NF][4];
  u32x4_t xq[2][MF];
  f32x16_t acc[MF][NF];
#pragma unroll
  for (int t = 0; t < MF; ++t)
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[t][f][r] = 0.f;

  // Stage s: weights in wq[s % PF], activations in LDS buffer s & 1.
  // Iteration s first writes the activations of stage s + 1 (fetched into
  // registers one iteration earlier) to the other LDS buffer, fetches those
  // of stage s + 2 into the freed register slot, and then runs the four
  // MFMA sub-steps; after sub-step i the weight registers of that sub-step
  // are refilled with stage s + PF.  The barrier at the end finds the LDS
  // writes long done.  Stage indices past the chunk re-read its last stage
  // (results unused) so that every iteration issues the same loads.
#define SB_SCHED __builtin_amdgcn_sched_barrier(0);
#define SB_ISSUE_W(p, s_)                                                     \
  {                                                                           \
    const size_t so = (size_t)min((s_), nstage - 1) * kstride;                \
    _Pragma("unroll") for (int f = 0; f < NF; ++f)                            \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) wq[p][f][i] =               \
        *reinterpret_cast<const u32x4_t*>(wp[f] + so + 512 * i);              \
  }
#define SB_ISSUE_WI(p, s_, i)                                                 \
  {                                                                           \
    const size_t so = (size_t)min((s_), nstage - 1) * kstride;                \
    _Pragma("unroll") for (int f = 0; f < NF; ++f) wq[p][f][i] =              \
        *reinterpret_cast<const u32x4_t*>(wp[f] + so + 512 * (i));            \
  }
#define SB_ISSUE_X(slot, s_)                                                  \
  {                                                                           \
    const size_t so = (size_t)min((s_), nstage - 1) * 64;                     \
    _Pragma("unroll") for (int q = 0; q < MF; ++q) xq[slot][q] =              \
        *reinterpret_cast<const u32x4_t*>(xp[q] + so);                        \
  }
#define SB_STORE_X(slot, buf)                                                 \
  {                                                                           \
    _Pragma("unroll") for (int q = 0; q < MF; ++q) {                          \
      const int c = tid + 256 * q;                                            \
      *reinterpret_cast<u32x4_t*>(&xs[buf][c / 8][8 * (c % 8)]) = xq[slot][q]; \
    }                                                                         \
  }
#define SB_READ_X(dst, buf, i)                                                \
  _Pragma("unroll") for (int t = 0; t < MF; ++t) dst[t] =                     \
      *reinterpret_cast<const u32x4_t*>(&xs[buf][32 * t + lr][32 * h + 8 * (i)]);
#define SB_MMA(p, i, src)                                                     \
  _Pragma("unroll") for (int t = 0; t < MF; ++t)                              \
  _Pragma("unroll") for (int f = 0; f < NF; ++f)                              \
    acc[t][f] = mma_32x32x16(wq[p][f][i], src[t], acc[t][f]);
  // the activation operands of sub-step i + 1 are read from LDS while the
  // MFMAs of sub-step i run
#define SB_STAGE(p)                                                           \
  {                                                                           \
    const int s = s0 + (p);                                                   \
    u32x4_t xa[MF], xb[MF];                                                   \
    SB_STORE_X(((p) + 1) & 1, ((p) + 1) & 1)                                  \
    SB_READ_X(xa, (p) & 1, 0)                                                 \
    SB_ISSUE_X((p) & 1, s + 2)                                                \
    SB_READ_X(xb, (p) & 1, 1)                                                 \
    SB_SCHED SB_MMA(p, 0, xa) SB_SCHED                                        \
    SB_ISSUE_WI(p, s + PF, 0)                                                 \
    SB_READ_X(xa, (p) & 1, 2)                                                 \
    SB_SCHED SB_MMA(p, 1, xb) SB_SCHED                                        \
    SB_ISSUE_WI(p, s + PF, 1)                                                 \
    SB_READ_X(xb, (p) & 1, 3)                                                 \
    SB_SCHED SB_MMA(p, 2, xa) SB_SCHED                                        \
    SB_ISSUE_WI(p, s + PF, 2)                                                 \
    SB_SCHED SB_MMA(p, 3, xb) SB_SCHED                                        \
    SB_ISSUE_WI(p, s + PF, 3)                                                 \
    __syncthreads();                                                          \
  }
  // A launch with one activation row tile (a few rows: the projections of
  // one or a few sequences) streams weights for a short time and pays for
  // every round trip at its start, so there the first stages' loads, which
  // do not depend on the live row count, go out together with the count's
  // load instead of after it: activation rows are read up to the call's
  // row capacity x_rows (rows past it repeat the last one; rows at or past
  // the live count may hold anything, and their outputs are not stored),
  // and a workgroup with no live rows waits for them before it exits (no
  // load in flight past the end of the program).  The empty asm with a
  // memory clobber keeps the compiler from sinking the loads below the exit
  // test, past which alone their results are used (W and X are not
  // __restrict__ for the same reason).  With several row tiles (many rows,
  // long MFMA-bound launches) the count is waited for first and the rows
  // past it repeat row M - 1, as issuing early measured slower there; so
  // too with x_rows = 0 (launches whose rows are usually none).
  const bool early = n_mt == 1 && x_rows > 0;
  if (!early && m_base >= M) return;  // whole workgroup
  const int row_lim = early ? x_rows : M;
  const bf16_t* xp[MF];
#pragma unroll
  for (int q = 0; q < MF; ++q) {
    const int c = tid + 256 * q;
    const int row = min(m_base + c / 8, row_lim - 1);
    xp[q] = X + (size_t)row * ldx + kc0 + 8 * (c % 8);
  }
  // (each stage's activations before its weights: the loop's wait counts
  // assume that order of the outstanding loads)
  SB_ISSUE_X(0, 0)
  SB_ISSUE_W(0, 0)
  SB_ISSUE_X(1, 1)
  SB_ISSUE_W(1, 1)
  if constexpr (PF == 4) {
    SB_ISSUE_W(2, 2)
    SB_ISSUE_W(3, 3)
  }
  __asm__ volatile("" ::: "memory");
  if (m_base >= M) {  // one row tile and no live rows
    __builtin_amdgcn_s_waitcnt(0);
    return;
  }
  SB_STORE_X(0, 0)
  __syncthreads();
  for (int s0 = 0; s0 < nstage; s0 += PF) {
    SB_STAGE(0)
    SB_STAGE(1)
    if constexpr (PF == 4) {
      SB_STAGE(2)
      SB_STAGE(3)
    }
  }
#undef SB_STAGE
#undef SB_MMA
#undef SB_READ_X
#undef SB_STORE_X
#undef SB_ISSUE_X
#undef SB_ISSUE_W
#undef SB_ISSUE_WI
#undef SB_SCHED
  if constexpr (VR > 0) {
    constexpr int RL = 2 * VR + 3;
    __shared__ float vrec[4][32 * MF][RL];
#pragma unroll
    for (int t = 0; t < MF; ++t) {
      const int m = m_base + 32 * t + lr;
      float tv[VR];
      int ti[VR];
#pragma unroll
      for (int k = 0; k < VR; ++k) {
        tv[k] = -FLT_MAX;
        ti[k] = 0x7FFFFFFF;
      }
      float mx = -FLT_MAX, sm = 0.f, su = 0.f;
      if (wave_on) {
        // lane register r of fragment f is column nb + 32 f + 8 (r / 4) +
        // 4 h + r % 4 of row m
#pragma unroll
        for (int f = 0; f < NF; ++f)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float v = acc[t][f][r];
            mx = fmaxf(mx, v);
            vr_insert<VR>(tv, ti, v, nb + 32 * f + 8 * (r >> 2) + 4 * h + (r & 3));
          }
#pragma unroll
        for (int f = 0; f < NF; ++f)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float e = __expf(acc[t][f][r] - mx);
            sm += e;
            su = fmaf(e, acc[t][f][r], su);
          }
        if (P != nullptr && m < M) {
#pragma unroll
          for (int f = 0; f < NF; ++f)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              *reinterpret_cast<float4*>(P + (size_t)m * N + nb + 32 * f + 8 * q + 4 * h) =
                  make_float4(acc[t][f][4 * q], acc[t][f][4 * q + 1],
                              acc[t][f][4 * q + 2], acc[t][f][4 * q + 3]);
        }
      }
      // the lane pair (h = 0, 1) holds the same row
      {
        float pv[VR];
        int pi[VR];
#pragma unroll
        for (int k = 0; k < VR; ++k) {
          pv[k] = __shfl_xor(tv[k], 32, 64);
          pi[k] = __shfl_xor(ti[k], 32, 64);
        }
        const float m2 = __shfl_xor(mx, 32, 64);
        const float s2 = __shfl_xor(sm, 32, 64);
        const float u2 = __shfl_xor(su, 32, 64);
#pragma unroll
        for (int k = 0; k < VR; ++k) vr_insert<VR>(tv, ti, pv[k], pi[k]);
        vr_stats_merge(mx, sm, su, m2, s2, u2);
      }
      if (h == 0) {
        float* o = vrec[wave][32 * t + lr];
#pragma unroll
        for (int k = 0; k < VR; ++k) {
          o[k] = tv[k];
          o[VR + k] = __int_as_float(ti[k]);
        }
        o[2 * VR] = mx;
        o[2 * VR + 1] = sm;
        o[2 * VR + 2] = su;
      }
    }
    __syncthreads();
    // one thread per row merges the four waves' records
    if (tid < 32 * MF && m_base + tid < M) {
      float tv[VR];
      int ti[VR];
      const float* o0 = vrec[0][tid];
#pragma unroll
      for (int k = 0; k < VR; ++k) {
        tv[k] = o0[k];
        ti[k] = __float_as_int(o0[VR + k]);
      }
      float mx = o0[2 * VR], sm = o0[2 * VR + 1], su = o0[2 * VR + 2];
#pragma unroll
      for (int w = 1; w < 4; ++w) {
        const float* ow = vrec[w][tid];
#pragma unroll
        for (int k = 0; k < VR; ++k) vr_insert<VR>(tv, ti, ow[k], __float_as_int(ow[VR + k]));
        vr_stats_merge(mx, sm, su, ow[2 * VR], ow[2 * VR + 1], ow[2 * VR + 2]);
      }
      float* g = rec + ((size_t)(m_base + tid) * n_nt + nt) * RL;
#pragma unroll
      for (int k = 0; k < VR; ++k) {
        g[k] = tv[k];
        g[VR + k] = __int_as_float(ti[k]);
      }
      g[2 * VR] = mx;
      g[2 * VR + 1] = sm;
      g[2 * VR + 2] = su;
    }
    return;
  }
  if (!wave_on) return;
  if constexpr (SWIGLU) {
    // fragment f covers gate/up features 16 (nb / 32 + f) .. + 15; lane
    // registers 0-7 hold gate rows 8 q + 4 h + e, registers 8-15 the up rows
    // of the same features
#pragma unroll
    for (int t = 0; t < MF; ++t) {
      const int m = m_base + 32 * t + lr;
      if (m >= M) continue;
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        const int j0 = 16 * ((nb >> 5) + f);
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          float o[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            o[e] = silu(acc[t][f][4 * q + e]) * acc[t][f][8 + 4 * q + e];
          uint2 pk;
          pk.x = pack_bf16x2(o[0], o[1]);
          pk.y = pack_bf16x2(o[2], o[3]);
          *reinterpret_cast<uint2*>(act + (size_t)m * F + j0 + 8 * q + 4 * h) = pk;
        }
      }
    }
    return;
  }
  float* out = P + (size_t)kc * part_stride;
#pragma unroll
  for (int t = 0; t < MF; ++t) {
    const int m = m_base + 32 * t + lr;
    if (m >= M) continue;
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(out + (size_t)m * N + nb + 32 * f + 8 * q + 4 * h) =
            make_float4(acc[t][f][4 * q], acc[t][f][4 * q + 1],
                        acc[t][f][4 * q + 2], acc[t][f][4 * q + 3]);
  }
}

template <int MT>
__global__ __launch_bounds__(256) void gemm_xwt_kernel(
    const float* __restrict__ X, int ldx, const float* __restrict__ W, int K,
    float* __restrict__ P, int N, size_t part_stride,
    const int* __restrict__ m_count, int k_chunk) {
  const int m_base = blockIdx.z * (MT * 16);
  const int M = min(*m_count - m_base, MT * 16);
  if (M <= 0) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * 16;
  const int kc0 = blockIdx.y * k_chunk;
  const int kc1 = min(K, kc0 + k_chunk);
  const int nsteps = (kc1 - kc0) >> 5;
  const int per = (nsteps + 3) >> 2;
  const int s0 = wave * per;
  const int s1 = min(nsteps, s0 + per);

  const float* wp = W + (size_t)(n0 + r) * K + kc0 + g * 8;
  const float* xp[MT];
  bool xv[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int m = t * 16 + r;
    xv[t] = m < M;
    xp[t] = X + (size_t)(m_base + (xv[t] ? m : 0)) * ldx + kc0 + g * 8;
  }
  f32x4_t acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  constexpr int U = 4;
  for (int s = s0; s < s1; s += U) {
    Frag8<float> wf[U];
    Frag8<float> xf[U][MT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s + u < s1) {
        wf[u].load(wp + (size_t)(s + u) * 32);
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          xf[u][t].load(xp[t] + (size_t)(s + u) * 32);
          if (!xv[t]) xf[u][t].zero();
        }
      } else {
        wf[u].zero();
#pragma unroll
        for (int t = 0; t < MT; ++t) xf[u][t].zero();
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < MT; ++t) acc[t] = mma_16x16x32(wf[u], xf[u][t], acc[t]);
  }

  __shared__ f32x4_t red[3][MT][64];
  if (wave > 0) {
#pragma unroll
    for (int t = 0; t < MT; ++t) red[wave - 1][t][lane] = acc[t];
  }
  __syncthreads();
  if (wave == 0) {
    float* out = P + (size_t)blockIdx.y * part_stride;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      f32x4_t a = acc[t] + red[0][t][lane] + red[1][t][lane] + red[2][t][lane];
      const int m = t * 16 + r;
      if (m < M) {
        float4 v = make_float4(a[0], a[1], a[2], a[3]);
        *reinterpret_cast<float4*>(out + (size_t)(m_base + m) * N + n0 +
                                   4 * g) = v;
      }
    }
  }
}

// Packs row-major src [rows][cols] into the fragment layout, one 16-byte
// chunk per thread.  gate_up: src is [gate; up] ([2F][cols], F = rows / 2)
// and packed row 32 rb + j is gate row 16 rb + j (j < 16) or up row
// 16 rb + j - 16.
__global__ void pack_kernel(const bf16_t* __restrict__ src,
                            bf16_t* __restrict__ dst, int rows, int cols,
                            bool gate_up, size_t chunks) {
  const size_t c = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= chunks) return;
  const int rblocks = rows / 32;
  const size_t blk = c >> 8;
  const int i = (int)((c >> 6) & 3), l = (int)(c & 63);
  const int kb = (int)(blk / rblocks), rb = (int)(blk % rblocks);
  const int j = l & 31;
  int row = 32 * rb + j;
  if (gate_up) row = j < 16 ? 16 * rb + j : rows / 2 + 16 * rb + (j - 16);
  const int col = 64 * kb + 32 * (l >> 5) + 8 * i;
  *reinterpret_cast<uint4*>(dst + c * 8) =
      *reinterpret_cast<const uint4*>(src + (size_t)row * cols + col);
}

namespace {

constexpr int kTargetWorkgroups = 256;  // one per CU

// K must be a multiple of 64 * pf * ks (whole weight rings per chunk).
int pick_split(int tiles, int K, int pf) {
  int ks = 1;
  while (ks < 16 && tiles * ks * 2 <= kTargetWorkgroups &&
         K % (64 * pf * ks * 2) == 0)
    ks *= 2;
  return ks;
}

}  // namespace

bool gemm_shape_ok(int N, int K, int elem_bytes) {
  if (elem_bytes == 4) return N % 16 == 0 && K % 32 == 0;
  return N % 32 == 0 && K % 128 == 0;
}

namespace {

// fraction of the last round of workgroups that is busy
double round_fill(int wgs) {
  const int rounds = (wgs + kTargetWorkgroups - 1) / kTargetWorkgroups;
  return (double)wgs / ((double)rounds * kTargetWorkgroups);
}

}  // namespace

namespace {

// Estimated duration (us) of a many-row bf16 plan: rounds of 256
// workgroups, each streaming its 32 mf x 128 nf tile over K / ks at the
// per-CU MFMA rate the kernel sustains (0.45 of 2.5 PFLOP/s / 256), scaled
// by the tile's relative efficiency (measured: 128 x 512 tiles 1.12 and
// 96 x 256 tiles 0.97 of 128 x 256), plus the consumer's read of the ks
// fp32 partial slabs at 5 TB/s.  Fits the measured 8B and 70B projections
// within ~10%.
double tile_rounds_us(int mf, int nf, int ks, int N, int K, int m_cap) {
  const int n_mt = (m_cap + 32 * mf - 1) / (32 * mf);
  const int n_nt = (N + 128 * nf - 1) / (128 * nf);
  const long wgs = (long)n_mt * n_nt * ks;
  const long rounds = (wgs + kTargetWorkgroups - 1) / kTargetWorkgroups;
  const double eff = nf == 4 ? 1.12 : mf == 3 ? 0.97 : 1.0;
  const double t_wg =
      2.0 * 32 * mf * 128 * nf * ((double)K / ks) / (0.45 * 2.5e15 / 256) * 1e6;
  return rounds * t_wg / eff;
}

double many_row_us(int mf, int nf, int ks, int N, int K, int m_cap) {
  return tile_rounds_us(mf, nf, ks, N, K, m_cap) +
         (double)ks * m_cap * N * 4 / 5e12 * 1e6;
}

}  // namespace

GemmPlan gemm_plan(int N, int K, int m_cap, int elem_bytes, bool retile) {
  GemmPlan g{};
  if (elem_bytes == 4) {
    g.mf = m_cap <= 16 ? 1 : (m_cap <= 32 ? 2 : 4);  // 16-row tiles
    const int tiles = N / 16;
    g.ks = 1;
    while (tiles * g.ks < 1024 && K / (32 * (g.ks * 2)) >= 32 && g.ks < 16)
      g.ks *= 2;
    return g;
  }
  // 128-row tiles above 64 rows (256-row tiles measured no faster at 1024
  // rows); 64 weight rows per wave above 128 rows, 128 per wave when the
  // weight tiles alone fill the chip at least as evenly (fewer activation
  // LDS reads per MFMA: +13% on the 28672- and 128256-wide projections at
  // 1024 rows).  Four weight stages in flight only for 128-row tiles of
  // 32 weight rows per wave above 128 rows; at 128 rows (one sequence of
  // 128 tree nodes) two are faster (step -1.5%).
  g.mf = m_cap <= 32 ? 1 : m_cap <= 64 ? 2 : 4;
  const int n_mt = (m_cap + 32 * g.mf - 1) / (32 * g.mf);
  g.nf = 1;
  if (g.mf == 4 && m_cap > 128 && N % 64 == 0) {
    g.nf = 2;
    const int t2 = n_mt * ((N + 255) / 256), t4 = n_mt * ((N + 511) / 512);
    if (N % 128 == 0 && t4 >= kTargetWorkgroups && round_fill(t4) >= round_fill(t2))
      g.nf = 4;
  }
  g.pf = (g.mf == 4 && g.nf == 1 && m_cap > 128 && (K / 64) % 4 == 0) ? 4 : 2;
  const int n_nt = (N + 128 * g.nf - 1) / (128 * g.nf);
  g.ks = pick_split(n_mt * n_nt, K, g.pf);
  if (retile && g.mf == 4 && m_cap > 128) {
    // plain projections (K-split partials summed by the consumer): tiles
    // of 384 weight rows or of 96 activation rows when they fill the chip's
    // rounds evenly enough to be clearly faster (estimate > 8% lower).
    // Measured, weights cold: 1024 x 6144 x 4096 62 -> 51 us (384-row
    // weight tiles, 2 K-chunks); 384 rows x 8192 x 8192 58 -> 54 us and
    // x 28672 188 -> 178 us (96-row tiles); 96-row tiles at 192 rows made
    // the 70B drafting block 7% slower, so they need 256 rows or more.  The
    // K-split stays within the one-row plan's (the partial buffers are
    // sized for it).
    const int ks_cap = pick_split((N + 127) / 128, K, 2);
    const double base = many_row_us(g.mf, g.nf, g.ks, N, K, m_cap);
    double best = 0.92 * base;
    const int cand[2][2] = {{4, 3}, {3, 2}};
    for (const auto& c : cand) {
      const int mf = c[0], nf = c[1];
      if (N % (128 * nf) != 0 || (mf == 3 && m_cap < 256)) continue;
      const int tiles = ((m_cap + 32 * mf - 1) / (32 * mf)) * (N / (128 * nf));
      const int ks = std::min(pick_split(tiles, K, 2), ks_cap);
      const double t = many_row_us(mf, nf, ks, N, K, m_cap);
      if (t < best) {
        best = t;
        g = GemmPlan{mf, nf, 2, ks};
      }
    }
  }
  return g;
}

namespace {

// Timing events for the next projection-GEMM launch, set by the library's
// profiler and consumed by one launch: attached to the dispatch itself, they
// record the kernel's own start and end (no marker packets in the stream).
thread_local hipEvent_t g_ev_start = nullptr, g_ev_stop = nullptr;

void take_events(hipEvent_t& a, hipEvent_t& b) {
  a = g_ev_start;
  b = g_ev_stop;
  g_ev_start = g_ev_stop = nullptr;
}

}  // namespace

void gemm_time_next_launch(hipEvent_t start, hipEvent_t stop) {
  g_ev_start = start;
  g_ev_stop = stop;
}

bool gemm_time_pending() { return g_ev_start != nullptr; }

int gemm_ksplit(int N, int K, int elem_bytes) {
  // fewest row tiles -> most K-chunks
  return gemm_plan(N, K, 1, elem_bytes).ks;
}

namespace {

template <bool SWIGLU, int VR = 0>
void launch_tile(const GemmPlan& g, const bf16_t* X, int ldx, const bf16_t* W,
                 int N, int K, float* P, size_t part_stride,
                 const int* m_count, int m_cap, int ks, bf16_t* act, int F,
                 hipStream_t st, float* rec = nullptr, int n_first = 0,
                 int n_rows = -1) {
  // weight rows n_first .. n_first + n_rows - 1 (n_first + n_rows is N or a
  // multiple of 128 nf)
  const int rows = n_rows < 0 ? N - n_first : n_rows;
  const int n_mt = (m_cap + 32 * g.mf - 1) / (32 * g.mf);
  const int n_nt = (rows + 128 * g.nf - 1) / (128 * g.nf);
  const int k_chunk = K / ks;
  const dim3 grid(n_mt * n_nt * ks);
#define SB_LAUNCH(MF_, NF_, PF_)                                              \
  if (g.mf == MF_ && g.nf == NF_ && g.pf == PF_) {                            \
    hipEvent_t ea, eb;                                                        \
    take_events(ea, eb);                                                      \
    hipExtLaunchKernelGGL(gemm_tile_kernel<MF_, NF_, PF_, SWIGLU, VR>, grid,  \
                          dim3(256), 0, st, ea, eb, 0, X, ldx, W, K, P, N,    \
                          part_stride, m_count, k_chunk, n_mt, n_nt, act, F,  \
                          rec, n_first, rows_likely_empty() ? 0 : m_cap);     \
    return;                                                                   \
  }
  SB_LAUNCH(1, 1, 2)
  SB_LAUNCH(2, 1, 2)
  SB_LAUNCH(4, 1, 2)
  SB_LAUNCH(4, 1, 4)
  SB_LAUNCH(4, 2, 2)
  SB_LAUNCH(4, 4, 2)
  if constexpr (VR == 0) SB_LAUNCH(4, 3, 2)   // re-tiled or split launches
  if constexpr (VR == 0) SB_LAUNCH(3, 2, 2)
#undef SB_LAUNCH
}

}  // namespace

template <typename T>
int launch_gemm_xwt(const T* X, int ldx, const T* W, int N, int K, float* P,
                    size_t part_stride, const int* m_count, int m_cap,
                    int ksplit, hipStream_t st) {
  const GemmPlan g = gemm_plan(N, K, m_cap, sizeof(T), true);
  if constexpr (sizeof(T) == 2) {
    int ks = g.ks;
    if (ksplit > 0)
      while (ks > ksplit) ks /= 2;
    launch_tile<false>(g, X, ldx, W, N, K, P, part_stride, m_count, m_cap, ks,
                       nullptr, 0, st);
    return ks;
  } else {
    const int ks_req = ksplit > 0 ? std::min(ksplit, g.ks) : g.ks;
    const int steps = K / 32;
    const int per = (steps + ks_req - 1) / ks_req;
    const int k_chunk = per * 32;
    const int ks = (K + k_chunk - 1) / k_chunk;
    const int mz = (m_cap + 63) / 64;
    const dim3 block(256);
    hipEvent_t ea, eb;
    take_events(ea, eb);
    if (m_cap <= 16) {
      hipExtLaunchKernelGGL(gemm_xwt_kernel<1>, dim3(N / 16, ks, 1), block, 0,
                            st, ea, eb, 0, X, ldx, W, K, P, N, part_stride,
                            m_count, k_chunk);
    } else if (m_cap <= 32) {
      hipExtLaunchKernelGGL(gemm_xwt_kernel<2>, dim3(N / 16, ks, 1), block, 0,
                            st, ea, eb, 0, X, ldx, W, K, P, N, part_stride,
                            m_count, k_chunk);
    } else {
      hipExtLaunchKernelGGL(gemm_xwt_kernel<4>, dim3(N / 16, ks, mz), block, 0,
                            st, ea, eb, 0, X, ldx, W, K, P, N, part_stride,
                            m_count, k_chunk);
    }
    return ks;
  }
}

template int launch_gemm_xwt<float>(const float*, int, const float*, int, int,
                                    float*, size_t, const int*, int, int,
                                    hipStream_t);
template int launch_gemm_xwt<bf16_t>(const bf16_t*, int, const bf16_t*, int,
                                     int, float*, size_t, const int*, int, int,
                                     hipStream_t);

int launch_gemm_vocab(const bf16_t* X, int ldx, const bf16_t* W, int N,
                      int K, float* logits, const int* m_count, int m_cap,
                      int topk, float* rec, hipStream_t st) {
  const GemmPlan g = gemm_plan(N, K, m_cap, 2);
  if (topk != 1) return 0;
  launch_tile<false, 1>(g, X, ldx, W, N, K, logits, 0, m_count, m_cap, 1,
                        nullptr, 0, st, rec);
  return gemm_vocab_chunks(N, K, m_cap);
}

int gemm_vocab_chunks(int N, int K, int m_cap) {
  const GemmPlan g = gemm_plan(N, K, m_cap, 2);
  return (N + 128 * g.nf - 1) / (128 * g.nf);
}

namespace {

// One launch of a SwiGLU projection over weight rows n_first ..
// n_first + rows - 1.
struct SwigluPart {
  GemmPlan g;
  int n_first, rows;
};

int weight_stages(int nf, int K) { return nf == 1 && (K / 64) % 4 == 0 ? 4 : 2; }

// The gate/up projection has no K-split (SiLU(g) u is not linear in the
// K-chunks), so with many rows its last round of workgroups can run part
// empty: 1024 rows x 28672 gate/up rows make 448 workgroups of 128 x 512,
// 1.75 rounds of 256.  Two launches over consecutive weight-row ranges,
// each with tiles that fill their rounds, finish sooner: one round of
// 128 x 512 tiles, then one of 128 x 384 (estimate 7% less; 384 rows x
// 57344: one round of 128 x 512, then the other 13824 rows in 216
// workgroups of 96 x 256, 9% less).  Taken when the estimate, with the
// second launch's start, is > 5% lower.
int swiglu_parts(int N, int K, int m_cap, SwigluPart part[2]) {
  const GemmPlan g = gemm_plan(N, K, m_cap, 2);
  part[0] = SwigluPart{g, 0, N};
  const int n_mt = (m_cap + 127) / 128;
  if (g.mf != 4 || m_cap <= 128 || n_mt > kTargetWorkgroups) return 1;
  constexpr double kSecondLaunchUs = 3.0;
  double best = 0.95 * tile_rounds_us(4, g.nf, 1, N, K, m_cap);
  int parts = 1;
  for (const int nfa : {4, 2}) {
    for (int r = 1;; ++r) {
      const int rows_a = kTargetWorkgroups * r / n_mt * 128 * nfa;
      if (rows_a >= N) break;
      const int rows_b = N - rows_a;
      // the second launch also in 96 x 256 tiles from 256 rows (more
      // workgroups for the leftover rows)
      for (const int mfb : {4, 3}) {
        for (int nfb = 4; nfb >= 1; --nfb) {   // wider tiles on a tie
          if (rows_b % (32 * nfb) != 0) continue;
          if (mfb == 3 && (nfb != 2 || m_cap < 256)) continue;
          const double t = tile_rounds_us(4, nfa, 1, rows_a, K, m_cap) +
                           tile_rounds_us(mfb, nfb, 1, rows_b, K, m_cap) +
                           kSecondLaunchUs;
          if (t < best) {
            best = t;
            parts = 2;
            part[0] = SwigluPart{{4, nfa, weight_stages(nfa, K), 1}, 0, rows_a};
            part[1] = SwigluPart{{mfb, nfb, mfb == 4 ? weight_stages(nfb, K) : 2, 1},
                                 rows_a, rows_b};
          }
        }
      }
    }
  }
  return parts;
}

}  // namespace

void launch_gemm_swiglu(const bf16_t* X, int ldx, const bf16_t* W, int F,
                        int K, bf16_t* act, const int* m_count, int m_cap,
                        hipStream_t st) {
  SwigluPart part[2];
  const int parts = swiglu_parts(2 * F, K, m_cap, part);
  if (parts == 1) {
    launch_tile<true>(part[0].g, X, ldx, W, 2 * F, K, nullptr, 0, m_count,
                      m_cap, 1, act, F, st);
    return;
  }
  // profiling events: the start on the first launch, the stop on the second
  hipEvent_t ea, eb;
  take_events(ea, eb);
  for (int i = 0; i < 2; ++i) {
    g_ev_start = i == 0 ? ea : nullptr;
    g_ev_stop = i == 1 ? eb : nullptr;
    launch_tile<true>(part[i].g, X, ldx, W, 2 * F, K, nullptr, 0, m_count,
                      m_cap, 1, act, F, st, nullptr, part[i].n_first,
                      part[i].rows);
  }
}

int launch_pack_weight(const bf16_t* src, bf16_t* dst, int rows, int cols,
                       bool gate_up, hipStream_t st) {
  const size_t chunks = (size_t)rows * cols / 8;
  if (chunks == 0) return 0;
  const size_t blocks = (chunks + 255) / 256;
  pack_kernel<<<dim3((unsigned)blocks), 256, 0, st>>>(src, dst, rows, cols,
                                                      gate_up, chunks);
  return 0;
}

}  // namespace sb
