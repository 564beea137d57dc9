// Weight-streaming projection GEMM on MFMA (gfx950).
//
//   P[ks][m][n] = sum_{k in K-chunk ks} X[m][k] * W[n][k]
//
// X holds the few activation rows of a call (<= 64 per m-chunk), W is a
// row-major [N][K] weight matrix streamed from HBM once per m-chunk.  MFMA
// 16x16x32 with weight rows as the A operand (16 features x 32 k) and
// activation rows as the B operand, so a lane's four results are four
// consecutive features of one row (one 16-byte store).  K-chunks
// (gridDim.y) write separate partial sums that the consumer kernel adds,
// which keeps results independent of scheduling order.
//
// bf16 path (gemm_stream_kernel): a workgroup of NW waves owns 16 NW
// features and one K-chunk.  Each wave streams its own 16 weight rows with
// row-contiguous 16-byte loads (a wave instruction covers 1 KiB of whole row
// segments, so every HBM line is used by one instruction), one K-stage ahead
// in registers, and transposes them into MFMA order through a wave-private
// LDS tile.  The workgroup stages the activation K-slice in LDS once
// (double buffered) and all its waves read it from there, so activation
// traffic does not grow with the number of weight rows.  fp32 path
// (gemm_xwt_kernel): weight fragments load straight into registers.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace sb {


__device__ __forceinline__ uint4 load_stream16(const void* p) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// SWIGLU: the weight is [gate; up] ([2F][K]) and the workgroup owns gate
// features j0 .. j0 + 8 NW - 1 (first NW/2 waves) and the matching up
// features (last NW/2 waves); with one K-chunk the epilogue writes
// act[m][j] = silu(gate) * up as bf16 instead of partial sums.
template <int MT, int NW, int KT, bool SWIGLU>
__global__ __launch_bounds__(NW * 64) void gemm_stream_kernel(
    const bf16_t* __restrict__ X, int ldx, const bf16_t* __restrict__ W,
    int K, float* __restrict__ P, int N, size_t part_stride,
    const int* __restrict__ m_count, int k_chunk, bf16_t* __restrict__ act,
    int F) {
  constexpr int LD = KT + 8;                        // padded LDS row
  constexpr int RPI = 1024 / (KT * 2);              // rows per wave load
  constexpr int NI = 16 / RPI;                      // loads per stage
  constexpr int XCH = MT * 16 * KT / 8;             // 16-byte X chunks
  constexpr int XPT = (XCH + NW * 64 - 1) / (NW * 64);
  __shared__ __attribute__((aligned(16))) bf16_t wl[NW][16][LD];
  __shared__ __attribute__((aligned(16))) bf16_t xs[2][MT * 16][LD];
  const int m_base = blockIdx.z * (MT * 16);
  const int M = min(*m_count - m_base, MT * 16);
  if (M <= 0) return;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int r = lane & 15, g = lane >> 4;
  int n0 = blockIdx.x * 16 * NW + wave * 16;
  if constexpr (SWIGLU) {
    constexpr int HW = NW / 2;
    n0 = blockIdx.x * 16 * HW + (wave % HW) * 16 + (wave >= HW ? F : 0);
  }
  const int kc0 = blockIdx.y * k_chunk;
  const int kc1 = min(K, kc0 + k_chunk);
  const int nstage = (kc1 - kc0) / KT;
  const int lrow = lane / (KT / 8), lcol = (lane % (KT / 8)) * 8;
  const bf16_t* wsrc = W + (size_t)(n0 + lrow) * K + kc0 + lcol;
  const bf16_t* xbase = X + (size_t)m_base * ldx + kc0;
  f32x4_t acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  uint4 stg[NI];
  uint4 xr[XPT];
#pragma unroll
  for (int i = 0; i < NI; ++i) stg[i] = load_stream16(wsrc + (size_t)(i * RPI) * K);
  auto xfetch = [&](int st) {
#pragma unroll
    for (int q = 0; q < XPT; ++q) {
      const int c = tid + q * NW * 64;
      const int row = c / (KT / 8), col = (c % (KT / 8)) * 8;
      xr[q] = (c < XCH && row < M)
                  ? *reinterpret_cast<const uint4*>(xbase + (size_t)row * ldx +
                                                    st * KT + col)
                  : make_uint4(0, 0, 0, 0);
    }
  };
  auto xstore = [&](int buf) {
#pragma unroll
    for (int q = 0; q < XPT; ++q) {
      const int c = tid + q * NW * 64;
      const int row = c / (KT / 8), col = (c % (KT / 8)) * 8;
      if (c < XCH) *reinterpret_cast<uint4*>(&xs[buf][row][col]) = xr[q];
    }
  };
  xfetch(0);
  xstore(0);
  __syncthreads();
  for (int st = 0; st < nstage; ++st) {
    const int buf = st & 1;
    // this stage's weight rows into the wave's LDS tile, next stage's loads
    // in flight during the MFMAs
#pragma unroll
    for (int i = 0; i < NI; ++i)
      *reinterpret_cast<uint4*>(&wl[wave][i * RPI + lrow][lcol]) = stg[i];
    if (st + 1 < nstage) {
#pragma unroll
      for (int i = 0; i < NI; ++i)
        stg[i] = load_stream16(wsrc + (size_t)(i * RPI) * K + (size_t)(st + 1) * KT);
      xfetch(st + 1);
    }
#pragma unroll
    for (int j = 0; j < KT / 32; ++j) {
      Frag8<bf16_t> wf;
      wf.v = *reinterpret_cast<const uint4*>(&wl[wave][r][j * 32 + g * 8]);
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        Frag8<bf16_t> xf;
        xf.v = *reinterpret_cast<const uint4*>(&xs[buf][t * 16 + r][j * 32 + g * 8]);
        acc[t] = mma_16x16x32(wf, xf, acc[t]);
      }
    }
    if (st + 1 < nstage) xstore(buf ^ 1);
    __syncthreads();
  }
  if constexpr (SWIGLU) {
    // up waves hand their sums to the gate waves through LDS (the loop
    // ended with a barrier, so the X tiles are free)
    constexpr int HW = NW / 2;
    f32x4_t* ex = reinterpret_cast<f32x4_t*>(&xs[0][0][0]);
    static_assert(sizeof(xs) >= HW * MT * 64 * sizeof(f32x4_t), "LDS");
    if (wave >= HW) {
#pragma unroll
      for (int t = 0; t < MT; ++t) ex[((wave - HW) * MT + t) * 64 + lane] = acc[t];
    }
    __syncthreads();
    if (wave < HW) {
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const int m = t * 16 + r;
        const f32x4_t u = ex[(wave * MT + t) * 64 + lane];
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float gt = acc[t][e];
          o[e] = gt / (1.0f + expf(-gt)) * u[e];
        }
        if (m < M) {
          uint2 pk;
          pk.x = (uint32_t)f32_to_bf16(o[0]) | ((uint32_t)f32_to_bf16(o[1]) << 16);
          pk.y = (uint32_t)f32_to_bf16(o[2]) | ((uint32_t)f32_to_bf16(o[3]) << 16);
          *reinterpret_cast<uint2*>(act + (size_t)(m_base + m) * F + n0 + 4 * g) = pk;
        }
      }
    }
    return;
  }
  float* out = P + (size_t)blockIdx.y * part_stride;
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int m = t * 16 + r;
    if (m < M)
      *reinterpret_cast<float4*>(out + (size_t)(m_base + m) * N + n0 + 4 * g) =
          make_float4(acc[t][0], acc[t][1], acc[t][2], acc[t][3]);
  }
}

template <typename T, int MT>
__global__ __launch_bounds__(256) void gemm_xwt_kernel(
    const T* __restrict__ X, int ldx, const T* __restrict__ W, int K,
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

  const T* wp = W + (size_t)(n0 + r) * K + kc0 + g * 8;
  const T* xp[MT];
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
    Frag8<T> wf[U];
    Frag8<T> xf[U][MT];
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

GemmPlan gemm_plan(int N, int K, int m_cap, int elem_bytes) {
  GemmPlan g{};
  g.mt = m_cap <= 16 ? 1 : (m_cap <= 32 ? 2 : 4);
  if (elem_bytes == 2 && N % 64 == 0 && K % 128 == 0) {
    g.stream = true;
    g.kt = (g.mt == 4 || K % 256 != 0) ? 128 : 256;
    g.nw = (g.mt == 4 && N >= 65536 && N % 128 == 0) ? 8 : 4;
    const int tiles = N / (16 * g.nw);
    g.ks = 1;
    // enough workgroups to fill the chip; each K-chunk a whole number of
    // stages and at least four of them
    while (tiles * g.ks < 400 && g.ks < 16 && K % (g.ks * 2 * g.kt) == 0 &&
           K / (g.ks * 2) >= 4 * g.kt)
      g.ks *= 2;
  } else {
    g.stream = false;
    const int tiles = N / 16;
    g.ks = 1;
    while (tiles * g.ks < 1024 && K / (32 * (g.ks * 2)) >= 32 && g.ks < 16)
      g.ks *= 2;
  }
  return g;
}

int gemm_ksplit(int N, int K, int ksplit_cap) {
  (void)ksplit_cap;
  int mx = 1;
  for (int mc : {16, 32, 64}) {
    mx = std::max(mx, gemm_plan(N, K, mc, 2).ks);
    mx = std::max(mx, gemm_plan(N, K, mc, 4).ks);
  }
  return mx;
}

template <typename T>
int launch_gemm_xwt(const T* X, int ldx, const T* W, int N, int K, float* P,
                    size_t part_stride, const int* m_count, int m_cap,
                    int ksplit, hipStream_t st) {
  const GemmPlan g = gemm_plan(N, K, m_cap, sizeof(T));
  const int ks_req = ksplit > 0 ? std::min(ksplit, g.ks) : g.ks;
  const int mz = (m_cap + 63) / 64;
  if constexpr (sizeof(T) == 2) {
    if (g.stream) {
      const int ks = ks_req;
      const int k_chunk = K / ks;
      const dim3 grid(N / (16 * g.nw), ks, g.mt == 4 ? mz : 1);
#define SB_LAUNCH(MT_, NW_, KT_)                                              \
  if (g.mt == MT_ && g.nw == NW_ && g.kt == KT_) {                            \
    gemm_stream_kernel<MT_, NW_, KT_, false><<<grid, NW_ * 64, 0, st>>>(      \
        X, ldx, W, K, P, N, part_stride, m_count, k_chunk, nullptr, 0);       \
    return ks;                                                                \
  }
      SB_LAUNCH(1, 4, 256)
      SB_LAUNCH(1, 4, 128)
      SB_LAUNCH(2, 4, 256)
      SB_LAUNCH(2, 4, 128)
      SB_LAUNCH(4, 4, 128)
      SB_LAUNCH(4, 8, 128)
#undef SB_LAUNCH
    }
  }
  const int steps = K / 32;
  const int per = (steps + ks_req - 1) / ks_req;
  const int k_chunk = per * 32;
  const int ks = (K + k_chunk - 1) / k_chunk;
  dim3 block(256);
  if (m_cap <= 16) {
    dim3 grid(N / 16, ks, 1);
    gemm_xwt_kernel<T, 1><<<grid, block, 0, st>>>(X, ldx, W, K, P, N,
                                                  part_stride, m_count, k_chunk);
  } else if (m_cap <= 32) {
    dim3 grid(N / 16, ks, 1);
    gemm_xwt_kernel<T, 2><<<grid, block, 0, st>>>(X, ldx, W, K, P, N,
                                                  part_stride, m_count, k_chunk);
  } else {
    dim3 grid(N / 16, ks, mz);
    gemm_xwt_kernel<T, 4><<<grid, block, 0, st>>>(X, ldx, W, K, P, N,
                                                  part_stride, m_count, k_chunk);
  }
  return ks;
}

bool gemm_swiglu_fits(int F, int K, int m_cap) {
  const GemmPlan g = gemm_plan(2 * F, K, m_cap, 2);
  return g.stream && g.ks == 1 && F % (8 * g.nw) == 0;
}

bool launch_gemm_swiglu(const bf16_t* X, int ldx, const bf16_t* W, int F,
                        int K, bf16_t* act, const int* m_count, int m_cap,
                        hipStream_t st) {
  if (!gemm_swiglu_fits(F, K, m_cap)) return false;
  const GemmPlan g = gemm_plan(2 * F, K, m_cap, 2);
  const int mz = (m_cap + 63) / 64;
  const dim3 grid(F / (8 * g.nw), 1, g.mt == 4 ? mz : 1);
#define SB_LAUNCH_SW(MT_, NW_, KT_)                                           \
  if (g.mt == MT_ && g.nw == NW_ && g.kt == KT_) {                            \
    gemm_stream_kernel<MT_, NW_, KT_, true><<<grid, NW_ * 64, 0, st>>>(       \
        X, ldx, W, K, nullptr, 2 * F, 0, m_count, K, act, F);                 \
    return true;                                                              \
  }
  SB_LAUNCH_SW(1, 4, 256)
  SB_LAUNCH_SW(1, 4, 128)
  SB_LAUNCH_SW(2, 4, 256)
  SB_LAUNCH_SW(2, 4, 128)
  SB_LAUNCH_SW(4, 4, 128)
  SB_LAUNCH_SW(4, 8, 128)
#undef SB_LAUNCH_SW
  return false;
}

template int launch_gemm_xwt<float>(const float*, int, const float*, int, int,
                                    float*, size_t, const int*, int, int,
                                    hipStream_t);
template int launch_gemm_xwt<bf16_t>(const bf16_t*, int, const bf16_t*, int,
                                     int, float*, size_t, const int*, int, int,
                                     hipStream_t);

}  // namespace sb
