// Weight-streaming projection GEMM on MFMA (gfx950).
//
//   P[ks][m][n] = sum_{k in K-chunk ks} X[m][k] * W[n][k]
//
// X holds the few activation rows of a call (M <= 64 per m-chunk), W is a
// row-major [N][K] weight matrix streamed from HBM exactly once per m-chunk.
// One workgroup (4 waves) owns 16 output features and one K-chunk; its waves
// split the chunk four ways and combine through LDS, so a weight row segment
// is read by exactly one wave with 16-byte loads.  W rows are the MFMA A
// operand (16 features x 32 k), activation rows the B operand, so a lane's
// four results are four consecutive features of one row: one 16-byte store.
// K-chunks (gridDim.y) write separate partial sums that the consumer kernel
// adds, which keeps the result independent of scheduling order.
#include "common.h"
#include "kernels.h"

namespace sb {

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

template <typename T>
int launch_gemm_xwt(const T* X, int ldx, const T* W, int N, int K, float* P,
                    size_t part_stride, const int* m_count, int m_cap,
                    int ksplit, hipStream_t st) {
  const int steps = K / 32;
  const int per = (steps + ksplit - 1) / ksplit;
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
    dim3 grid(N / 16, ks, (m_cap + 63) / 64);
    gemm_xwt_kernel<T, 4><<<grid, block, 0, st>>>(X, ldx, W, K, P, N,
                                                  part_stride, m_count, k_chunk);
  }
  return ks;
}

int gemm_ksplit(int N, int K, int ksplit_cap) {
  // Enough workgroups to cover the chip several times, K-chunks of at
  // least 1024 (each wave then streams >= 256 elements per weight row).
  const int tiles = N / 16;
  int ks = 1;
  while (tiles * ks < 1024 && K / (32 * (ks * 2)) >= 32 && ks * 2 <= ksplit_cap)
    ks *= 2;
  return ks;
}

template int launch_gemm_xwt<float>(const float*, int, const float*, int, int,
                                    float*, size_t, const int*, int, int,
                                    hipStream_t);
template int launch_gemm_xwt<bf16_t>(const bf16_t*, int, const bf16_t*, int,
                                     int, float*, size_t, const int*, int, int,
                                     hipStream_t);

}  // namespace sb
