// Head-only serving-time update of the drafter (Sec. 3.4; the per-query
// adaptation procedure of App. A.3): buffered rejected positions step the
// drafter's LM head and rank head on their cross-entropy against the
// verifier's token plus a KL penalty towards the pre-deployment head, one
// SGD step on a training copy of the weights.  The decoder trunk and the
// final norm stay frozen.  The logit statistics and gradients of each
// position are computed by adapt_row_kernel (vocab.hip); here are the
// operand preparation and the two weight updates.
#include "common.h"
#include "kernels.h"

namespace sb {

namespace {

constexpr int kStripeRows = 64;      // LM-head rows per update workgroup

}  // namespace

// a_i = RMSNorm(h_i) * g in the weights' element type (the LM head's operand
// in the drafter forward), for i < n = min(count, cap); n_eff = n.
template <typename T>
__global__ __launch_bounds__(256) void adapt_prep_kernel(
    const float* __restrict__ h, const int* __restrict__ count, int cap,
    const float* __restrict__ g, float eps, int d, T* __restrict__ A,
    int* __restrict__ n_eff) {
  __shared__ float red[4];
  const int i = blockIdx.x;
  const int n = min(*count, cap);
  if (i == 0 && threadIdx.x == 0) *n_eff = n;
  if (i >= n) return;
  const float* hr = h + (size_t)i * d;
  float ss = 0.f;
  for (int k = threadIdx.x; k < d; k += 256) ss += hr[k] * hr[k];
  ss = block_sum(ss, red);
  const float rs = 1.0f / sqrtf(ss / (float)d + eps);
  for (int k = threadIdx.x; k < d; k += 256)
    A[(size_t)i * d + k] = Elem<T>::from_f32(hr[k] * rs * g[k]);
}

// W -= lr * G^T A over a stripe of 64 LM-head rows x CW columns, with
// G [n][Vd] the (already 1/n-scaled) logit gradients and A [n][d] the
// operands, n <= 64.  bf16 weights are fragment-packed (32 x 64 blocks of
// four 1 KiB sub-steps); a thread owns 8 consecutive stored elements, which
// are 8 consecutive columns of one row in either layout.
template <typename T, int CW>
__global__ __launch_bounds__(256) void lm_update_kernel(
    T* __restrict__ W, int Vd, int d, const float* __restrict__ G,
    const T* __restrict__ A, const int* __restrict__ n_eff, float lr) {
  __shared__ float gs[64][kStripeRows];
  __shared__ float as[64][CW];
  const int n = *n_eff;
  if (n <= 0) return;
  const int r0 = blockIdx.x * kStripeRows, c0 = blockIdx.y * CW;
  for (int e = threadIdx.x; e < n * kStripeRows; e += 256) {
    const int i = e / kStripeRows, r = e % kStripeRows;
    gs[i][r] = G[(size_t)i * Vd + r0 + r];
  }
  for (int e = threadIdx.x; e < n * CW; e += 256) {
    const int i = e / CW, c = e % CW;
    as[i][c] = Elem<T>::to_f32(A[(size_t)i * d + c0 + c]);
  }
  __syncthreads();
  constexpr int kChunks = kStripeRows * CW / 8;
  for (int q = threadIdx.x; q < kChunks; q += 256) {
    int r, c;
    size_t addr;
    if constexpr (sizeof(T) == 2) {
      // stripe = 2 row blocks x CW/64 column blocks of 256 chunks each
      const int blk = q >> 8, cc = q & 255;
      const int rbi = blk / (CW / 64), kbi = blk % (CW / 64);
      const int sub = cc >> 6, l = cc & 63;
      r = 32 * rbi + (l & 31);
      c = 64 * kbi + 32 * (l >> 5) + 8 * sub;
      const int rb = (r0 >> 5) + rbi, kb = (c0 >> 6) + kbi;
      addr = ((((size_t)kb * (Vd >> 5) + rb) * 4 + sub) * 512) + (size_t)l * 8;
    } else {
      r = q / (CW / 8);
      c = 8 * (q % (CW / 8));
      addr = (size_t)(r0 + r) * d + c0 + c;
    }
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int i = 0; i < n; ++i) {
      const float gv = gs[i][r];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += gv * as[i][c + e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e)
      W[addr + e] = Elem<T>::from_f32(Elem<T>::to_f32(W[addr + e]) - lr * acc[e]);
  }
}

// Rank head: W_r[b][j] -= lr * sum_i ds[i][b] x_i[j], x_i = [h_i, psi_i];
// b_r[b] -= lr * sum_i ds[i][b]; the mean loss; the buffer is emptied.
__global__ __launch_bounds__(256) void rank_update_kernel(
    float* __restrict__ rank_w, float* __restrict__ rank_b,
    const float* __restrict__ ds, const float* __restrict__ h,
    const float* __restrict__ psi, int d, const int* __restrict__ n_eff,
    float lr, const float* __restrict__ loss, float* __restrict__ loss_out,
    int* __restrict__ count) {
  const int n = *n_eff;
  const int b = blockIdx.y;
  const int ld = d + SB_PSI;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j < ld) {
    float grad = 0.f;
    for (int i = 0; i < n; ++i)
      grad += ds[(size_t)i * 4 + b] *
              (j < d ? h[(size_t)i * d + j] : psi[(size_t)i * SB_PSI + j - d]);
    rank_w[(size_t)b * ld + j] -= lr * grad;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    float gb = 0.f;
    for (int i = 0; i < n; ++i) gb += ds[(size_t)i * 4 + b];
    rank_b[b] -= lr * gb;
    if (b == 0) {
      if (loss_out) {
        float t = 0.f;
        for (int i = 0; i < n; ++i) t += loss[i];
        *loss_out = n > 0 ? t / (float)n : 0.f;
      }
      *count = 0;
    }
  }
}

template <typename T>
void launch_adapt_prep(const float* h, const int* count, int cap,
                       const float* g, float eps, int d, T* A, int* n_eff,
                       hipStream_t st) {
  adapt_prep_kernel<T><<<cap, 256, 0, st>>>(h, count, cap, g, eps, d, A,
                                            n_eff);
}

template <typename T>
void launch_lm_update(T* W, int Vd, int d, const float* G, const T* A,
                      const int* n_eff, float lr, hipStream_t st) {
  constexpr int CW = sizeof(T) == 2 ? 256 : 128;
  const dim3 grid(Vd / kStripeRows, d / CW);
  lm_update_kernel<T, CW><<<grid, 256, 0, st>>>(W, Vd, d, G, A, n_eff, lr);
}

void launch_rank_update(float* rank_w, float* rank_b, const float* ds,
                        const float* h, const float* psi, int d,
                        const int* n_eff, float lr, const float* loss,
                        float* loss_out, int* count, hipStream_t st) {
  const dim3 grid((d + SB_PSI + 255) / 256, 4);
  rank_update_kernel<<<grid, 256, 0, st>>>(rank_w, rank_b, ds, h, psi, d,
                                           n_eff, lr, loss, loss_out, count);
}

int adapt_column_width(int elem_bytes) { return elem_bytes == 2 ? 256 : 128; }
int adapt_stripe_rows() { return kStripeRows; }

template void launch_adapt_prep<float>(const float*, const int*, int,
                                       const float*, float, int, float*, int*,
                                       hipStream_t);
template void launch_adapt_prep<bf16_t>(const float*, const int*, int,
                                        const float*, float, int, bf16_t*,
                                        int*, hipStream_t);
template void launch_lm_update<float>(float*, int, int, const float*,
                                      const float*, const int*, float,
                                      hipStream_t);
template void launch_lm_update<bf16_t>(bf16_t*, int, int, const float*,
                                       const bf16_t*, const int*, float,
                                       hipStream_t);

}  // namespace sb
