// Tree attention over a paged prefix plus a bit-masked segment (gfx950).
//
// Every query row of a sequence attends to all committed prefix entries
// and to the segment slots whose bit is set in its visibility words (tree
// ancestors-or-self for verification, on-path rows of earlier blocks plus
// its own block's rows <= k for the drafter, a causal chain for prefill).
//
// One wave owns 16 query vectors of one KV head (grouped-query attention:
// the G = H / Hkv query heads of a row share the KV head, so the 16 vectors
// are consecutive (row, head) pairs) and one split of the prefix.  Per tile
// of 32 keys it computes S^T = K Q^T with the keys as MFMA rows and the
// queries as columns, which leaves each lane holding the 8 scores of one
// query - exactly the B operand of O^T += V^T P^T - so the online softmax
// needs only a 4-lane reduction and P never leaves registers.  V pages are
// stored transposed ([hd][16 slots]) so the V^T operand is two 8/16-byte
// loads.  Splits are combined by attn_merge with log-sum-exp weights.
#include "common.h"
#include "kernels.h"

namespace sb {

#define SB_NEG (-1.0e30f)

template <typename T, int HD>
__device__ __forceinline__ void attn_tile(
    const T* __restrict__ k_base0, const T* __restrict__ k_base1,
    const T* __restrict__ v_base0, const T* __restrict__ v_base1,
    bool ok0, bool ok1, const Frag8<T> (&qf)[HD / 32], uint32_t valid_bits,
    float scale, float& m_run, float& l_run, f32x4_t (&acc)[HD / 16]) {
  const int lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  // S^T for the two 16-key halves
  f32x4_t s[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    s[h] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const T* kb = h ? k_base1 : k_base0;
    const bool ok = h ? ok1 : ok0;
#pragma unroll
    for (int c = 0; c < HD / 32; ++c) {
      Frag8<T> kf;
      if (ok)
        kf.load(kb + (size_t)r * HD + c * 32 + g * 8);
      else
        kf.zero();
      s[h] = mma_16x16x32(kf, qf[c], s[h]);
    }
  }
  // lane holds keys 16h + 4g + rr for query r; bit (16h + 4g + rr) of
  // valid_bits says whether that key is visible to this lane's query.
  float sc[8];
  float mx = SB_NEG;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int kk = 16 * h + 4 * g + rr;
      const bool v = (valid_bits >> kk) & 1u;
      const float x = v ? s[h][rr] * scale : SB_NEG;
      sc[h * 4 + rr] = x;
      mx = fmaxf(mx, x);
    }
  mx = fmaxf(mx, __shfl_xor(mx, 16, SB_WAVE));
  mx = fmaxf(mx, __shfl_xor(mx, 32, SB_WAVE));
  const float m_new = fmaxf(m_run, mx);
  const float alpha = __expf(m_run - m_new);
  float p[8];
  float ps = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int kk = 16 * (e >> 2) + 4 * g + (e & 3);
    const bool v = (valid_bits >> kk) & 1u;
    p[e] = v ? __expf(sc[e] - m_new) : 0.f;
    ps += p[e];
  }
  ps += __shfl_xor(ps, 16, SB_WAVE);
  ps += __shfl_xor(ps, 32, SB_WAVE);
  l_run = l_run * alpha + ps;
  m_run = m_new;
#pragma unroll
  for (int c = 0; c < HD / 16; ++c) acc[c] *= alpha;
  // P^T operand (keys {4g..4g+3, 16+4g..16+4g+3} x query r)
  Frag8<T> pf;
  if constexpr (sizeof(T) == 2) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = (uint32_t)f32_to_bf16(p[2 * e]) |
             ((uint32_t)f32_to_bf16(p[2 * e + 1]) << 16);
    pf.v = make_uint4(w[0], w[1], w[2], w[3]);
  } else {
    pf.a = make_float4(p[0], p[1], p[2], p[3]);
    pf.b = make_float4(p[4], p[5], p[6], p[7]);
  }
  // V^T operand: hd row 16c + r, the same 8 keys
#pragma unroll
  for (int c = 0; c < HD / 16; ++c) {
    Frag8<T> vf;
    const size_t off = ((size_t)(16 * c + r)) * 16 + 4 * g;
    if constexpr (sizeof(T) == 2) {
      uint2 a = ok0 ? *reinterpret_cast<const uint2*>(v_base0 + off)
                    : make_uint2(0, 0);
      uint2 b = ok1 ? *reinterpret_cast<const uint2*>(v_base1 + off)
                    : make_uint2(0, 0);
      vf.v = make_uint4(a.x, a.y, b.x, b.y);
    } else {
      vf.a = ok0 ? *reinterpret_cast<const float4*>(v_base0 + off)
                 : make_float4(0.f, 0.f, 0.f, 0.f);
      vf.b = ok1 ? *reinterpret_cast<const float4*>(v_base1 + off)
                 : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    acc[c] = mma_16x16x32(vf, pf, acc[c]);
  }
}

template <typename T, int HD>
__global__ __launch_bounds__(64) void tree_attn_kernel(
    const T* __restrict__ q, CallPlan p, KVView kv, int n_seqs, int H,
    int Hkv, int split_tokens, float scale, float* __restrict__ o_part,
    float* __restrict__ ml) {
  const int s = blockIdx.y / Hkv, kh = blockIdx.y % Hkv;
  if (s >= n_seqs) return;
  const int G = H / Hkv;
  const int row0 = p.seq_off[s];
  const int nrows = p.seq_off[s + 1] - row0;
  const int qv0 = blockIdx.x * 16;
  if (qv0 >= nrows * G) return;
  const int lane = threadIdx.x;
  const int r = lane & 15, g = lane >> 4;
  const int qv = qv0 + r;
  const bool qvalid = qv < nrows * G;
  const int qrow = row0 + (qvalid ? qv / G : 0);
  const int qh = kh * G + (qvalid ? qv % G : 0);

  Frag8<T> qf[HD / 32];
#pragma unroll
  for (int c = 0; c < HD / 32; ++c) {
    qf[c].load(q + ((size_t)qrow * H + qh) * HD + c * 32 + g * 8);
    if (!qvalid) qf[c].zero();
  }
  float m_run = SB_NEG, l_run = 0.f;
  f32x4_t acc[HD / 16];
#pragma unroll
  for (int c = 0; c < HD / 16; ++c) acc[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const T* kpool = static_cast<const T*>(kv.k);
  const T* vpool = static_cast<const T*>(kv.v);
  const int* ptab = kv.page_table + (size_t)s * kv.max_pages;
  const int Tp = min(p.prefix_len[s], kv.max_pages * 16);
  const int t0 = blockIdx.z * split_tokens;
  const int t1 = min(Tp, t0 + split_tokens);
  // the lane's query sees every prefix key < Tp: one bit per key of a tile
  for (int k0 = t0; k0 < t1; k0 += 32) {
    const int pg0 = k0 >> 4, pg1 = pg0 + 1;
    const bool ok0 = k0 < t1, ok1 = k0 + 16 < t1;
    const int pa = min(max(ok0 ? ptab[pg0] : 0, 0), kv.n_pages - 1);
    const int pb = min(max(ok1 ? ptab[pg1] : 0, 0), kv.n_pages - 1);
    const size_t b0 = ((size_t)pa * Hkv + kh) * 16 * HD;
    const size_t b1 = ((size_t)pb * Hkv + kh) * 16 * HD;
    const int nvalid = t1 - k0;
    const uint32_t bits = nvalid >= 32 ? 0xFFFFFFFFu : ((1u << nvalid) - 1u);
    attn_tile<T, HD>(kpool + b0, kpool + b1, vpool + b0, vpool + b1, ok0,
                     ok1, qf, bits, scale, m_run, l_run, acc);
  }
  if (blockIdx.z == gridDim.z - 1) {
    const int L = min(p.seg_len[s], kv.seg_pages * 16);
    const T* sk = static_cast<const T*>(kv.seg_k);
    const T* sv = static_cast<const T*>(kv.seg_v);
    const uint32_t* vis = p.vis + (size_t)qrow * p.vis_words;
    for (int k0 = 0; k0 < L; k0 += 32) {
      const int pg0 = k0 >> 4, pg1 = pg0 + 1;
      const bool ok0 = pg0 < kv.seg_pages, ok1 = pg1 < kv.seg_pages && k0 + 16 < L;
      const size_t b0 =
          (((size_t)s * kv.seg_pages + (ok0 ? pg0 : 0)) * Hkv + kh) * 16 * HD;
      const size_t b1 =
          (((size_t)s * kv.seg_pages + (ok1 ? pg1 : 0)) * Hkv + kh) * 16 * HD;
      const int nvalid = L - k0;
      uint32_t bits = nvalid >= 32 ? 0xFFFFFFFFu : ((1u << nvalid) - 1u);
      bits &= qvalid ? vis[k0 >> 5] : 0u;
      attn_tile<T, HD>(sk + b0, sk + b1, sv + b0, sv + b1, ok0, ok1, qf, bits,
                       scale, m_run, l_run, acc);
    }
  }
  if (!qvalid) return;
  const size_t cap = p.cap;
  float* o = o_part + (((size_t)blockIdx.z * cap + qrow) * H + qh) * HD;
#pragma unroll
  for (int c = 0; c < HD / 16; ++c)
    *reinterpret_cast<float4*>(o + 16 * c + 4 * g) =
        make_float4(acc[c][0], acc[c][1], acc[c][2], acc[c][3]);
  if (g == 0) {
    float* mlp = ml + (((size_t)blockIdx.z * cap + qrow) * H + qh) * 2;
    mlp[0] = m_run;
    mlp[1] = l_run;
  }
}

// Combine the splits of every (row, head): out = sum_z w_z O_z / sum_z w_z l_z
// with w_z = exp(m_z - max m).
template <typename T>
__global__ __launch_bounds__(256) void attn_merge_kernel(
    const float* __restrict__ o_part, const float* __restrict__ ml,
    const int* __restrict__ n, int cap, int H, int hd, int n_split,
    T* __restrict__ out) {
  __shared__ float wgt[64][32];
  __shared__ float inv_l[64];
  const int i = blockIdx.x;
  if (i >= *n) return;
  for (int h = threadIdx.x; h < H; h += blockDim.x) {
    float mx = SB_NEG;
    for (int z = 0; z < n_split; ++z)
      mx = fmaxf(mx, ml[(((size_t)z * cap + i) * H + h) * 2]);
    float L = 0.f;
    for (int z = 0; z < n_split; ++z) {
      const float* e = ml + (((size_t)z * cap + i) * H + h) * 2;
      const float w = (e[1] > 0.f) ? __expf(e[0] - mx) : 0.f;
      wgt[h][z] = w;
      L += w * e[1];
    }
    inv_l[h] = L > 0.f ? 1.0f / L : 0.f;
  }
  __syncthreads();
  for (int j = threadIdx.x; j < H * hd; j += blockDim.x) {
    const int h = j / hd;
    float v = 0.f;
    for (int z = 0; z < n_split; ++z)
      if (wgt[h][z] != 0.f) v += wgt[h][z] * o_part[((size_t)z * cap + i) * H * hd + j];
    out[(size_t)i * H * hd + j] = Elem<T>::from_f32(v * inv_l[h]);
  }
}

template <typename T>
void launch_tree_attn(const T* q, const CallPlan& p, const KVView& kv,
                      int rows_per_seq_cap, int H, int Hkv, int hd,
                      int n_split, int max_prefix, float* o_part, float* ml,
                      T* out, hipStream_t st) {
  const int G = H / Hkv;
  int split_tokens = (max_prefix + n_split - 1) / n_split;
  split_tokens = ((split_tokens + 31) / 32) * 32;
  if (split_tokens == 0) split_tokens = 32;
  const int n_seqs = p.n_seqs;
  dim3 grid((rows_per_seq_cap * G + 15) / 16, n_seqs * Hkv, n_split);
  const float scale = 1.0f / sqrtf((float)hd);
  if (hd == 128)
    tree_attn_kernel<T, 128><<<grid, 64, 0, st>>>(q, p, kv, n_seqs, H, Hkv,
                                                   split_tokens, scale, o_part,
                                                   ml);
  else
    tree_attn_kernel<T, 64><<<grid, 64, 0, st>>>(q, p, kv, n_seqs, H, Hkv,
                                                  split_tokens, scale, o_part,
                                                  ml);
  attn_merge_kernel<T><<<p.cap, 256, 0, st>>>(o_part, ml, p.n, p.cap, H, hd,
                                              n_split, out);
}

template void launch_tree_attn<float>(const float*, const CallPlan&,
                                      const KVView&, int, int, int, int, int,
                                      int, float*, float*, float*,
                                      hipStream_t);
template void launch_tree_attn<bf16_t>(const bf16_t*, const CallPlan&,
                                       const KVView&, int, int, int, int, int,
                                       int, float*, float*, bf16_t*,
                                       hipStream_t);

}  // namespace sb
