// Device-side helpers shared by the gfx950 kernels: bf16 storage,
// MFMA fragments, wavefront reductions.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define SB_WAVE 64
#define SB_TOPK_K 10   // top-k kept per drafter row
#define SB_PSI 15      // distribution summary size
#define SB_MAX_ANC_WORDS 16  // ancestor bit words (budget <= 512)

typedef uint16_t bf16_t;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// float -> bfloat16, round to nearest, ties to even (v_cvt_pk_bf16_f32;
// checked bit-exact against the integer rounding on finite inputs, ties
// included).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, (__bf16)f);
}
// Two values packed as (lo, hi) bf16 halves of one word.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// Storage-type traits: elem is float (SB_F32) or bf16_t (SB_BF16).
template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p) { return *p; }
  __device__ __forceinline__ static float to_f32(float v) { return v; }
  __device__ __forceinline__ static float from_f32(float v) { return v; }
};
template <> struct Elem<bf16_t> {
  __device__ __forceinline__ static float load(const bf16_t* p) {
    return bf16_to_f32(*p);
  }
  __device__ __forceinline__ static float to_f32(bf16_t v) {
    return bf16_to_f32(v);
  }
  __device__ __forceinline__ static bf16_t from_f32(float v) {
    return f32_to_bf16(v);
  }
};

// An MFMA operand fragment: 8 consecutive elements along the contraction
// dimension held by one lane (16 B for bf16, 32 B for float).
template <typename T> struct Frag8;
template <> struct Frag8<bf16_t> {
  uint4 v;
  __device__ __forceinline__ void load(const bf16_t* p) {
    v = *reinterpret_cast<const uint4*>(p);
  }
  __device__ __forceinline__ void zero() { v = make_uint4(0, 0, 0, 0); }
};
template <> struct Frag8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = reinterpret_cast<const float4*>(p)[0];
    b = reinterpret_cast<const float4*>(p)[1];
  }
  __device__ __forceinline__ void zero() {
    a = make_float4(0.f, 0.f, 0.f, 0.f);
    b = a;
  }
};

// acc[16x16] += A[16 x 32] * B[32 x 16] where lane l holds row (l % 16) of A
// and column (l % 16) of B, each with the 8 contraction indices of lane
// group l / 16.  Output: lane l holds acc[4 * (l / 16) + r][l % 16].
// bf16: one v_mfma_f32_16x16x32_bf16; float: eight v_mfma_f32_16x16x4_f32
// (element j of the fragment is contraction step j).
__device__ __forceinline__ f32x4_t mma_16x16x32(const Frag8<bf16_t>& a,
                                                const Frag8<bf16_t>& b,
                                                f32x4_t acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(
      __builtin_bit_cast(bf16x8_t, a.v), __builtin_bit_cast(bf16x8_t, b.v),
      acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mma_16x16x32(const Frag8<float>& a,
                                                const Frag8<float>& b,
                                                f32x4_t acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.a.x, b.a.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.a.y, b.a.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.a.z, b.a.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.a.w, b.a.w, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.b.x, b.b.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.b.y, b.b.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.b.z, b.b.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.b.w, b.b.w, acc, 0, 0, 0);
  return acc;
}

// Cross-lane exchanges on the VALU (no LDS permute): DPP within rows of 16
// lanes, v_permlane16_swap / v_permlane32_swap across rows.  Each step pairs
// every lane with one partner so that a symmetric op (sum, max) combines
// disjoint groups: xor 1 and xor 2 (quad_perm), 4-lane groups mirrored within
// 8 (row_half_mirror), 8-lane groups mirrored within 16 (row_mirror), then
// rows 2r <-> 2r+1 and halves 0-31 <-> 32-63.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
// op(v, v of lane l ^ 16) and op(v, v of lane l ^ 32), in every lane
__device__ __forceinline__ float2 swap16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v),
                                                  __float_as_uint(v), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float2 swap32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v),
                                                  __float_as_uint(v), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_x16(float v) { const float2 p = swap16(v); return p.x + p.y; }
__device__ __forceinline__ float sum_x32(float v) { const float2 p = swap32(v); return p.x + p.y; }
__device__ __forceinline__ float max_x16(float v) { const float2 p = swap16(v); return fmaxf(p.x, p.y); }
__device__ __forceinline__ float max_x32(float v) { const float2 p = swap32(v); return fmaxf(p.x, p.y); }

__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(v);    // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);    // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(v);   // row_half_mirror
  v += dpp_f<0x140>(v);   // row_mirror
  return sum_x32(sum_x16(v));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));
  v = fmaxf(v, dpp_f<0x4E>(v));
  v = fmaxf(v, dpp_f<0x141>(v));
  v = fmaxf(v, dpp_f<0x140>(v));
  return max_x32(max_x16(v));
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, SB_WAVE);
  return v;
}

// Sum over a block of `nthreads` threads (multiple of 64); `red` holds
// nthreads/64 floats of LDS.  Every thread gets the total.
__device__ __forceinline__ float block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

// Logical workgroup id for a launch of `total` workgroups whose neighbours
// should share an XCD's L2.  The dispatcher deals workgroups out round-robin
// over the 8 XCDs (id b to XCD b % 8); with total = 8 q + r, XCD x holds
// q + (x < r) of them and is given the contiguous logical ids starting at
// x q + min(x, r).  A bijection for every total (for r = 0 it is
// (b % 8) q + b / 8).
__device__ __forceinline__ int xcd_grouped(int b, int total) {
  const int x = b & 7, q = total >> 3, r = total & 7;
  return x * q + min(x, r) + (b >> 3);
}

// Larger (value, smaller id) first.
__device__ __forceinline__ bool better(float v, int id, float bv, int bid) {
  return v > bv || (v == bv && id < bid);
}

template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
__device__ __forceinline__ int2 swap16_i(int v) {
  const auto r = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v,
                                                  false, false);
  return make_int2((int)r[0], (int)r[1]);
}
__device__ __forceinline__ int2 swap32_i(int v) {
  const auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v,
                                                  false, false);
  return make_int2((int)r[0], (int)r[1]);
}
__device__ __forceinline__ void take_better(float& v, int& id, float v2,
                                            int i2) {
  if (better(v2, i2, v, id)) {
    v = v2;
    id = i2;
  }
}
// Wave-wide best (larger value, then smaller id); every lane gets it.  The
// same DPP / permlane pairing as wave_max (the combine is symmetric and
// idempotent), a few VALU cycles per step instead of an LDS permute.
__device__ __forceinline__ void wave_best_pair(float& v, int& id) {
  take_better(v, id, dpp_f<0xB1>(v), dpp_i<0xB1>(id));
  take_better(v, id, dpp_f<0x4E>(v), dpp_i<0x4E>(id));
  take_better(v, id, dpp_f<0x141>(v), dpp_i<0x141>(id));
  take_better(v, id, dpp_f<0x140>(v), dpp_i<0x140>(id));
  {
    const float2 a = swap16(v);
    const int2 b = swap16_i(id);
    v = a.x;
    id = b.x;
    take_better(v, id, a.y, b.y);
  }
  {
    const float2 a = swap32(v);
    const int2 b = swap32_i(id);
    v = a.x;
    id = b.x;
    take_better(v, id, a.y, b.y);
  }
}

// Wave-wide minimum of an int (DPP / permlane pairing as wave_max).
__device__ __forceinline__ int wave_min_i(int v) {
  v = min(v, dpp_i<0xB1>(v));
  v = min(v, dpp_i<0x4E>(v));
  v = min(v, dpp_i<0x141>(v));
  v = min(v, dpp_i<0x140>(v));
  const int2 a = swap16_i(v);
  v = min(a.x, a.y);
  const int2 b = swap32_i(v);
  return min(b.x, b.y);
}

// Exclusive wave prefix sum of small non-negative values (v < 2^BITS) by
// bit planes: one ballot and one masked bit count per bit; total in every
// lane.
template <int BITS>
__device__ __forceinline__ int wave_excl_scan_small(int v, int& total) {
  int excl = 0;
  total = 0;
#pragma unroll
  for (int b = 0; b < BITS; ++b) {
    const unsigned long long m = __ballot((v >> b) & 1);
    const int below = (int)__builtin_amdgcn_mbcnt_hi(
        (unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
    excl += below << b;
    total += __popcll(m) << b;
  }
  return excl;
}
