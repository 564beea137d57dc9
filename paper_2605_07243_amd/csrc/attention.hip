// Tree attention over a paged prefix plus a bit-masked segment (gfx950).
//
// Every query row of a sequence attends to all committed prefix entries
// and to the segment slots whose bit is set in its visibility words (tree
// ancestors-or-self for verification, on-path rows of earlier blocks plus
// its own block's rows <= k for the drafter, a causal chain for prefill).
//
// A q-tile is 16 query vectors of one KV head (grouped-query attention: the
// G = H / Hkv query heads of a row share the KV head, so the 16 vectors are
// consecutive (row, head) pairs); a wave owns one to four q-tiles and one
// split of the prefix.  Per tile
// of 32 keys it computes S^T = K Q^T with the keys as MFMA rows and the
// queries as columns, which leaves each lane holding the 8 scores of one
// query - exactly the B operand of O^T += V^T P^T - so the online softmax
// needs only a 4-lane reduction and P never leaves registers.  V pages are
// stored transposed ([hd][16 slots]) so the V^T operand is two 8/16-byte
// loads.  Splits are combined with log-sum-exp weights.
#include <hip/hip_ext.h>
#include "bounds.h"
#include "common.h"
#include "kernels.h"

namespace sb {

#define SB_NEG (-1.0e30f)

// Elements of a 16-byte V chunk whose key slot (first + e) is at or past
// nvalid are zeroed: slots that no call has written may hold anything, and
// a zero probability times a non-finite value would still poison the
// output (K needs no such care: masked scores are replaced, not scaled).
template <int ES>
__device__ __forceinline__ uint4 keep_slots(uint4 v, int first, int nvalid) {
  constexpr int EPC = 16 / ES;                      // elements per chunk
  if (first + EPC <= nvalid) return v;
  if (first >= nvalid) return make_uint4(0, 0, 0, 0);
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < EPC; ++e) {
    if (first + e < nvalid) continue;
    if constexpr (ES == 2)
      w[e >> 1] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
    else
      w[e] = 0u;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// One workgroup = NQ waves x QT q-tiles of 16 query vectors of one KV head
// (q-tile j of wave w is tile group * NQ * QT + j * NQ + w) and one split of
// the prefix (the last split also takes the segment).  K and V tiles of 32
// keys are staged once per workgroup in LDS (double buffered; global loads
// run four tiles ahead in registers) and read by every wave; a wave reuses
// every K and V operand it reads for its QT q-tiles, so a split's K/V is
// read once for up to 16 NQ QT query vectors.  With several splits each
// workgroup writes (O, m, l) partials that attn_merge combines; with one
// split the kernel writes the output.
template <typename T, int HD, int NQ, int QT>
__global__ __launch_bounds__(NQ * 64) void tree_attn_kernel(
    const T* __restrict__ q, CallPlan p, KVView kv, int H, int Hkv,
    int split_tokens, float scale, float* __restrict__ o_part,
    float* __restrict__ ml, T* __restrict__ out, int key_cap) {
  constexpr int ES = sizeof(T);
  constexpr int LDK = HD + 16 / ES;                 // padded K row
  constexpr int LDV = 32 + 16 / ES;                 // padded V^T row
  constexpr int KCH = 32 * HD * ES / 16;            // 16-byte chunks per K tile
  constexpr int VCH = HD * 32 * ES / 16;            // ... per V tile
  constexpr int CPR = HD * ES / 16;                 // chunks per K row
  constexpr int VCR = 16 * ES / 16;                 // chunks per V page row
  constexpr int NT = NQ * 64;
  constexpr int PER = (KCH + VCH + NT - 1) / NT;
  constexpr int QPW = NQ * QT;                      // q-tiles per workgroup
  __shared__ __attribute__((aligned(16))) T ksh[2][32][LDK];
  __shared__ __attribute__((aligned(16))) T vsh[2][HD][LDV];
  // XCD-grouped order: the dispatcher deals workgroups out round-robin over
  // the 8 XCDs, so neighbouring ids would land on different XCDs and each
  // fetch the same K/V or Q into its own L2.  Remapped, a run of consecutive
  // logical ids shares an XCD, and the logical order is q-group, then split,
  // then (sequence, KV head): the q-groups of a split share its K/V tiles,
  // the splits of a q-group its Q (one sequence of 60 nodes: one KV head per
  // XCD; fetched bytes per call 17.8 -> 7.9 MB with q-groups alone grouped)
  int bx = blockIdx.x, by = blockIdx.y, bz = blockIdx.z;
  {
    const int gx = gridDim.x, gy = gridDim.y;
    const int total = gx * gy * (int)gridDim.z;
    const int l = xcd_grouped(bx + gx * (by + gy * bz), total);
    const int gz = (int)gridDim.z;
    bx = l % gx;
    bz = (l / gx) % gz;
    by = l / (gx * gz);
  }
  const int s = by / Hkv, kh = by % Hkv;
  const int G = H / Hkv;
  const int row0 = p.seq_off[s];
  const int nq = (p.seq_off[s + 1] - row0) * G;
  const int qg = bx;
  if (qg * QPW * 16 >= nq) return;                  // uniform for the group
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int r = lane & 15, g = lane >> 4;
  bool qvalid[QT], live[QT];
  int qrow[QT], qh[QT];
  Frag8<T> qf[QT][HD / 32];
  float m_run[QT], l_run[QT];
  f32x4_t acc[QT][HD / 16];
#pragma unroll
  for (int j = 0; j < QT; ++j) {
    const int tile = qg * QPW + j * NQ + wave;
    const int qv = tile * 16 + r;
    qvalid[j] = qv < nq;
    live[j] = tile * 16 < nq;
    qrow[j] = row0 + (qvalid[j] ? qv / G : 0);
    qh[j] = kh * G + (qvalid[j] ? qv % G : 0);
#pragma unroll
    for (int c = 0; c < HD / 32; ++c) {
      qf[j][c].load(q + ((size_t)qrow[j] * H + qh[j]) * HD + c * 32 + g * 8);
      if (!qvalid[j]) qf[j][c].zero();
    }
    m_run[j] = SB_NEG;
    l_run[j] = 0.f;
#pragma unroll
    for (int c = 0; c < HD / 16; ++c) acc[j][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  bool wave_live = false;
#pragma unroll
  for (int j = 0; j < QT; ++j) wave_live |= live[j];

  const T* kpool = static_cast<const T*>(kv.k);
  const T* vpool = static_cast<const T*>(kv.v);
  const T* skp = static_cast<const T*>(kv.seg_k);
  const T* svp = static_cast<const T*>(kv.seg_v);
  const int* ptab = kv.page_table + (size_t)s * kv.max_pages;
  // committed keys: the prefix, within the page table and the length bound
  // (a bound below a prefix skips the entries past it)
  const int Tp = min(min(p.prefix_len[s], kv.max_pages * 16), key_cap);
  // the splits run over this sequence's own prefix: equal runs of whole
  // 32-key tiles (the host's split_tokens comes from a length bound that
  // can run well ahead of the prefix, which would leave the last splits
  // empty and the first ones longer); never longer than split_tokens, which
  // keeps a split within the page-table stage
  const int sp_tok =
      min(split_tokens, ((Tp + (int)gridDim.z - 1) / (int)gridDim.z + 31) & ~31);
  const int t0 = bz * sp_tok;
  const int t1 = min(Tp, t0 + sp_tok);
  const bool last_split = bz == gridDim.z - 1;
  const int L = last_split ? min(p.seg_len[s], kv.seg_pages * 16) : 0;
  const int n_pre = t1 > t0 ? (t1 - t0 + 31) / 32 : 0;
  const int n_tiles = n_pre + (L + 31) / 32;
  // the split's page-table entries, read once so that no tile fetch waits
  // on a dependent global load
  constexpr int MAXP = 1024;
  __shared__ int pg_sh[MAXP];
  const int pg0 = t0 >> 4;
  const int n_pg = t1 > t0 ? ((t1 + 15) >> 4) - pg0 : 0;
  for (int j = tid; j < n_pg && j < MAXP; j += NT)
    pg_sh[j] = checked_index(ptab[pg0 + j], kv.n_pages, kv.err, kDevPage);
  __syncthreads();

  // page base (element offset) of half h of tile i, or -1 when empty.  The
  // launch keeps a split within MAXP pages.
  auto page_base = [&](int i, int h) -> long long {
    if (i < n_pre) {
      const int k = t0 + i * 32 + h * 16;
      if (k >= t1) return -1;
      const int pg = pg_sh[min((k >> 4) - pg0, MAXP - 1)];
      return ((long long)pg * Hkv + kh) * 16 * HD;
    }
    const int k = (i - n_pre) * 32 + h * 16;
    if (k >= L || (k >> 4) >= kv.seg_pages) return -1;
    return (((long long)s * kv.seg_pages + (k >> 4)) * Hkv + kh) * 16 * HD;
  };
  // register ring of DEPTH tiles in flight; slot = tile index mod DEPTH.
  // Segment tiles also bring the visibility word of every q-tile's row
  // (segment tile w is word w).  Loads go to clamped addresses and their
  // values are used raw until the stash / compute of the tile (an empty
  // half reads page 0: its keys are masked and its V slots zeroed there),
  // so no load is consumed before its turn and the ring stays in flight.
  constexpr int DEPTH = 4;
  uint4 stg[DEPTH][PER];
  uint32_t visr[DEPTH][QT];
  auto fetch = [&](int i, uint4 (&dst)[PER], uint32_t (&vdst)[QT]) {
    const bool seg = i >= n_pre;
    const T* kp = seg ? skp : kpool;
    const T* vp = seg ? svp : vpool;
    const long long b0 = max(page_base(i, 0), 0LL);
    const long long b1 = max(page_base(i, 1), 0LL);
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int c = tid + e * NT;
      const int ck = min(c, KCH - 1);
      const int key = ck / CPR, kpart = ck % CPR;
      const T* ka = kp + (key < 16 ? b0 : b1) + (key & 15) * HD + kpart * (16 / ES);
      const int cv = min(max(c - KCH, 0), VCH - 1);
      const int hd = cv / (2 * VCR), rem = cv % (2 * VCR);
      const int h = rem / VCR, vpart = rem % VCR;
      const T* va = vp + (h ? b1 : b0) + hd * 16 + vpart * (16 / ES);
      dst[e] = *reinterpret_cast<const uint4*>(c < KCH ? ka : va);
    }
    const int wc = min(max(i - n_pre, 0), p.vis_words - 1);
#pragma unroll
    for (int j = 0; j < QT; ++j) vdst[j] = p.vis[(size_t)qrow[j] * p.vis_words + wc];
  };
  // valid keys of tile i
  auto n_valid = [&](int i) -> int {
    return i < n_pre ? min(32, t1 - (t0 + i * 32)) : min(32, L - (i - n_pre) * 32);
  };
  auto stash = [&](int i, int buf, const uint4 (&src)[PER]) {
    const int nv = n_valid(i);
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int c = tid + e * NT;
      if (c < KCH) {
        const int key = c / CPR, part = c % CPR;
        *reinterpret_cast<uint4*>(&ksh[buf][key][part * (16 / ES)]) = src[e];
      } else if (c < KCH + VCH) {
        const int cc = c - KCH;
        const int hd = cc / (2 * VCR), rem = cc % (2 * VCR);
        const int h = rem / VCR, part = rem % VCR;
        const int first = h * 16 + part * (16 / ES);
        *reinterpret_cast<uint4*>(&vsh[buf][hd][first]) = keep_slots<ES>(src[e], first, nv);
      }
    }
  };
  auto compute = [&](int i, int buf, const uint32_t (&vword)[QT]) {
    if (!wave_live) return;
    const bool seg = i >= n_pre;
    const bool vis_ok = seg && i - n_pre < p.vis_words;
    const int nvalid = n_valid(i);
    const uint32_t valid = nvalid >= 32 ? 0xFFFFFFFFu : ((1u << nvalid) - 1u);
    // S^T = K Q^T for the two 16-key halves, every q-tile
    f32x4_t sc4[QT][2];
#pragma unroll
    for (int j = 0; j < QT; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) sc4[j][h] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int c = 0; c < HD / 32; ++c) {
        Frag8<T> kf;
        kf.load(&ksh[buf][h * 16 + r][c * 32 + g * 8]);
#pragma unroll
        for (int j = 0; j < QT; ++j) sc4[j][h] = mma_16x16x32(kf, qf[j][c], sc4[j][h]);
      }
    Frag8<T> pf[QT];
#pragma unroll
    for (int j = 0; j < QT; ++j) {
      const uint32_t bits =
          seg ? ((vis_ok && qvalid[j]) ? (valid & vword[j]) : 0u) : valid;
      float sc[8];
      float mx = SB_NEG;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int kk = 16 * (e >> 2) + 4 * g + (e & 3);
        const bool v = (bits >> kk) & 1u;
        sc[e] = v ? sc4[j][e >> 2][e & 3] * scale : SB_NEG;
        mx = fmaxf(mx, sc[e]);
      }
      mx = max_x32(max_x16(mx));
      const float m_new = fmaxf(m_run[j], mx);
      const float alpha = __expf(m_run[j] - m_new);
      float pv[8];
      float ps = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int kk = 16 * (e >> 2) + 4 * g + (e & 3);
        pv[e] = ((bits >> kk) & 1u) ? __expf(sc[e] - m_new) : 0.f;
        ps += pv[e];
      }
      ps = sum_x32(sum_x16(ps));
      l_run[j] = l_run[j] * alpha + ps;
      m_run[j] = m_new;
#pragma unroll
      for (int c = 0; c < HD / 16; ++c) acc[j][c] *= alpha;
      if constexpr (ES == 2) {
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = pack_bf16x2(pv[2 * e], pv[2 * e + 1]);
        pf[j].v = make_uint4(w[0], w[1], w[2], w[3]);
      } else {
        pf[j].a = make_float4(pv[0], pv[1], pv[2], pv[3]);
        pf[j].b = make_float4(pv[4], pv[5], pv[6], pv[7]);
      }
    }
#pragma unroll
    for (int c = 0; c < HD / 16; ++c) {
      Frag8<T> vf;
      const T* vr = &vsh[buf][16 * c + r][4 * g];
      if constexpr (ES == 2) {
        const uint2 a = *reinterpret_cast<const uint2*>(vr);
        const uint2 b = *reinterpret_cast<const uint2*>(vr + 16);
        vf.v = make_uint4(a.x, a.y, b.x, b.y);
      } else {
        vf.a = *reinterpret_cast<const float4*>(vr);
        vf.b = *reinterpret_cast<const float4*>(vr + 16);
      }
#pragma unroll
      for (int j = 0; j < QT; ++j) acc[j][c] = mma_16x16x32(vf, pf[j], acc[j][c]);
    }
  };
  if (n_tiles > 0) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) fetch(min(d, n_tiles - 1), stg[d], visr[d]);
    stash(0, 0, stg[0]);
    __syncthreads();
    // tile i lives in slot i % DEPTH; after it is stashed the slot is
    // refilled with tile i + DEPTH (the last tile again past the end); its
    // visibility words are copied out before the refill
    for (int i0 = 0; i0 < n_tiles; i0 += DEPTH) {
#pragma unroll
      for (int d = 0; d < DEPTH; ++d) {
        const int i = i0 + d;
        uint32_t vword[QT];
#pragma unroll
        for (int j = 0; j < QT; ++j) vword[j] = visr[d][j];
        fetch(min(i + DEPTH, n_tiles - 1), stg[d], visr[d]);
        if (i < n_tiles) compute(i, i & 1, vword);
        if (i + 1 < n_tiles) stash(i + 1, (i + 1) & 1, stg[(d + 1) % DEPTH]);
        __syncthreads();
      }
    }
  }

  const int n_split = gridDim.z;
  const size_t cap = p.cap;
#pragma unroll
  for (int j = 0; j < QT; ++j) {
    if (!qvalid[j]) continue;
    if (n_split == 1) {
      const float il = l_run[j] > 0.f ? 1.0f / l_run[j] : 0.f;
      T* o = out + (size_t)qrow[j] * H * HD + (size_t)qh[j] * HD;
#pragma unroll
      for (int c = 0; c < HD / 16; ++c)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
          o[16 * c + 4 * g + rr] = Elem<T>::from_f32(acc[j][c][rr] * il);
      continue;
    }
    float* o = o_part + (((size_t)bz * cap + qrow[j]) * H + qh[j]) * HD;
#pragma unroll
    for (int c = 0; c < HD / 16; ++c)
      *reinterpret_cast<float4*>(o + 16 * c + 4 * g) =
          make_float4(acc[j][c][0], acc[j][c][1], acc[j][c][2], acc[j][c][3]);
    if (g == 0) {
      float* mlp = ml + (((size_t)bz * cap + qrow[j]) * H + qh[j]) * 2;
      mlp[0] = m_run[j];
      mlp[1] = l_run[j];
    }
  }
}


// bf16 tree attention on 32x32x16 MFMAs.  A wave owns 32 query vectors of
// one KV head (lane l: query l % 32; the two lane halves split the
// contraction), a workgroup NW waves, one split of the prefix; keys come in
// tiles of 64 (four 16-key pages).  Per tile a wave computes
// S^T = K Q^T for two 32-key blocks (8 MFMAs each over head_dim 128), so a
// lane holds 16 scores of its query per block and the softmax reductions
// are in-lane plus one swap with lane l ^ 32.  The scores of key-block b,
// converted to bf16, are directly the B operand of O^T += V^T P^T when V^T
// is read from LDS with the same key permutation (keys 4h..4h+3 and
// 8+4h..8+4h+3 of each 16-key step for lane half h), so P never leaves
// registers.  K [64][HD] and V^T [HD][64] tiles are staged once per
// workgroup in LDS (double buffered, padded rows: conflict-free 16-byte K
// reads and 8-byte V^T reads), global loads run DEPTH tiles ahead.
// Balanced splits (one 8-wave workgroup of the 32x32 kernel fills a CU, so
// a launch runs in one round only with at most kAttnSlots workgroups): the
// prefix of every sequence with rows is cut into splits of sp tiles of 64
// keys, sp the smallest value for which all (sequence, split, KV head,
// query group) items fit the slots (and no sequence needs more than
// max_split splits); workgroup b takes item b, items ordered by sequence,
// then split, then KV head and query group.  Every wave works this out on
// its own from the prefix lengths (binary search over sp, then a wave scan
// of the items per sequence); the host guarantees at most 64 sequences,
// prefixes of at most 256 tiles and sequences x items per split <= slots,
// so sp = 256 always fits.
constexpr int kAttnSlots = 256;

struct SplitItem {
  bool live;
  int s, z, nz, sp, item;
};

__device__ __forceinline__ int n_splits_of(int tiles, int sp) {
  return tiles > 0 ? (tiles + sp - 1) / sp : 1;
}

__device__ SplitItem balanced_split(const CallPlan& p, int max_pages, int gx,
                                    int max_split, int b, int key_cap) {
  const int lane = threadIdx.x & 63;
  bool act = false;
  int t = 0;
  if (lane < p.n_seqs) {
    act = p.seq_off[lane + 1] > p.seq_off[lane];
    t = (min(min(p.prefix_len[lane], max_pages * 16), key_cap) + 63) >> 6;
  }
  const int total = wave_sum_i(act ? t : 0);
  int tmax = act ? t : 0;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) tmax = max(tmax, __shfl_xor(tmax, o, SB_WAVE));
  int lo = max(1, max((total * gx + kAttnSlots - 1) / kAttnSlots,
                      (tmax + max_split - 1) / max_split));
  int hi = max(lo, 256);
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    const int used = wave_sum_i(act ? n_splits_of(t, mid) : 0);
    if (used * gx <= kAttnSlots) hi = mid;
    else lo = mid + 1;
  }
  const int nz = act ? n_splits_of(t, lo) : 0;
  int inc = nz * gx;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(inc, o, SB_WAVE);
    if (lane >= o) inc += v;
  }
  const int exc = inc - nz * gx;
  const unsigned long long m = __ballot(act && exc <= b && b < inc);
  SplitItem r{};
  if (m == 0) return r;
  const int sl = __builtin_ctzll(m);
  const int local = b - __shfl(exc, sl, SB_WAVE);
  r.live = true;
  r.s = sl;
  r.sp = lo;
  r.nz = __shfl(nz, sl, SB_WAVE);
  r.z = local / gx;
  r.item = local % gx;
  return r;
}

typedef float attn_f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int attn_u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ attn_f32x16_t mma32_attn(attn_u32x4_t a, attn_u32x4_t b,
                                                   attn_f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(
      __builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c, 0,
      0, 0);
}

// split_rows == nullptr: grid (query groups, sequences x KV heads, splits)
// with fixed splits of split_tokens keys; else a grid of kAttnSlots
// balanced items (above), and the split count of every row's sequence is
// written to split_rows for the merge.
template <int HD, int NW>
__global__ __launch_bounds__(NW * 64) void tree_attn32_kernel(
    const bf16_t* __restrict__ q, CallPlan p, KVView kv, int H, int Hkv,
    int split_tokens, float scale, float* __restrict__ o_part,
    float* __restrict__ ml, bf16_t* __restrict__ out, int n_groups,
    int max_split, int* __restrict__ split_rows, int key_cap) {
  constexpr int KT = 64;                    // keys per tile
  constexpr int LDK = HD + 8;               // K row: 16 B mod 256 B
  constexpr int LDV = KT + 4;               // V^T row: 136 B, 8-byte reads
  constexpr int NT = NW * 64;
  constexpr int KCH = KT * HD / 8;          // 16-byte chunks of a K tile
  constexpr int CH = 2 * KCH;               // K + V chunks per tile
  constexpr int PER = (CH + NT - 1) / NT;
  constexpr int HB = HD / 32;               // head_dim blocks of 32
  constexpr int QK = HD / 16;               // contraction steps of S^T
  constexpr int DEPTH = NW >= 8 ? 1 : 3;     // staging registers: 16 PER each
  __shared__ __attribute__((aligned(16))) bf16_t ksh[2][KT][LDK];
  __shared__ __attribute__((aligned(16))) bf16_t vsh[2][HD][LDV];
  constexpr int MAXP = 1024;
  __shared__ int pg_sh[MAXP];
  // XCD-grouped order as in the 16-row kernel (fixed splits: q-group, split,
  // then (sequence, KV head)); balanced items are ordered by sequence, split,
  // KV head and q-group, so neighbouring items again share K/V or Q
  int bx = blockIdx.x, by = blockIdx.y, bz = blockIdx.z;
  {
    const int gx = gridDim.x, gy = gridDim.y;
    const int total = gx * gy * (int)gridDim.z;
    const int l = xcd_grouped(bx + gx * (by + gy * bz), total);
    const int gz = (int)gridDim.z;
    bx = l % gx;
    bz = (l / gx) % gz;
    by = l / (gx * gz);
  }
  int s, kh, qg, zs, nzs, split_tok;
  if (split_rows != nullptr) {
    const SplitItem it =
        balanced_split(p, kv.max_pages, Hkv * n_groups, max_split, bx, key_cap);
    if (!it.live) return;                   // uniform: every wave agrees
    s = it.s;
    kh = it.item / n_groups;
    qg = it.item % n_groups;
    zs = it.z;
    nzs = it.nz;
    split_tok = it.sp * 64;
  } else {
    s = by / Hkv;
    kh = by % Hkv;
    qg = bx;
    zs = bz;
    nzs = gridDim.z;
    split_tok = -1;   // set from the prefix below
  }
  const int G = H / Hkv;
  const int row0 = p.seq_off[s];
  const int nq = (p.seq_off[s + 1] - row0) * G;
  if (split_rows != nullptr && zs == 0 && kh == 0 && qg == 0)
    for (int r = row0 + (int)threadIdx.x; r < p.seq_off[s + 1]; r += NW * 64)
      split_rows[r] = nzs;
  if (qg * NW * 32 >= nq) return;           // uniform for the group
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lq = lane & 31, h = lane >> 5;
  const int qv = (qg * NW + wave) * 32 + lq;
  const bool qvalid = qv < nq;
  const bool wave_live = (qg * NW + wave) * 32 < nq;
  const int qrow = row0 + (qvalid ? qv / G : 0);
  const int qh = kh * G + (qvalid ? qv % G : 0);
  attn_u32x4_t qf[QK];
#pragma unroll
  for (int j = 0; j < QK; ++j) {
    qf[j] = *reinterpret_cast<const attn_u32x4_t*>(
        q + ((size_t)qrow * H + qh) * HD + 16 * j + 8 * h);
    if (!qvalid) qf[j] = attn_u32x4_t{0u, 0u, 0u, 0u};
  }
  float m_run = SB_NEG, l_run = 0.f;
  attn_f32x16_t acc[HB];
#pragma unroll
  for (int b = 0; b < HB; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[b][r] = 0.f;

  const bf16_t* kpool = static_cast<const bf16_t*>(kv.k);
  const bf16_t* vpool = static_cast<const bf16_t*>(kv.v);
  const bf16_t* skp = static_cast<const bf16_t*>(kv.seg_k);
  const bf16_t* svp = static_cast<const bf16_t*>(kv.seg_v);
  const int* ptab = kv.page_table + (size_t)s * kv.max_pages;
  // committed keys: the prefix, within the page table and the length bound
  // (a bound below a prefix skips the entries past it)
  const int Tp = min(min(p.prefix_len[s], kv.max_pages * 16), key_cap);
  // fixed splits run over this sequence's own prefix (equal runs of whole
  // 64-key tiles, never longer than split_tokens), as in tree_attn_kernel
  if (split_tok < 0)
    split_tok = min(split_tokens, ((Tp + nzs - 1) / nzs + 63) & ~63);
  const int t0 = zs * split_tok;
  const int t1 = min(Tp, t0 + split_tok);
  const bool last_split = zs == nzs - 1;
  const int L = last_split ? min(p.seg_len[s], kv.seg_pages * 16) : 0;
  const int n_pre = t1 > t0 ? (t1 - t0 + KT - 1) / KT : 0;
  const int n_tiles = n_pre + (L + KT - 1) / KT;
  const int pg0 = t0 >> 4;
  const int n_pg = t1 > t0 ? ((t1 + 15) >> 4) - pg0 : 0;
  for (int j = tid; j < n_pg && j < MAXP; j += NT)
    pg_sh[j] = checked_index(ptab[pg0 + j], kv.n_pages, kv.err, kDevPage);
  __syncthreads();

  // element offset of page pp (0..3) of tile i in its pool, or -1 (empty;
  // the launch keeps a split within MAXP pages)
  auto page_base = [&](int i, int pp) -> long long {
    if (i < n_pre) {
      const int k = t0 + i * KT + pp * 16;
      if (k >= t1) return -1;
      const int pg = pg_sh[min((k >> 4) - pg0, MAXP - 1)];
      return ((long long)pg * Hkv + kh) * 16 * HD;
    }
    const int k = (i - n_pre) * KT + pp * 16;
    if (k >= L || (k >> 4) >= kv.seg_pages) return -1;
    return (((long long)s * kv.seg_pages + (k >> 4)) * Hkv + kh) * 16 * HD;
  };
  // Chunk c of a tile (16 bytes): c < KCH is K of page c / KPC, key
  // (c % KPC) / (HD / 8), elements 8 (c % (HD / 8)); c = KCH + c' is V^T of
  // page c' / (2 HD), head_dim row (c' % (2 HD)) / 2, slots 8 (c' % 2).
  // Every thread's chunks sit at the same page and offset in every tile.
  constexpr int KPC = 16 * HD / 8;          // K chunks per page
  static_assert(KCH % NT == 0, "a thread's chunks are all K or all V");
  int c_pg[PER], c_off[PER], c_lds[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int c = tid + e * NT;
    if (e * NT < KCH) {
      const int krem = c % KPC, key = 16 * (c / KPC) + krem / (HD / 8);
      c_pg[e] = c / KPC;
      c_off[e] = (krem / (HD / 8)) * HD + (krem % (HD / 8)) * 8;
      c_lds[e] = key * LDK + (krem % (HD / 8)) * 8;
    } else {
      const int cv = min(c - KCH, KCH - 1);
      const int vrem = cv % (2 * HD);
      c_pg[e] = cv / (2 * HD);
      c_off[e] = (vrem / 2) * 16 + (vrem % 2) * 8;
      c_lds[e] = (vrem / 2) * LDV + 16 * (cv / (2 * HD)) + 8 * (vrem % 2);
    }
  }
  attn_u32x4_t stg[DEPTH][PER];
  uint32_t visr[DEPTH][2];
  auto fetch = [&](int i, attn_u32x4_t (&dst)[PER], uint32_t (&vdst)[2]) {
    const bool seg = i >= n_pre;
    const bf16_t* kp = seg ? skp : kpool;
    const bf16_t* vp = seg ? svp : vpool;
    long long pb[4];
#pragma unroll
    for (int pp = 0; pp < 4; ++pp) pb[pp] = max(page_base(i, pp), 0LL);
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const long long base = c_pg[e] == 0 ? pb[0] : c_pg[e] == 1 ? pb[1]
                           : c_pg[e] == 2 ? pb[2] : pb[3];
      const bf16_t* src = (e * NT < KCH ? kp : vp) + base + c_off[e];
      dst[e] = *reinterpret_cast<const attn_u32x4_t*>(src);
    }
    const int w0 = min(max(2 * (i - n_pre), 0), p.vis_words - 1);
    const int w1 = min(w0 + 1, p.vis_words - 1);
    vdst[0] = p.vis[(size_t)qrow * p.vis_words + w0];
    vdst[1] = p.vis[(size_t)qrow * p.vis_words + w1];
  };
  auto n_valid = [&](int i) -> int {
    return i < n_pre ? min(KT, t1 - (t0 + i * KT)) : min(KT, L - (i - n_pre) * KT);
  };
  // V^T slots at or past the tile's valid keys are zeroed (never-written
  // slots may hold anything; a zero probability would not cancel a NaN)
  auto stash = [&](int i, int buf, const attn_u32x4_t (&src)[PER]) {
    const int nv = n_valid(i);
    bf16_t* kb = &ksh[buf][0][0];
    bf16_t* vb = &vsh[buf][0][0];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      if (e * NT < KCH) {
        *reinterpret_cast<attn_u32x4_t*>(kb + c_lds[e]) = src[e];
      } else if (tid + e * NT < CH) {
        uint4 v = make_uint4(src[e][0], src[e][1], src[e][2], src[e][3]);
        if (nv < KT) v = keep_slots<2>(v, c_lds[e] % LDV, nv);
        *reinterpret_cast<uint2*>(vb + c_lds[e]) = make_uint2(v.x, v.y);
        *reinterpret_cast<uint2*>(vb + c_lds[e] + 4) = make_uint2(v.z, v.w);
      }
    }
  };
  // Scores in log2 units (scale * log2 e folded in).  The reference max
  // used for the exponentials moves only when a score exceeds it by more
  // than 8 (then every probability is <= 2^8 and O, l are rescaled once);
  // O / l is exact either way, and the (O, m, l) partials carry the
  // reference.
  const float sl2 = scale * 1.44269504088896341f;
  constexpr float kMasked = -3.0e38f;
  auto compute = [&](int i, int buf, const uint32_t (&vw)[2]) {
    if (!wave_live) return;
    const bool seg = i >= n_pre;
    const int nv = n_valid(i);
    const bool full = !seg && nv == KT;
    const int w = i - n_pre;
    attn_f32x16_t sc[2];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[b][r] = 0.f;
    // the two 32-key blocks' chains interleaved, each K fragment read one
    // contraction step ahead of its MFMA
    auto kfrag = [&](int b, int j) {
      return *reinterpret_cast<const attn_u32x4_t*>(&ksh[buf][32 * b + lq][16 * j + 8 * h]);
    };
    attn_u32x4_t kf0 = kfrag(0, 0), kf1 = kfrag(1, 0);
#pragma unroll
    for (int j = 0; j < QK; ++j) {
      const attn_u32x4_t nx0 = kfrag(0, min(j + 1, QK - 1));
      const attn_u32x4_t nx1 = kfrag(1, min(j + 1, QK - 1));
      sc[0] = mma32_attn(kf0, qf[j], sc[0]);
      sc[1] = mma32_attn(kf1, qf[j], sc[1]);
      kf0 = nx0;
      kf1 = nx1;
    }
    // V^T fragment of PV step t = (2 b + u) HB + hb; each is read two steps
    // ahead, the first two before the softmax (the barrier keeps the
    // compiler from sinking them next to their MFMAs)
    constexpr int NPV = 4 * HB;
    auto vfrag = [&](int t) {
      const int b = t / (2 * HB), u = (t / HB) % 2, hb = t % HB;
      const bf16_t* vr = &vsh[buf][32 * hb + lq][32 * b + 16 * u + 4 * h];
      const uint2 lo = *reinterpret_cast<const uint2*>(vr);
      const uint2 hi = *reinterpret_cast<const uint2*>(vr + 8);
      return attn_u32x4_t{lo.x, lo.y, hi.x, hi.y};
    };
    attn_u32x4_t vf0 = vfrag(0), vf1 = vfrag(1);
    __builtin_amdgcn_sched_barrier(0);
    // lane register r of block b is key 32 b + 8 (r / 4) + 4 h + r % 4
    float mx = SB_NEG;
    if (full) {
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sc[b][r] *= sl2;
          mx = fmaxf(mx, sc[b][r]);
        }
    } else {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int nb = min(max(nv - 32 * b, 0), 32);
        uint32_t m = nb >= 32 ? 0xFFFFFFFFu : ((1u << nb) - 1u);
        if (seg) m &= (qvalid && 2 * w + b < p.vis_words) ? vw[b] : 0u;
        m >>= 4 * h;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int k = 8 * (r >> 2) + (r & 3);
          sc[b][r] = ((m >> k) & 1u) ? sc[b][r] * sl2 : kMasked;
          mx = fmaxf(mx, sc[b][r]);
        }
      }
    }
    mx = max_x32(mx);
    // move the reference (wave-uniform decision) only when needed
    if (__builtin_amdgcn_ballot_w64(mx > m_run + 8.0f) != 0) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int hb = 0; hb < HB; ++hb) acc[hb] *= alpha;
      m_run = m_new;
    }
    float ps = 0.f;
    attn_u32x4_t pf[2][2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      float pv[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        // masked scores sit far below any reference (which starts at
        // -1e30): exp2 underflows to 0
        pv[r] = __builtin_amdgcn_exp2f(sc[b][r] - m_run);
        ps += pv[r];
      }
#pragma unroll
      for (int u = 0; u < 2; ++u)
        pf[b][u] = attn_u32x4_t{pack_bf16x2(pv[8 * u], pv[8 * u + 1]),
                                pack_bf16x2(pv[8 * u + 2], pv[8 * u + 3]),
                                pack_bf16x2(pv[8 * u + 4], pv[8 * u + 5]),
                                pack_bf16x2(pv[8 * u + 6], pv[8 * u + 7])};
    }
    l_run += sum_x32(ps);
    // O^T[hd][query] += V^T[hd][keys] P^T[keys][query], 16 keys per step
#pragma unroll
    for (int t = 0; t < NPV; ++t) {
      const attn_u32x4_t vf2 = vfrag(min(t + 2, NPV - 1));
      const int b = t / (2 * HB), u = (t / HB) % 2, hb = t % HB;
      acc[hb] = mma32_attn(vf0, pf[b][u], acc[hb]);
      vf0 = vf1;
      vf1 = vf2;
    }
  };
  if (n_tiles > 0) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) fetch(min(d, n_tiles - 1), stg[d], visr[d]);
    stash(0, 0, stg[0]);
    __syncthreads();
    for (int i0 = 0; i0 < n_tiles; i0 += DEPTH) {
#pragma unroll
      for (int d = 0; d < DEPTH; ++d) {
        const int i = i0 + d;
        uint32_t vw[2] = {visr[d][0], visr[d][1]};
        fetch(min(i + DEPTH, n_tiles - 1), stg[d], visr[d]);
        if (i < n_tiles) compute(i, i & 1, vw);
        if (i + 1 < n_tiles) stash(i + 1, (i + 1) & 1, stg[(d + 1) % DEPTH]);
        __syncthreads();
      }
    }
  }
  if (!qvalid) return;
  // lane register r of head_dim block hb is element 32 hb + 8 (r / 4) +
  // 4 h + r % 4 of this lane's query
  if (split_rows == nullptr && gridDim.z == 1) {
    const float il = l_run > 0.f ? 1.0f / l_run : 0.f;
    bf16_t* o = out + ((size_t)qrow * H + qh) * HD;
#pragma unroll
    for (int hb = 0; hb < HB; ++hb)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        *reinterpret_cast<uint2*>(o + 32 * hb + 8 * g4 + 4 * h) =
            make_uint2(pack_bf16x2(acc[hb][4 * g4] * il, acc[hb][4 * g4 + 1] * il),
                       pack_bf16x2(acc[hb][4 * g4 + 2] * il, acc[hb][4 * g4 + 3] * il));
    return;
  }
  float* o = o_part + (((size_t)zs * p.cap + qrow) * H + qh) * HD;
#pragma unroll
  for (int hb = 0; hb < HB; ++hb)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4)
      *reinterpret_cast<float4*>(o + 32 * hb + 8 * g4 + 4 * h) =
          make_float4(acc[hb][4 * g4], acc[hb][4 * g4 + 1], acc[hb][4 * g4 + 2],
                      acc[hb][4 * g4 + 3]);
  if (h == 0) {
    float* mlp = ml + (((size_t)zs * p.cap + qrow) * H + qh) * 2;
    mlp[0] = m_run * 0.69314718055994531f;   // natural-log units
    mlp[1] = l_run;
  }
}


// Combine the splits of every (row, head): out = sum_z w_z O_z / sum_z w_z l_z
// with w_z = exp(m_z - max m).  A separate launch: the kernel boundary
// orders the partial writes of every XCD before the reads.  One workgroup
// per row; a thread owns one float4 column per pass, and the first pass's
// partial loads are issued before the (m, l) loads and the weights, so a
// row of up to 4 BT columns costs one memory round trip.
template <int NS>
constexpr int merge_threads() { return NS <= 16 ? 1024 : 512; }

template <int NS>
__global__ __launch_bounds__(merge_threads<NS>()) void attn_merge_kernel_t(
    const float* __restrict__ o_part, const float* __restrict__ ml,
    const int* __restrict__ n, int cap, int H, int hd, int n_split,
    void* out_v, int es, const int* __restrict__ split_rows) {
  constexpr int BT = merge_threads<NS>();
  __shared__ float wgt[64][NS];
  __shared__ float inv_l[64];
  const int i = blockIdx.x;
  if (i >= *n) return;
  // splits written for this row (balanced launches: its sequence's count;
  // the other slots hold stale data and are never read)
  if (split_rows != nullptr) n_split = min(n_split, split_rows[i]);
  const size_t zs = (size_t)cap * H * hd;
  const int ncol = (H * hd) >> 2;
  const float* row = o_part + (size_t)i * H * hd;
  auto load = [&](int c, float4 (&o)[NS]) {
#pragma unroll
    for (int z = 0; z < NS; ++z)
      o[z] = (z < n_split && c < ncol)
                 ? *reinterpret_cast<const float4*>(row + z * zs + 4 * c)
                 : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  auto combine = [&](int c, const float4 (&o)[NS]) {
    if (c >= ncol) return;
    const int j = 4 * c, hh = j / hd;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int z = 0; z < NS; ++z) {
      const float w = wgt[hh][z];
      v.x += w * o[z].x;
      v.y += w * o[z].y;
      v.z += w * o[z].z;
      v.w += w * o[z].w;
    }
    const float il = inv_l[hh];
    v = make_float4(v.x * il, v.y * il, v.z * il, v.w * il);
    const size_t off = (size_t)i * H * hd + j;
    if (es == 2) {
      uint2 u;
      u.x = pack_bf16x2(v.x, v.y);
      u.y = pack_bf16x2(v.z, v.w);
      *reinterpret_cast<uint2*>(static_cast<bf16_t*>(out_v) + off) = u;
    } else {
      *reinterpret_cast<float4*>(static_cast<float*>(out_v) + off) = v;
    }
  };
  float4 o[NS];
  load(threadIdx.x, o);
  const int h = threadIdx.x;
  if (h < H) {
    float mz[NS], lz[NS];
    float mx = SB_NEG;
#pragma unroll
    for (int z = 0; z < NS; ++z) {
      float2 e = make_float2(SB_NEG, 0.f);
      if (z < n_split)
        e = *reinterpret_cast<const float2*>(ml + (((size_t)z * cap + i) * H + h) * 2);
      mz[z] = e.x;
      lz[z] = e.y;
      if (e.y > 0.f) mx = fmaxf(mx, e.x);
    }
    float L = 0.f;
#pragma unroll
    for (int z = 0; z < NS; ++z) {
      const float w = lz[z] > 0.f ? __expf(mz[z] - mx) : 0.f;
      wgt[h][z] = w;
      L += w * lz[z];
    }
    inv_l[h] = L > 0.f ? 1.0f / L : 0.f;
  }
  __syncthreads();
  combine(threadIdx.x, o);
  for (int c = threadIdx.x + BT; c < ncol; c += BT) {
    load(c, o);
    combine(c, o);
  }
}

template <typename T>
void launch_attn_merge(const CallPlan& p, int H, int hd, int n_split,
                       const float* o_part, const float* ml, T* out,
                       hipStream_t st, hipEvent_t stop,
                       const int* split_rows = nullptr);

namespace {

// q-tiles of 16 query vectors per workgroup: NQ waves x QT tiles each.  Two
// q-tiles per wave (one read of a split's K/V for twice the queries) pay
// off when there are enough (sequence, KV head) pairs to fill the chip
// without cutting the prefix into short splits; with few pairs the
// parallelism has to come from the splits, and one q-tile per wave keeps
// each split's chain short (measured: 16 sequences x 8 KV heads gain 14%,
// one sequence loses 8-15%).
struct AttnShape {
  bool mfma32;   // bf16 32x32x16 kernel (else 16-row q-tiles)
  int nq, qt, groups;
};
AttnShape attn_shape(int rows_per_seq_cap, int G, int seq_heads, int es) {
  AttnShape a{};
  if (es == 2 && (seq_heads >= 32 || rows_per_seq_cap * G >= 512)) {
    // many (sequence, KV head) pairs, or at least 512 query vectors per KV
    // head: the 32x32x16 kernel, waves of 32 query vectors, 4 or 8 per
    // workgroup (at least four waves share the tile loads; waves past the
    // queries only load).  With few pairs and few queries the parallelism
    // has to come from the splits and the 16-row q-tiles of the other
    // kernel keep each split's chain shorter (measured faster for one
    // sequence of 60 tree nodes; at 128 nodes x 4 query heads the 32x32
    // kernel with balanced splits reads each K/V tile for 256 queries
    // instead of 64: +12% attention throughput).
    const int qblocks = (rows_per_seq_cap * G + 31) / 32;
    a.mfma32 = true;
    a.nq = qblocks > 4 ? 8 : 4;
    a.qt = 1;
    a.groups = (qblocks + a.nq - 1) / a.nq;
    return a;
  }
  const int qtiles = (rows_per_seq_cap * G + 15) / 16;
  a.mfma32 = false;
  a.nq = qtiles >= 8 ? 8 : (qtiles >= 4 ? 4 : (qtiles >= 2 ? 2 : 1));
  // bf16 with few pairs: at most four waves per workgroup (one per SIMD, so
  // a split's tile chain is not shared with a second wave; twice the
  // workgroups): 5% faster at 60 tree nodes, 12% at 128 (measured)
  if (es == 2) a.nq = a.nq > 4 ? 4 : a.nq;
  a.qt = (qtiles > 8 && seq_heads >= 32) ? 2 : 1;  // 8 x 2 fits 256 VGPRs
  a.groups = (qtiles + a.nq * a.qt - 1) / (a.nq * a.qt);
  return a;
}

}  // namespace

namespace {

// Timing events for the next tree-attention call (kernel start, merge or
// kernel end), set by the library's profiler and consumed by one call.
thread_local hipEvent_t g_attn_start = nullptr, g_attn_stop = nullptr;

}  // namespace

void attn_time_next_launch(hipEvent_t start, hipEvent_t stop) {
  g_attn_start = start;
  g_attn_stop = stop;
}

bool attn_time_pending() { return g_attn_start != nullptr; }

template <typename T>
void launch_tree_attn(const T* q, const CallPlan& p, const KVView& kv,
                      int rows_per_seq_cap, int H, int Hkv, int hd,
                      int n_split, int max_prefix, float* o_part, float* ml,
                      T* out, int max_split, int* split_rows, hipStream_t st) {
  hipEvent_t ea = g_attn_start, eb = g_attn_stop;
  g_attn_start = g_attn_stop = nullptr;
  // with a merge, the kernel carries the start event and the merge the stop
  hipEvent_t ka = ea, kb = n_split > 1 ? nullptr : eb;
  AttnShape a =
      attn_shape(rows_per_seq_cap, H / Hkv, p.n_seqs * Hkv, (int)sizeof(T));
  if (sizeof(T) == 4 && hd == 128) {
    // fp32 with 128-wide heads: at least two waves and one q-tile each (a
    // lone wave's registers spill, and so do two q-tiles per wave); waves
    // past the queries only load
    const int qtiles = (rows_per_seq_cap * (H / Hkv) + 15) / 16;
    a.nq = std::max(a.nq, 2);
    a.qt = 1;
    a.groups = (qtiles + a.nq - 1) / a.nq;
  }
  // the caller picks n_split so that a split spans at most 1024 pages (the
  // kernels' page-table stage): max_prefix <= 1024 * 16 * n_split
  int split_tokens = (max_prefix + n_split - 1) / n_split;
  split_tokens = ((split_tokens + 63) / 64) * 64;
  if (split_tokens == 0) split_tokens = 64;
  const dim3 grid(a.groups, p.n_seqs * Hkv, n_split);
  const float scale = 1.0f / sqrtf((float)hd);
  if constexpr (sizeof(T) == 2) {
    if (a.mfma32) {
      // balanced splits (see balanced_split) when the fixed plan would take
      // more than one round of workgroups and the split can be worked out
      // on the device: the grid is kAttnSlots items, each sequence's splits
      // at most ms (the partial slots, and what the other sequences leave
      // of the slots).  Measured: 4 sequences of equal 2048-key prefixes
      // with 96 rows (fixed plan 3 splits, 288 workgroups) 74 vs 90 us; 16
      // ragged prefixes with 64 rows take the fixed plan's one round
      // (balanced: 83 vs 66 us)
      const int gx = a.groups * Hkv;
      const bool bal = split_rows != nullptr && p.n_seqs <= 64 &&
                       p.n_seqs * gx <= kAttnSlots && max_prefix <= 256 * 64 &&
                       (p.n_seqs == 1 ||          // even splits, no rounding
                        (long)p.n_seqs * gx * n_split > kAttnSlots);
      const int ms = bal ? std::max(1, std::min(max_split,
                                                kAttnSlots / gx - (p.n_seqs - 1)))
                         : n_split;
      const dim3 g32 = bal ? dim3(kAttnSlots) : grid;
      int* sr = bal ? split_rows : nullptr;
      const bool merge = bal || n_split > 1;
      const hipEvent_t kb32 = merge ? nullptr : eb;
#define SB_ATTN32(HD_, NW_)                                                    \
  if (hd == HD_ && a.nq == NW_) {                                             \
    hipExtLaunchKernelGGL(tree_attn32_kernel<HD_, NW_>, g32, dim3(NW_ * 64),  \
                          0, st, ka, kb32, 0, q, p, kv, H, Hkv, split_tokens, \
                          scale, o_part, ml, out, a.groups, ms, sr,           \
                          max_prefix);                                        \
    if (merge)                                                                \
      launch_attn_merge<T>(p, H, hd, ms, o_part, ml, out, st, eb, sr);        \
    return;                                                                   \
  }
    SB_ATTN32(128, 8) SB_ATTN32(128, 4) SB_ATTN32(64, 8) SB_ATTN32(64, 4)
#undef SB_ATTN32
    }
  }
  {
#define SB_ATTN(HD_, NQ_, QT_)                                                 \
  if (hd == HD_ && a.nq == NQ_ && a.qt == QT_) {                              \
    hipExtLaunchKernelGGL(tree_attn_kernel<T, HD_, NQ_, QT_>, grid,           \
                          dim3(NQ_ * 64), 0, st, ka, kb, 0, q, p, kv, H, Hkv, \
                          split_tokens, scale, o_part, ml, out, max_prefix);  \
    if (n_split > 1)                                                          \
      launch_attn_merge<T>(p, H, hd, n_split, o_part, ml, out, st, eb);       \
    return;                                                                   \
  }
    if constexpr (sizeof(T) == 2) SB_ATTN(128, 8, 2)
    SB_ATTN(128, 8, 1) SB_ATTN(128, 4, 1) SB_ATTN(128, 2, 1)
    if constexpr (sizeof(T) == 2) SB_ATTN(128, 1, 1)
    SB_ATTN(64, 8, 2) SB_ATTN(64, 8, 1) SB_ATTN(64, 4, 1)
    SB_ATTN(64, 2, 1) SB_ATTN(64, 1, 1)
#undef SB_ATTN
  }
}

template <typename T>
void launch_attn_merge(const CallPlan& p, int H, int hd, int n_split,
                       const float* o_part, const float* ml, T* out,
                       hipStream_t st, hipEvent_t stop,
                       const int* split_rows) {
  // every split's (m, l) and partial row is loaded at once (no dependent
  // chain); the template size is n_split rounded up, extra slots read as
  // empty splits
#define SB_MERGE(NS_)                                                          \
  if (n_split <= NS_) {                                                       \
    hipExtLaunchKernelGGL(attn_merge_kernel_t<NS_>, dim3(p.cap),              \
                          dim3(merge_threads<NS_>()), 0, st, nullptr, stop,   \
                          0, o_part, ml, p.n, p.cap, H, hd, n_split, out,     \
                          (int)sizeof(T), split_rows);                        \
    return;                                                                   \
  }
  SB_MERGE(2) SB_MERGE(4) SB_MERGE(8) SB_MERGE(16) SB_MERGE(32)
#undef SB_MERGE
}

int attn_qgroups(int rows_per_seq_cap, int G, int seq_heads, int es) {
  return attn_shape(rows_per_seq_cap, G, seq_heads, es).groups;
}

// The 32x32 kernel: one round of kAttnSlots workgroups.  Every split adds a
// full fp32 partial of its rows (written, then read by the merge), which at
// 16 sequences x 64 rows is 16.8 MB per split: 2 splits (one round) measured
// 66 us against 84 us for 4 splits (two rounds) at 16 prefixes of 512-2000
// keys; a 128-row tree drafting block at the same shape 67 vs 78 us.  The
// 16-row kernel: two rounds (its workgroups are smaller; at one sequence of
// 60 nodes the splits stay at 128 keys or more, see the caller).
int attn_workgroup_target(int rows_per_seq_cap, int G, int seq_heads, int es) {
  return attn_shape(rows_per_seq_cap, G, seq_heads, es).mfma32
             ? kAttnSlots
             : 2 * kAttnSlots;
}

template void launch_tree_attn<float>(const float*, const CallPlan&,
                                      const KVView&, int, int, int, int, int,
                                      int, float*, float*, float*, int, int*,
                                      hipStream_t);
template void launch_tree_attn<bf16_t>(const bf16_t*, const CallPlan&,
                                       const KVView&, int, int, int, int, int,
                                       int, float*, float*, bf16_t*, int, int*,
                                       hipStream_t);

}  // namespace sb
