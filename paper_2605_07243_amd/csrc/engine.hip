// C-ABI entry points: argument validation, workspace layout and the launch
// sequence of each call.  All device work is enqueued on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "specblock.h"

using namespace sb;

namespace {

constexpr size_t kAlign = 256;
constexpr int kVocabRec10 = 2 * SB_TOPK + 3;
// row counts captured for profiled GEMM launches (one int each); launches
// past the last slot are credited at their row capacity
constexpr int kProfSlots = 32768;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int ceil_div(int a, int b) { return (a + b - 1) / b; }

struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <typename P>
  P* take(size_t bytes) {
    P* p = base ? reinterpret_cast<P*>(base + off) : nullptr;
    off = align_up(off + bytes);
    return p;
  }
};

struct Dims {
  int S, d, H, Hkv, hd, F, V, Vd, L, LD, qkv_n, es;
  int K, M, B_max, budget, row_cap, rw, bw, vis_words, R_cap, chunk;
  int tpages, dpages, n_chunks, n_chunks_d, n_chunks_f, n_split;
  int adapt_cap;
  size_t part_elems;
};

Dims derive(const sb_config& c) {
  Dims D{};
  D.S = c.max_seqs;
  D.d = c.target.d_model;
  D.H = c.target.n_heads;
  D.Hkv = c.target.n_kv_heads;
  D.hd = c.target.head_dim;
  D.F = c.target.d_ff;
  D.V = c.target.vocab;
  D.Vd = c.draft_vocab > 0 ? c.draft_vocab : c.target.vocab;
  D.L = c.target.n_layers;
  D.LD = c.drafter_layers;
  D.qkv_n = (D.H + 2 * D.Hkv) * D.hd;
  D.es = c.dtype == SB_BF16 ? 2 : 4;
  D.K = c.K;
  D.M = c.M;
  D.B_max = c.B_max;
  D.budget = c.budget;
  D.row_cap = c.K + (c.M - 1) * c.B_max * c.K;
  D.rw = ceil_div(D.row_cap, 32);
  D.bw = ceil_div(D.budget, 32);
  D.chunk = c.prefill_chunk;
  D.vis_words = ceil_div(std::max(std::max(D.budget, D.row_cap), D.chunk), 32);
  D.R_cap = std::max(std::max(D.S * D.budget, D.S * D.B_max * D.K),
                     std::max(D.chunk, D.S));
  D.tpages = ceil_div(std::max(D.budget, D.chunk), 16);
  D.dpages = ceil_div(std::max(D.row_cap, D.chunk), 16);
  // record slots per row for the vocabulary reductions: up to 64 chunks,
  // and always enough for chunks of at most kVocabChunkMax logits
  const int min_v = (D.V + kVocabChunkMax - 1) / kVocabChunkMax;
  const int min_vd = (D.Vd + kVocabChunkMax - 1) / kVocabChunkMax;
  D.n_chunks = std::max({1, std::min(64, D.V / 2048), min_v});
  D.n_chunks_d = std::max({1, std::min(64, D.Vd / 2048), min_vd});
  D.adapt_cap = c.adapt_cap;
  // column tiles of the LM heads' fused reduction (at most one per 128
  // vocabulary ids)
  D.n_chunks_f = (std::max(D.V, D.Vd) + 127) / 128;
  D.n_split = 32;
  // partial-sum buffer: the largest ks * N over the projections
  size_t mx = 0;
  auto upd = [&](int N, int Kd) {
    mx = std::max(mx, (size_t)gemm_ksplit(N, Kd, D.es) * N);
  };
  upd(D.qkv_n, D.d);
  upd(D.d, D.H * D.hd);
  upd(2 * D.F, D.d);
  upd(D.d, D.F);
  upd(D.d, 3 * D.d);
  upd(D.d, 2 * D.d);
  upd(D.d, D.d);
  D.part_elems = mx * D.R_cap;
  return D;
}

}  // namespace

struct AdaptBufs {
  void* A;        // [adapt_cap][d] elem: LM-head operands
  float* Z;       // [adapt_cap][Vd] training-head logits, then gradients
  float* Z0;      // [adapt_cap][Vd] pre-deployment-head logits
  float* part;    // vocabulary chunk records of Z (top-10)
  float* part0;   // vocabulary chunk records of Z0 (top-1)
  float* psi;     // [adapt_cap][15]
  float* ds;      // [adapt_cap][4] rank-head score gradients
  float* loss;    // [adapt_cap]
  int* n;         // positions in this update
};

struct sb_ctx {
  sb_config cfg{};
  Dims D{};
  std::string err;
  bool bound = false;
  sb_target_weights tw{};
  std::vector<sb_layer_weights> tl;
  sb_drafter_weights dw{};
  std::vector<sb_layer_weights> dl;
  // workspace
  float* x = nullptr;
  void* A = nullptr;
  void* A2 = nullptr;   // SwiGLU output (down-projection operand)
  float* P = nullptr;
  void* q = nullptr;
  float* o_part = nullptr;
  float* ml = nullptr;
  int* split_rows = nullptr;     // [R] attention splits of each row's sequence
  float* logits = nullptr;
  float2* node_stats = nullptr;  // [S][budget][tiles] softmax stats of z / T
  float* row_lse = nullptr;      // [S][row_cap] drafter rows' log-sum-exp
  AdaptBufs ad{};                // head-update workspace
  float* vpart = nullptr;
  float* cond_buf = nullptr;
  float* taps_pf = nullptr;
  int* taps_idx = nullptr;
  int* n_aux = nullptr;
  int* one = nullptr;
  int* root_arg = nullptr;
  int* blk_row0 = nullptr;
  int* blk_nst = nullptr;
  int* prof_rows = nullptr;      // [kProfSlots] rows of profiled GEMM launches
  // Eq. 2 split (bf16): vq[k] = W_f3 norm_q(q_{k+1}), cached per bind
  float* vq = nullptr;           // [K][d]
  int* vq_n = nullptr;           // [1] = K on the device
  bool vq_ready = false;
  CommitInfo ci{};
  CallPlan plan{};
  CallPlan fb{};
  void* tseg_k = nullptr;
  void* tseg_v = nullptr;
  void* dseg_k = nullptr;
  void* dseg_v = nullptr;
  int* zero = nullptr;
  // debug status word: bits of the range checks on caller-supplied indices
  // (page-table entries, token ids), raised by the kernels while debug is
  // set; read and cleared by sb_device_check
  int* dev_status = nullptr;
  bool debug = false;
  bool status_live = false;   // cleared by sb_set_debug since the last bind
  int* dbg() const { return debug ? dev_status : nullptr; }
  // running upper bound of every sequence's T (0: unknown)
  int T_bound = 0;
  // forced drafter-row buckets [max_seqs][row_cap] (NULL: rank-head argmax)
  const int* bucket_in = nullptr;
  // kernel timing
  struct ProfRec {
    int cls;
    hipEvent_t a, b;
    double bytes, flops;
    // projection GEMMs: group, row-count slot (-1: none), row capacity and
    // the per-launch / per-row algorithmic counts
    int group = -1, slot = -1, m_cap = 0;
    double w_bytes = 0, in_row = 0, out_row = 0, flops_row = 0;
  };
  bool prof = false;
  int prof_group = SB_GEMM_TARGET;   // group of the projections being run
  int prof_slots_used = 0;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  std::vector<ProfRec> recs;
  ~sb_ctx() {
    for (hipEvent_t e : ev_pool) (void)hipEventDestroy(e);
  }
};

static thread_local std::string g_create_err;

static int fail(sb_ctx* c, int code, const std::string& msg) {
  if (c)
    c->err = msg;
  else
    g_create_err = msg;
  return code;
}

static size_t layout(const Dims& D, void* base, sb_ctx* c) {
  Carver cv(base);
  const size_t R = D.R_cap;
  const int es = D.es;
  const int widest = std::max(std::max(3 * D.d, D.F), std::max(D.H * D.hd, 2 * D.d));
  float* x = cv.take<float>(R * D.d * 4);
  void* A = cv.take<char>(R * widest * es);
  void* A2 = cv.take<char>(R * D.F * es);
  float* P = cv.take<float>(D.part_elems * 4);
  void* q = cv.take<char>(R * D.H * D.hd * es);
  float* o_part = cv.take<float>((size_t)D.n_split * R * D.H * D.hd * 4);
  float* ml = cv.take<float>((size_t)D.n_split * R * D.H * 2 * 4);
  int* split_rows = cv.take<int>(R * 4);
  float* logits = cv.take<float>(R * D.V * 4);
  float* row_lse = cv.take<float>((size_t)D.S * D.row_cap * 4);
  // head-update region (its own buffers: the update may run on another
  // stream while inference uses the ones above)
  const size_t ac = (size_t)D.adapt_cap;
  void* ad_A = cv.take<char>(ac * D.d * es);
  float* ad_Z = cv.take<float>(ac * D.Vd * 4);
  float* ad_Z0 = cv.take<float>(ac * D.Vd * 4);
  float* ad_part = cv.take<float>(ac * D.n_chunks_d * kVocabRec10 * 4);
  float* ad_part0 = cv.take<float>(ac * D.n_chunks_d * 5 * 4);
  float* ad_psi = cv.take<float>(ac * SB_PSI_DIM * 4);
  float* ad_ds = cv.take<float>(ac * 4 * 4);
  float* ad_loss = cv.take<float>(ac * 4);
  int* ad_n = cv.take<int>(4);
  float2* node_stats = cv.take<float2>((size_t)D.S * D.budget *
                                       sample_tiles(D.V) * 8);
  float* vpart = cv.take<float>(R * std::max(D.n_chunks, D.n_chunks_f) *
                                 kVocabRec10 * 4);
  float* cond_buf = cv.take<float>(R * D.d * 4);
  float* taps_pf = cv.take<float>((size_t)(D.chunk + 1) * 3 * D.d * 4);
  int* taps_idx = cv.take<int>(R * 4);
  int* n_aux = cv.take<int>(4);
  int* one = cv.take<int>(4);
  int* root_arg = cv.take<int>(4);
  int* zero = cv.take<int>(4);
  int* dev_status = cv.take<int>(4);
  int* blk_row0 = cv.take<int>(D.S * 4);
  int* blk_nst = cv.take<int>(D.S * 4);
  int* prof_rows = cv.take<int>((size_t)kProfSlots * 4);
  float* vq = cv.take<float>((size_t)D.K * D.d * 4);
  int* vq_n = cv.take<int>(4);
  CommitInfo ci{cv.take<int>(D.S * 4), cv.take<int>(D.S * 4),
                cv.take<int>(D.S * 4), cv.take<int>(D.S * 4)};
  auto make_plan = [&](int cap) {
    CallPlan p{};
    p.n = cv.take<int>(4);
    p.seq = cv.take<int>(cap * 4);
    p.slot = cv.take<int>(cap * 4);
    p.pos = cv.take<int>(cap * 4);
    p.token = cv.take<int>(cap * 4);
    p.vis = cv.take<uint32_t>((size_t)cap * D.vis_words * 4);
    p.k = cv.take<int>(cap * 4);
    p.pred = cv.take<int>(cap * 4);
    p.cond = cv.take<int>(cap * 4);
    p.seq_off = cv.take<int>((D.S + 1) * 4);
    p.prefix_len = cv.take<int>(D.S * 4);
    p.seg_len = cv.take<int>(D.S * 4);
    p.out_row = cv.take<int>(cap * 4);
    p.kv_dst = cv.take<int>(cap * 4);
    p.cap = cap;
    p.vis_words = D.vis_words;
    p.n_seqs = D.S;
    return p;
  };
  CallPlan plan = make_plan(D.R_cap);
  CallPlan fb = make_plan(D.S);
  const size_t page = (size_t)D.Hkv * 16 * D.hd * es;
  void* tseg_k = cv.take<char>((size_t)D.L * D.S * D.tpages * page);
  void* tseg_v = cv.take<char>((size_t)D.L * D.S * D.tpages * page);
  void* dseg_k = cv.take<char>((size_t)D.LD * D.S * D.dpages * page);
  void* dseg_v = cv.take<char>((size_t)D.LD * D.S * D.dpages * page);
  if (c) {
    c->x = x;
    c->A = A;
    c->A2 = A2;
    c->P = P;
    c->q = q;
    c->o_part = o_part;
    c->ml = ml;
    c->split_rows = split_rows;
    c->logits = logits;
    c->node_stats = node_stats;
    c->row_lse = row_lse;
    c->ad = AdaptBufs{ad_A, ad_Z, ad_Z0, ad_part, ad_part0, ad_psi, ad_ds,
                      ad_loss, ad_n};
    c->vpart = vpart;
    c->cond_buf = cond_buf;
    c->taps_pf = taps_pf;
    c->taps_idx = taps_idx;
    c->n_aux = n_aux;
    c->one = one;
    c->root_arg = root_arg;
    c->zero = zero;
    c->dev_status = dev_status;
    c->blk_row0 = blk_row0;
    c->blk_nst = blk_nst;
    c->prof_rows = prof_rows;
    c->vq = vq;
    c->vq_n = vq_n;
    c->ci = ci;
    c->plan = plan;
    c->fb = fb;
    c->tseg_k = tseg_k;
    c->tseg_v = tseg_v;
    c->dseg_k = dseg_k;
    c->dseg_v = dseg_v;
  }
  return cv.off;
}

static int validate_cfg(const sb_config* c, std::string& msg) {
  if (!c) {
    msg = "cfg is NULL";
    return SB_EINVAL;
  }
  if (c->dtype != SB_F32 && c->dtype != SB_BF16) {
    msg = "dtype must be SB_F32 or SB_BF16";
    return SB_EDTYPE;
  }
  const sb_model_dims& t = c->target;
  if (t.n_layers < 1 || t.d_model < 32 || t.n_heads < 1 || t.n_kv_heads < 1 ||
      t.head_dim < 1 || t.d_ff < 32 || t.vocab < SB_TOPK) {
    msg = "model dimensions out of range";
    return SB_ESHAPE;
  }
  if (t.head_dim != 64 && t.head_dim != 128) {
    msg = "head_dim must be 64 or 128";
    return SB_ESHAPE;
  }
  if (t.n_heads % t.n_kv_heads || t.n_heads > 64) {
    msg = "n_heads must be a multiple of n_kv_heads and <= 64";
    return SB_ESHAPE;
  }
  if (t.d_model % 32 || t.d_ff % 32 || t.d_model > 8192 ||
      (t.n_heads * t.head_dim) % 32) {
    msg = "d_model and d_ff must be multiples of 32 (d_model <= 8192)";
    return SB_ESHAPE;
  }
  if (t.vocab % 16 || ((t.n_heads + 2 * t.n_kv_heads) * t.head_dim) % 16) {
    msg = "vocab and the QKV width must be multiples of 16";
    return SB_ESHAPE;
  }
  if (c->adapt_cap < 0 || c->adapt_cap > 64) {
    msg = "adapt_cap must be in 0..64";
    return SB_EINVAL;
  }
  if (c->adapt_cap > 0) {
    const int vd = c->draft_vocab > 0 ? c->draft_vocab : t.vocab;
    const int cw = sb::adapt_column_width(c->dtype == SB_BF16 ? 2 : 4);
    if (vd % sb::adapt_stripe_rows() || t.d_model % cw) {
      msg = "head updates need the drafter vocabulary % 64 == 0 and d_model % " +
            std::to_string(cw) + " == 0";
      return SB_ESHAPE;
    }
  }
  if (c->draft_vocab != 0 &&
      (c->draft_vocab < SB_TOPK || c->draft_vocab > t.vocab ||
       c->draft_vocab % 16)) {
    msg = "draft_vocab must be 0 or a multiple of 16 in 10..vocab";
    return SB_ESHAPE;
  }
  {
    const int es = c->dtype == SB_BF16 ? 2 : 4;
    const int d = t.d_model, F = t.d_ff, hq = t.n_heads * t.head_dim;
    const int qkv = (t.n_heads + 2 * t.n_kv_heads) * t.head_dim;
    const int vd = c->draft_vocab > 0 ? c->draft_vocab : t.vocab;
    const int shapes[][2] = {{qkv, d},   {d, hq},    {2 * F, d}, {d, F},
                             {d, 3 * d}, {d, 2 * d}, {t.vocab, d}, {vd, d}};
    for (const auto& nk : shapes)
      if (!sb::gemm_shape_ok(nk[0], nk[1], es) || (es == 2 && F % 16)) {
        msg = es == 2 ? "bf16 projections need output widths % 32 == 0 and "
                        "input widths % 128 == 0 (d_model, d_ff, heads*head_dim)"
                      : "projection widths must be multiples of 16 / 32";
        return SB_ESHAPE;
      }
  }
  if (!(t.rope_theta > 0.f) || !(t.norm_eps > 0.f)) {
    msg = "rope_theta and norm_eps must be positive";
    return SB_EINVAL;
  }
  if (c->drafter_layers < 1) {
    msg = "drafter_layers must be >= 1";
    return SB_ESHAPE;
  }
  for (int i = 0; i < 3; ++i)
    if (c->tap_layers[i] < 0 || c->tap_layers[i] >= t.n_layers) {
      msg = "tap layer out of range";
      return SB_ESHAPE;
    }
  if (c->K < 1 || c->M < 1 || c->B_max < 1 || c->B_max > 64) {
    msg = "need K >= 1, M >= 1, 1 <= B_max <= 64";
    return SB_EINVAL;
  }
  if (c->budget < 1 || c->budget > 512) {
    msg = "budget must be in 1..512";
    return SB_EBUDGET;
  }
  const int row_cap = c->K + (c->M - 1) * c->B_max * c->K;
  if (row_cap > 512 || c->M * c->K > 512) {
    msg = "K + (M-1) B_max K must be <= 512";
    return SB_EBUDGET;
  }
  for (int i = 0; i < 4; ++i)
    if (c->branch_map[i] < 0 || c->branch_map[i] > SB_TOPK) {
      msg = "branch_map entries must be in 0..10";
      return SB_EINVAL;
    }
  if (c->max_seqs < 1 || c->max_seqs > SB_MAX_SEQS) {
    msg = "max_seqs must be in 1..64";
    return SB_EINVAL;
  }
  if (c->page_size != 16) {
    msg = "page_size must be 16";
    return SB_ESHAPE;
  }
  if (c->max_pages < 1 || c->max_pages > 16384) {
    msg = "max_pages must be in 1..16384";
    return SB_EINVAL;
  }
  if (c->prefill_chunk < 16 || c->prefill_chunk % 16 || c->prefill_chunk > 512) {
    msg = "prefill_chunk must be a multiple of 16 in 16..512";
    return SB_EINVAL;
  }
  return SB_OK;
}

extern "C" {

int32_t sb_row_capacity(const sb_config* cfg) {
  std::string m;
  if (validate_cfg(cfg, m) != SB_OK) return 0;
  return cfg->K + (cfg->M - 1) * cfg->B_max * cfg->K;
}

size_t sb_workspace_bytes(const sb_config* cfg) {
  std::string m;
  if (validate_cfg(cfg, m) != SB_OK) return 0;
  return layout(derive(*cfg), nullptr, nullptr);
}

int sb_create(const sb_config* cfg, sb_ctx** out) {
  if (!out) return fail(nullptr, SB_EINVAL, "out is NULL");
  *out = nullptr;
  std::string m;
  const int rc = validate_cfg(cfg, m);
  if (rc != SB_OK) return fail(nullptr, rc, m);
  sb_ctx* c = new sb_ctx();
  c->cfg = *cfg;
  c->D = derive(*cfg);
  *out = c;
  return SB_OK;
}

void sb_destroy(sb_ctx* ctx) { delete ctx; }

const char* sb_last_error(const sb_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_create_err.c_str();
}

static bool bad_ptr(const void* p, size_t align) {
  return p == nullptr || (reinterpret_cast<uintptr_t>(p) % align) != 0;
}

static int check_layer(sb_ctx* c, const sb_layer_weights& l, bool drafter) {
  if (bad_ptr(l.attn_norm, 4) || bad_ptr(l.mlp_norm, 4) || bad_ptr(l.w_qkv, 16) ||
      bad_ptr(l.w_o, 16) || bad_ptr(l.w_gate_up, 16) || bad_ptr(l.w_down, 16))
    return fail(c, SB_EINVAL, "layer weight pointer NULL or misaligned");
  if (drafter && bad_ptr(l.w_shift, 16))
    return fail(c, SB_EINVAL, "drafter layer needs w_shift");
  return SB_OK;
}

int sb_pack_weight(const void* src, void* dst, int32_t rows, int32_t cols,
                   int32_t dtype, int32_t gate_up, void* stream) {
  auto err = [](int code, const char* m) {
    g_create_err = m;
    return code;
  };
  if (dtype != SB_F32 && dtype != SB_BF16)
    return err(SB_EDTYPE, "sb_pack_weight: dtype must be SB_F32 or SB_BF16");
  if (rows < 1 || cols < 1)
    return err(SB_EINVAL, "sb_pack_weight: rows and cols must be >= 1");
  const size_t bytes = (size_t)rows * cols * (dtype == SB_BF16 ? 2 : 4);
  if (bad_ptr(src, 16) || bad_ptr(dst, 16))
    return err(SB_EINVAL, "sb_pack_weight: src/dst NULL or not 16-byte aligned");
  const uintptr_t a = reinterpret_cast<uintptr_t>(src);
  const uintptr_t b = reinterpret_cast<uintptr_t>(dst);
  if (a < b + bytes && b < a + bytes)
    return err(SB_EINVAL, "sb_pack_weight: src and dst overlap");
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (dtype == SB_F32) {
    if (hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, st) != hipSuccess)
      return err(SB_EHIP, "sb_pack_weight: hipMemcpyAsync failed");
    return SB_OK;
  }
  if (rows % 32 || cols % 64)
    return err(SB_ESHAPE, "sb_pack_weight: bf16 needs rows % 32 == 0 and cols % 64 == 0");
  (void)hipGetLastError();
  sb::launch_pack_weight(static_cast<const sb::bf16_t*>(src),
                         static_cast<sb::bf16_t*>(dst), rows, cols, gate_up != 0,
                         st);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    g_create_err = std::string("sb_pack_weight: ") + hipGetErrorString(e);
    return SB_EHIP;
  }
  return SB_OK;
}

int sb_bind(sb_ctx* c, const sb_target_weights* tw,
            const sb_drafter_weights* dw, void* ws, size_t ws_bytes) {
  if (!c) return SB_EINVAL;
  if (!tw || !dw || !tw->layers || !dw->layers)
    return fail(c, SB_EINVAL, "weight tables must not be NULL");
  if (bad_ptr(tw->embed, 16) || bad_ptr(tw->final_norm, 4) ||
      bad_ptr(tw->lm_head, 16))
    return fail(c, SB_EINVAL, "target weight pointer NULL or misaligned");
  if (bad_ptr(dw->w_cond, 16) || bad_ptr(dw->norm_c, 4) ||
      bad_ptr(dw->norm_e, 4) || bad_ptr(dw->norm_q, 4) ||
      bad_ptr(dw->pos_query, 16) || bad_ptr(dw->w_fuse, 16) ||
      bad_ptr(dw->final_norm, 4) || bad_ptr(dw->lm_head, 16) ||
      bad_ptr(dw->rank_w, 4) || bad_ptr(dw->rank_b, 4))
    return fail(c, SB_EINVAL, "drafter weight pointer NULL or misaligned");
  if (dw->d2t == nullptr && c->D.Vd != c->D.V)
    return fail(c, SB_EINVAL, "a reduced drafter vocabulary needs d2t");
  if (dw->d2t != nullptr) {
    if (bad_ptr(dw->d2t, 4)) return fail(c, SB_EINVAL, "d2t misaligned");
    // setup-time check of the id map (it indexes the embedding later)
    std::vector<int32_t> m(c->D.Vd);
    if (hipMemcpy(m.data(), dw->d2t, m.size() * sizeof(int32_t),
                  hipMemcpyDefault) != hipSuccess)
      return fail(c, SB_EHIP, "d2t: copy to host failed");
    for (int i = 0; i < c->D.Vd; ++i)
      if (m[i] < 0 || m[i] >= c->D.V || (i > 0 && m[i] <= m[i - 1]))
        return fail(c, SB_EINVAL,
                    "d2t must be strictly increasing target ids in [0, vocab)");
  }
  for (int i = 0; i < c->D.L; ++i) {
    const int rc = check_layer(c, tw->layers[i], false);
    if (rc) return rc;
  }
  for (int i = 0; i < c->D.LD; ++i) {
    const int rc = check_layer(c, dw->layers[i], true);
    if (rc) return rc;
  }
  const size_t need = layout(c->D, nullptr, nullptr);
  if (bad_ptr(ws, kAlign)) return fail(c, SB_EINVAL, "workspace NULL or not 256-byte aligned");
  if (ws_bytes < need)
    return fail(c, SB_EBUDGET, "workspace too small: need " + std::to_string(need));
  c->tw = *tw;
  c->tl.assign(tw->layers, tw->layers + c->D.L);
  c->tw.layers = c->tl.data();
  c->dw = *dw;
  c->dl.assign(dw->layers, dw->layers + c->D.LD);
  c->dw.layers = c->dl.data();
  layout(c->D, ws, c);
  c->status_live = false;
  c->debug = false;
  c->vq_ready = false;
  c->bound = true;
  return SB_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// forward passes

namespace {

hipStream_t S_(void* s) { return static_cast<hipStream_t>(s); }

int hip_check(sb_ctx* c, const char* where) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return fail(c, SB_EHIP, std::string(where) + ": " + hipGetErrorString(e));
  return SB_OK;
}

hipEvent_t next_event(sb_ctx* c) {
  if (c->ev_used == c->ev_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    c->ev_pool.push_back(e);
  }
  return c->ev_pool[c->ev_used++];
}

// Times the launches of one class inside its scope.  The projection GEMM
// (one launch per scope) and the tree attention (kernel + merge) take events
// attached to their dispatches, which mark the kernels' own start and end;
// other classes record stream events around their launches.  A GEMM scope
// also copies the launch's live row count (*n, read on the device) into a
// profiler slot after the launch, so that its algorithmic bytes and flops
// are credited for the rows it actually processed (none when it had none).
struct ProfScope {
  sb_ctx* c;
  hipStream_t st;
  int cls;
  double bytes, flops;
  hipEvent_t a = nullptr, b = nullptr;
  const int* rows = nullptr;
  sb_ctx::ProfRec g{};
  ProfScope(sb_ctx* c_, hipStream_t st_, int cls_, double bytes_ = 0,
            double flops_ = 0)
      : c(c_), st(st_), cls(cls_), bytes(bytes_), flops(flops_) {
    if (!c->prof || (a = next_event(c)) == nullptr) return;
    if (cls == SB_PROF_GEMM || cls == SB_PROF_ATTN) {
      if ((b = next_event(c)) == nullptr) a = nullptr;
      else if (cls == SB_PROF_GEMM) gemm_time_next_launch(a, b);
      else attn_time_next_launch(a, b);
    } else {
      (void)hipEventRecord(a, st);
    }
  }
  // GEMM launch shape: N x K weights of `es` bytes per element, `n` live
  // rows of capacity m_cap, out_es bytes per output element (4: fp32 rows
  // of N; the SwiGLU projection writes N / 2 bf16 values per row)
  // (out_row >= 0: bytes written per row, e.g. the vocabulary records of
  // the fused LM heads)
  ProfScope(sb_ctx* c_, hipStream_t st_, const int* n, int m_cap, int N,
            int K, double es, bool swiglu, int group, double out_row = -1.0)
      : ProfScope(c_, st_, SB_PROF_GEMM,
                  (double)N * K * es + (double)m_cap * K * es +
                      (double)m_cap * (out_row >= 0.0 ? out_row
                                       : swiglu ? N / 2 * es : N * 4.0),
                  2.0 * m_cap * N * K) {
    if (!a) return;
    rows = n;
    g.group = group;
    g.m_cap = m_cap;
    g.w_bytes = (double)N * K * es;
    g.in_row = (double)K * es;
    g.out_row = out_row >= 0.0 ? out_row : swiglu ? N / 2 * es : N * 4.0;
    g.flops_row = 2.0 * N * K;
  }
  ~ProfScope() {
    if (!a) return;
    if (cls == SB_PROF_GEMM) {
      if (gemm_time_pending()) {   // no launch took the events
        gemm_time_next_launch(nullptr, nullptr);
        return;
      }
    } else if (cls == SB_PROF_ATTN) {
      if (attn_time_pending()) {
        attn_time_next_launch(nullptr, nullptr);
        return;
      }
    } else {
      if ((b = next_event(c)) == nullptr) return;
      (void)hipEventRecord(b, st);
    }
    sb_ctx::ProfRec r = g;
    r.cls = cls;
    r.a = a;
    r.b = b;
    r.bytes = bytes;
    r.flops = flops;
    if (rows != nullptr && c->prof_slots_used < kProfSlots) {
      r.slot = c->prof_slots_used++;
      launch_copy_int(c->prof_rows + r.slot, rows, st);
    }
    c->recs.push_back(r);
  }
};

template <typename T>
int gemm(sb_ctx* c, const void* X, int ldx, const void* W, int N, int K,
         const int* n, int m_cap, hipStream_t st) {
  const int ks = 0;   // the shape's own split
  ProfScope ps(c, st, n, m_cap, N, K, sizeof(T), false, c->prof_group);
  return launch_gemm_xwt<T>(static_cast<const T*>(X), ldx,
                            static_cast<const T*>(W), N, K, c->P,
                            (size_t)c->D.R_cap * N, n, m_cap, ks, st);
}

// Gate/up projection + SwiGLU into out: bf16 in the GEMM epilogue (the
// weight carries the gate/up interleave), f32 through partial sums and a
// separate SwiGLU pass.
template <typename T>
void gate_up_swiglu(sb_ctx* c, const void* X, const void* W, const int* n,
                    int m_cap, T* out, hipStream_t st) {
  const Dims& D = c->D;
  if constexpr (sizeof(T) == 2) {
    ProfScope ps(c, st, n, m_cap, 2 * D.F, D.d, sizeof(T), true,
                 SB_GEMM_SWIGLU);
    launch_gemm_swiglu(static_cast<const bf16_t*>(X), D.d,
                       static_cast<const bf16_t*>(W), D.F, D.d, out, n, m_cap,
                       st);
  } else {
    const int ks = gemm<T>(c, X, D.d, W, 2 * D.F, D.d, n, m_cap, st);
    launch_swiglu<T>(c->P, ks, (size_t)D.R_cap * 2 * D.F, n, m_cap, D.F, out,
                     st);
  }
}

struct Prefix {
  const sb_kv* kv;
  void* seg_k;   // all layers
  void* seg_v;
  int seg_pages;
};

// Decoder layer body after the attention-norm operand is in A: QKV + RoPE,
// tree attention, O + residual, MLP + residual.  next_g: gain of the norm
// that follows (written into A), or nullptr.
template <typename T>
void layer_body(sb_ctx* c, const sb_layer_weights& lw, int layer,
                const CallPlan& p, const Prefix& pf, int rows_per_seq,
                const float* next_g, float* taps, int tap_mask,
                hipStream_t st) {
  const Dims& D = c->D;
  const float eps = c->cfg.target.norm_eps;
  const int R = p.cap;
  const size_t page = (size_t)D.Hkv * 16 * D.hd;
  T* A = static_cast<T*>(c->A);
  int ks = gemm<T>(c, A, D.d, lw.w_qkv, D.qkv_n, D.d, p.n, R, st);
  T* segk = static_cast<T*>(pf.seg_k) + (size_t)layer * D.S * pf.seg_pages * page;
  T* segv = static_cast<T*>(pf.seg_v) + (size_t)layer * D.S * pf.seg_pages * page;
  launch_qkv_post<T>(c->P, ks, (size_t)D.R_cap * D.qkv_n, p, D.H, D.Hkv, D.hd,
                     c->cfg.target.rope_theta, static_cast<T*>(c->q), segk,
                     segv, pf.seg_pages, st);
  KVView kv{};
  kv.k = static_cast<const T*>(pf.kv->k) + (size_t)layer * pf.kv->n_pages * page;
  kv.v = static_cast<const T*>(pf.kv->v) + (size_t)layer * pf.kv->n_pages * page;
  kv.page_table = pf.kv->page_table;
  kv.max_pages = c->cfg.max_pages;
  kv.n_pages = pf.kv->n_pages;
  kv.err = c->dbg();
  kv.seg_k = segk;
  kv.seg_v = segv;
  kv.seg_pages = pf.seg_pages;
  // prefix length bound: the host-side running bound when known, else the
  // page-table capacity
  const int cap_tokens = c->cfg.max_pages * 16;
  const int max_prefix = c->T_bound > 0 ? std::min(c->T_bound, cap_tokens)
                                        : cap_tokens;
  const int G = D.H / D.Hkv, seq_heads = p.n_seqs * D.Hkv;
  const int groups = attn_qgroups(rows_per_seq, G, seq_heads, D.es) * seq_heads;
  // enough workgroups for the chip, splits of at least 128 keys (the
  // kernel keeps four 32-key tiles in flight; shorter splits measured slower)
  int n_split = std::max(
      1, ceil_div(attn_workgroup_target(rows_per_seq, G, seq_heads, D.es), groups));
  n_split = std::min(n_split, std::max(1, max_prefix / 128));
  // a split spans at most 1024 pages of 16 keys
  n_split = std::max(n_split, ceil_div(max_prefix, 1024 * 16));
  n_split = std::min(n_split, D.n_split);
  {
    ProfScope ps(c, st, SB_PROF_ATTN);
    launch_tree_attn<T>(static_cast<const T*>(c->q), p, kv, rows_per_seq, D.H,
                        D.Hkv, D.hd, n_split, max_prefix, c->o_part, c->ml, A,
                        D.n_split, c->split_rows, st);
  }
  ks = gemm<T>(c, A, D.H * D.hd, lw.w_o, D.d, D.H * D.hd, p.n, R, st);
  launch_residual<T>(c->x, c->P, ks, (size_t)D.R_cap * D.d, p.n, R, D.d, true,
                     lw.mlp_norm ? static_cast<const float*>(lw.mlp_norm) : nullptr,
                     eps, A, D.d, nullptr, 0, nullptr, st);
  T* A2 = static_cast<T*>(c->A2);
  gate_up_swiglu<T>(c, A, lw.w_gate_up, p.n, R, A2, st);
  ks = gemm<T>(c, A2, D.F, lw.w_down, D.d, D.F, p.n, R, st);
  launch_residual<T>(c->x, c->P, ks, (size_t)D.R_cap * D.d, p.n, R, D.d, true,
                     next_g, eps, A, D.d, taps, tap_mask, p.out_row, st);
}

// Target forward over the plan's rows.  Ends with rmsnorm(final) in A when
// lm_rows is true (the LM head is run by the caller).
template <typename T>
void target_forward(sb_ctx* c, const CallPlan& p, const Prefix& pf,
                    int rows_per_seq, float* taps, hipStream_t st) {
  const Dims& D = c->D;
  const float eps = c->cfg.target.norm_eps;
  c->prof_group = SB_GEMM_TARGET;
  launch_embed<T>(p, static_cast<const T*>(c->tw.embed), D.d, c->x, st);
  launch_rmsnorm<T>(c->x, p.n, p.cap, D.d,
                    static_cast<const float*>(c->tw.layers[0].attn_norm), eps,
                    static_cast<T*>(c->A), D.d, st);
  for (int l = 0; l < D.L; ++l) {
    const float* next_g = l + 1 < D.L
                              ? static_cast<const float*>(c->tw.layers[l + 1].attn_norm)
                              : static_cast<const float*>(c->tw.final_norm);
    int mask = 0;
    for (int j = 0; j < 3; ++j)
      if (c->cfg.tap_layers[j] == l) mask |= 1 << j;
    layer_body<T>(c, c->tw.layers[l], l, p, pf, rows_per_seq, next_g,
                  taps, mask, st);
  }
}

// Drafter forward over the plan's rows (Eq. 2, Eq. 3, decoder layers).
// cond_base: rows of conditions indexed by p.cond.  Leaves the final
// residual h^(L) in x and, when lm is true, rmsnorm(final) in A.
template <typename T>
void drafter_forward(sb_ctx* c, const CallPlan& p, const float* cond_base,
                     const Prefix& pf, int rows_per_seq, bool lm,
                     hipStream_t st) {
  const Dims& D = c->D;
  const float eps = c->cfg.target.norm_eps;
  const int R = p.cap;
  T* A = static_cast<T*>(c->A);
  c->prof_group = SB_GEMM_DRAFTER;
  // Eq. 2: h0_k = W_f1 n_c(c) + W_f2 n_e(e) + W_f3 n_q(q_k).  With bf16 the
  // packed W_fuse splits into its first 2d columns and its last d columns
  // (both contiguous packed matrices, the packing being K-block-major), and
  // the q_k part, which depends on the weights only, is computed once per
  // bind and added by the residual kernel: each call streams 2d x d of
  // W_fuse instead of 3d x d.
  const bool split = sizeof(T) == 2;
  if (split && !c->vq_ready) {
    launch_set_int(c->vq_n, D.K, st);
    launch_norm_rows<T>(static_cast<const T*>(c->dw.pos_query), D.K, D.d,
                        static_cast<const float*>(c->dw.norm_q), eps, A, st);
    const T* wf3 = static_cast<const T*>(c->dw.w_fuse) + (size_t)2 * D.d * D.d;
    const int kq = gemm<T>(c, A, D.d, wf3, D.d, D.d, c->vq_n, D.K, st);
    launch_residual<T>(c->vq, c->P, kq, (size_t)D.R_cap * D.d, c->vq_n, D.K,
                       D.d, false, nullptr, eps, A, D.d, nullptr, 0, nullptr,
                       st);
    c->vq_ready = true;
  }
  const int parts = split ? 2 : 3;
  launch_fuse_prep<T>(cond_base, p, static_cast<const T*>(c->tw.embed),
                      static_cast<const T*>(c->dw.pos_query),
                      static_cast<const float*>(c->dw.norm_c),
                      static_cast<const float*>(c->dw.norm_e),
                      static_cast<const float*>(c->dw.norm_q), eps, D.d, A,
                      parts, st);
  int ks = gemm<T>(c, A, parts * D.d, c->dw.w_fuse, D.d, parts * D.d, p.n, R,
                   st);
  launch_residual<T>(c->x, c->P, ks, (size_t)D.R_cap * D.d, p.n, R, D.d, false,
                     nullptr, eps, A, D.d, nullptr, 0, nullptr, st,
                     split ? c->vq : nullptr, split ? p.k : nullptr);
  for (int l = 0; l < D.LD; ++l) {
    const sb_layer_weights& lw = c->dw.layers[l];
    launch_shift_prep<T>(c->x, p, D.d, A, st);
    ks = gemm<T>(c, A, 2 * D.d, lw.w_shift, D.d, 2 * D.d, p.n, R, st);
    launch_residual<T>(c->x, c->P, ks, (size_t)D.R_cap * D.d, p.n, R, D.d,
                       false, static_cast<const float*>(lw.attn_norm), eps, A,
                       D.d, nullptr, 0, nullptr, st);
    const float* next_g = (l + 1 == D.LD && lm)
                              ? static_cast<const float*>(c->dw.final_norm)
                              : nullptr;
    layer_body<T>(c, lw, l, p, pf, rows_per_seq, next_g, nullptr, 0, st);
  }
}

// W_cond rows: cond_buf[i] = W_cond [taps of row idx[i]] for i < *n.
template <typename T>
void cond_rows(sb_ctx* c, const float* taps, const int* idx, const int* n,
               int cap, hipStream_t st) {
  const Dims& D = c->D;
  T* A = static_cast<T*>(c->A);
  c->prof_group = SB_GEMM_DRAFTER;
  launch_rows_to_elem<T>(taps, idx, n, cap, 3 * D.d, A, st);
  const int ks = gemm<T>(c, A, 3 * D.d, c->dw.w_cond, D.d, 3 * D.d, n, cap, st);
  launch_residual<T>(c->cond_buf, c->P, ks, (size_t)D.R_cap * D.d, n, cap, D.d,
                     false, nullptr, c->cfg.target.norm_eps, A, D.d, nullptr, 0,
                     nullptr, st);
}


// LM head: logits[i] = W_lm A[i] for the plan's rows (one K-chunk, written
// straight into the logits buffer).
template <typename T>
void lm_head(sb_ctx* c, const void* A, const void* W, int V, float* logits,
             const int* n, int cap, hipStream_t st) {
  const Dims& D = c->D;
  ProfScope ps(c, st, n, cap, V, D.d, sizeof(T), false, SB_GEMM_LM_HEAD);
  launch_gemm_xwt<T>(static_cast<const T*>(A), D.d, static_cast<const T*>(W),
                     V, D.d, logits, (size_t)cap * V, n, cap, 1, st);
}

// LM head with the vocabulary reduction.  bf16 greedy verification (top-1)
// runs it in the GEMM epilogue: chunk records straight from the
// accumulators, logits written only when the caller asked for them.  The
// drafter's top-10 (and f32) write the logits and reduce them in a second
// pass: a top-10 merge in the epilogue measured slower than that pass at
// the 8B shape (0.42 vs 0.40 ms per block).  Returns the chunk records per
// row in c->vpart.
template <typename T>
int lm_head_reduce(sb_ctx* c, const void* W, int V, float* logits_out,
                   const int* n, int cap, int topk, int max_chunks,
                   hipStream_t st) {
  const Dims& D = c->D;
  if (sizeof(T) == 2 && topk == 1) {
    const int nc = gemm_vocab_chunks(V, D.d, cap);
    const double out_row = (double)nc * (2 * topk + 3) * 4 +
                           (logits_out != nullptr ? (double)V * 4 : 0.0);
    ProfScope ps(c, st, n, cap, V, D.d, sizeof(T), false, SB_GEMM_LM_HEAD,
                 out_row);
    return launch_gemm_vocab(static_cast<const bf16_t*>(c->A), D.d,
                             static_cast<const bf16_t*>(W), V, D.d,
                             logits_out, n, cap, topk, c->vpart, st);
  } else {
    float* logits = logits_out ? logits_out : c->logits;
    lm_head<T>(c, c->A, W, V, logits, n, cap, st);
    ProfScope ps(c, st, SB_PROF_VOCAB);
    return launch_vocab_partial(logits, n, cap, V, max_chunks, topk, c->vpart,
                                st);
  }
}

TreeDims tree_dims(const sb_ctx* c, int n_seqs) {
  const Dims& D = c->D;
  return TreeDims{n_seqs, D.K,  D.M,  D.B_max, D.budget, D.bw,
                  D.row_cap, D.rw, D.d, D.V, c->dbg()};
}

template <typename T>
int draft_expand_impl(sb_ctx* c, int m, const sb_seqs* sq, const sb_kv* dkv,
                      sb_tree* t, sb_draft_out* o, hipStream_t st) {
  const Dims& D = c->D;
  const TreeDims td = tree_dims(c, sq->n_seqs);
  CallPlan p = c->plan;
  p.n_seqs = sq->n_seqs;
  p.cap = sq->n_seqs * (m == 1 ? D.K : D.B_max * D.K);   // rows this call
  const float* cond_base = t->h_last;
  if (m == 1) {
    launch_block1_reset(td, *t, sq->root, c->n_aux, st);
    cond_rows<T>(c, sq->cond_taps, nullptr, c->n_aux, D.S, st);
    cond_base = c->cond_buf;
  }
  launch_plan_block(td, m, *t, sq->T, p, c->blk_row0, c->blk_nst,
                    D.S * D.B_max * D.K, o->call_seq, o->call_row, o->n_call,
                    st);
  const Prefix pf{dkv, c->dseg_k, c->dseg_v, D.dpages};
  drafter_forward<T>(c, p, cond_base, pf, D.B_max * D.K, true, st);
  const int n_chunks = lm_head_reduce<T>(c, c->dw.lm_head, D.Vd, o->logits,
                                         p.n, p.cap, SB_TOPK, D.n_chunks_d,
                                         st);
  {
    ProfScope ps(c, st, SB_PROF_VOCAB);
    const DraftRowOut ro{o->topk_id, o->topk_logit, o->lse, o->psi,
                         o->bucket, o->branch, t->h_last, c->bucket_in,
                         c->dw.d2t, c->row_lse, D.Vd, D.row_cap};
    const int4 bmap = make_int4(c->cfg.branch_map[0], c->cfg.branch_map[1],
                                c->cfg.branch_map[2], c->cfg.branch_map[3]);
    launch_draft_finalize(c->vpart, n_chunks, p, c->x,
                          static_cast<const float*>(c->dw.rank_w),
                          static_cast<const float*>(c->dw.rank_b), D.d, bmap,
                          ro, st);
  }
  launch_attach(td, *t, *o, c->blk_row0, c->blk_nst, st);
  return hip_check(c, "sb_draft_block_expand");
}

template <typename T>
int verify_impl(sb_ctx* c, const sb_seqs* sq, const sb_tree* t,
                const sb_kv* tkv, sb_verify_out* out, hipStream_t st) {
  const Dims& D = c->D;
  const TreeDims td = tree_dims(c, sq->n_seqs);
  CallPlan p = c->plan;
  p.n_seqs = sq->n_seqs;
  p.cap = sq->n_seqs * D.budget;
  launch_plan_verify(td, *t, sq->T, p, st);
  const Prefix pf{tkv, c->tseg_k, c->tseg_v, D.tpages};
  target_forward<T>(c, p, pf, D.budget, out->taps, st);
  const int n_chunks = lm_head_reduce<T>(c, c->tw.lm_head, D.V, out->logits,
                                         p.n, p.cap, 1, D.n_chunks, st);
  {
    ProfScope ps(c, st, SB_PROF_VOCAB);
    launch_verify_finalize(c->vpart, n_chunks, p.n, p.cap, p.out_row,
                           out->argmax, st);
  }
  return hip_check(c, "sb_tree_verify");
}

template <typename T>
int commit_impl(sb_ctx* c, sb_seqs* sq, const sb_tree* t,
                const sb_verify_out* v, const sb_accept_out* acc,
                sb_kv* tkv, sb_kv* dkv, hipStream_t st) {
  const Dims& D = c->D;
  const TreeDims td = tree_dims(c, sq->n_seqs);
  launch_commit_plan(td, *t, *acc, sq->T, c->ci, c->fb, c->taps_idx, c->n_aux,
                     st);
  const KVPools tp{tkv->k, tkv->v, tkv->page_table, c->cfg.max_pages,
                   tkv->n_pages, c->tseg_k, c->tseg_v, D.tpages, c->dbg()};
  const KVPools dp{dkv->k, dkv->v, dkv->page_table, c->cfg.max_pages,
                   dkv->n_pages, c->dseg_k, c->dseg_v, D.dpages, c->dbg()};
  launch_commit_copy<T>(td, *t, *acc, c->ci, false, tp, D.S, D.L, D.Hkv, D.hd,
                        st);
  launch_commit_copy<T>(td, *t, *acc, c->ci, true, dp, D.S, D.LD, D.Hkv, D.hd,
                        st);
  // catch-up rows where the tree has no row continuing the accepted path
  // (usually none: its launches test the live count before loading)
  set_rows_likely_empty(true);
  cond_rows<T>(c, v->taps, c->taps_idx, c->n_aux, D.S, st);
  const Prefix pf{dkv, c->dseg_k, c->dseg_v, D.dpages};
  CallPlan fb = c->fb;
  fb.n_seqs = sq->n_seqs;
  fb.cap = sq->n_seqs;
  drafter_forward<T>(c, fb, c->cond_buf, pf, 1, false, st);
  set_rows_likely_empty(false);
  launch_seg_to_cache<T>(fb, dp, D.S, D.LD, D.Hkv, D.hd, st);
  launch_commit_state(td, *sq, *acc, c->ci, v->taps, st);
  if (c->T_bound > 0) c->T_bound += D.M * D.K + 1;
  return hip_check(c, "sb_commit");
}

template <typename T>
int prefill_impl(sb_ctx* c, const sb_seqs* sq, const int32_t* prompt, int ld,
                 const int32_t* lens, sb_kv* tkv, sb_kv* dkv, hipStream_t st) {
  const Dims& D = c->D;
  CallPlan p = c->plan;
  p.cap = D.chunk;
  const int S = D.S;
  launch_set_int(c->one, 1, st);
  launch_set_int(c->zero, 0, st);
  const KVPools tp{tkv->k, tkv->v, tkv->page_table, c->cfg.max_pages,
                   tkv->n_pages, c->tseg_k, c->tseg_v, D.tpages, c->dbg()};
  const KVPools dp{dkv->k, dkv->v, dkv->page_table, c->cfg.max_pages,
                   dkv->n_pages, c->dseg_k, c->dseg_v, D.dpages, c->dbg()};
  const Prefix tpf{tkv, c->tseg_k, c->tseg_v, D.tpages};
  const Prefix dpf{dkv, c->dseg_k, c->dseg_v, D.dpages};
  const size_t tap_row = (size_t)3 * D.d;
  int longest = 0;
  for (int s = 0; s < sq->n_seqs; ++s) longest = std::max(longest, lens[s]);
  c->T_bound = longest + 1;
  for (int s = 0; s < sq->n_seqs; ++s) {
    const int len = lens[s];
    for (int a = 0; a < len; a += D.chunk) {
      const int n = std::min(D.chunk, len - a);
      launch_plan_prefill_target(S, s, a, n, prompt, ld, p, D.V, c->dbg(), st);
      target_forward<T>(c, p, tpf, D.chunk, c->taps_pf, st);
      launch_seg_to_cache<T>(p, tp, S, D.L, D.Hkv, D.hd, st);
      if (a + n == len) {
        const T* last = static_cast<const T*>(c->A) + (size_t)(n - 1) * D.d;
        lm_head<T>(c, last, c->tw.lm_head, D.V, c->logits, c->one, 1, st);
        const int n_chunks = launch_vocab_partial(
            c->logits, c->one, 1, D.V, D.n_chunks, 1, c->vpart, st);
        launch_verify_finalize(c->vpart, n_chunks, c->one, 1, c->zero,
                               c->root_arg, st);
      }
      launch_plan_prefill_draft(S, s, a, n, prompt, ld, p, c->n_aux, D.V,
                                c->dbg(), st);
      cond_rows<T>(c, c->taps_pf, nullptr, c->n_aux, D.chunk, st);
      drafter_forward<T>(c, p, c->cond_buf, dpf, D.chunk, false, st);
      launch_seg_to_cache<T>(p, dp, S, D.LD, D.Hkv, D.hd, st);
      launch_copy_f32(c->taps_pf, c->taps_pf + (size_t)n * tap_row,
                      (int)tap_row, st);
    }
    launch_prefill_finish(*sq, s, len, D.d, c->taps_pf, 0, c->root_arg, st);
  }
  return hip_check(c, "sb_prefill");
}

int check_common(sb_ctx* c) {
  if (!c) return SB_EINVAL;
  if (!c->bound) return fail(c, SB_ESTATE, "context not bound (call sb_bind)");
  return SB_OK;
}

int check_seqs(sb_ctx* c, const sb_seqs* sq) {
  if (!sq) return fail(c, SB_EINVAL, "seqs is NULL");
  if (sq->n_seqs < 1 || sq->n_seqs > c->cfg.max_seqs)
    return fail(c, SB_ESHAPE, "n_seqs must be in 1..max_seqs");
  if (bad_ptr(sq->root, 4) || bad_ptr(sq->T, 4) || bad_ptr(sq->cond_taps, 4))
    return fail(c, SB_EINVAL, "seqs pointer NULL or misaligned");
  return SB_OK;
}

int check_kv(sb_ctx* c, const sb_kv* kv, int n_layers, const char* what) {
  if (!kv) return fail(c, SB_EINVAL, std::string(what) + " is NULL");
  if (bad_ptr(kv->k, 16) || bad_ptr(kv->v, 16) || bad_ptr(kv->page_table, 4))
    return fail(c, SB_EINVAL, std::string(what) + " pointer NULL or misaligned");
  if (kv->n_layers != n_layers)
    return fail(c, SB_ESHAPE, std::string(what) + " has the wrong layer count");
  if (kv->n_pages < 1) return fail(c, SB_EINVAL, std::string(what) + " has no pages");
  return SB_OK;
}

int check_tree(sb_ctx* c, const sb_tree* t) {
  if (!t) return fail(c, SB_EINVAL, "tree is NULL");
  const void* ps[] = {t->n_nodes, t->token, t->parent, t->depth, t->row,
                      t->rank, t->logp, t->cum_logp, t->anc, t->n_rows,
                      t->row_block, t->row_start, t->row_k, t->row_pos,
                      t->row_vis, t->h_last, t->n_starts, t->starts};
  for (const void* q : ps)
    if (bad_ptr(q, 4)) return fail(c, SB_EINVAL, "tree pointer NULL or misaligned");
  return SB_OK;
}

bool is_bf16(const sb_ctx* c) { return c->cfg.dtype == SB_BF16; }

}  // namespace

extern "C" {

int sb_draft_block_expand(sb_ctx* c, int32_t block_index, int32_t K,
                          const sb_seqs* seqs, const sb_kv* draft_kv,
                          sb_tree* tree, sb_draft_out* out, void* stream) {
  int rc = check_common(c);
  if (rc) return rc;
  if (K != c->cfg.K) return fail(c, SB_ESHAPE, "K differs from cfg.K");
  if (block_index < 1 || block_index > c->cfg.M)
    return fail(c, SB_EINVAL, "block_index must be in 1..M");
  if ((rc = check_seqs(c, seqs)) || (rc = check_kv(c, draft_kv, c->D.LD, "draft_kv")) ||
      (rc = check_tree(c, tree)))
    return rc;
  if (!out) return fail(c, SB_EINVAL, "out is NULL");
  const void* ps[] = {out->topk_id, out->topk_logit, out->lse, out->psi,
                      out->bucket, out->branch, out->call_seq, out->call_row,
                      out->n_call};
  for (const void* q : ps)
    if (bad_ptr(q, 4)) return fail(c, SB_EINVAL, "out pointer NULL or misaligned");
  if (out->logits && bad_ptr(out->logits, 16))
    return fail(c, SB_EINVAL, "out->logits misaligned");
  return is_bf16(c) ? draft_expand_impl<bf16_t>(c, block_index, seqs, draft_kv, tree, out, S_(stream))
                    : draft_expand_impl<float>(c, block_index, seqs, draft_kv, tree, out, S_(stream));
}

int sb_tree_verify(sb_ctx* c, const sb_seqs* seqs, const sb_tree* tree,
                   const sb_kv* target_kv, sb_verify_out* out, void* stream) {
  int rc = check_common(c);
  if (rc) return rc;
  if ((rc = check_seqs(c, seqs)) || (rc = check_kv(c, target_kv, c->D.L, "target_kv")) ||
      (rc = check_tree(c, tree)))
    return rc;
  if (!out || bad_ptr(out->argmax, 4) || bad_ptr(out->taps, 4))
    return fail(c, SB_EINVAL, "verify out pointer NULL or misaligned");
  if (out->logits && bad_ptr(out->logits, 16))
    return fail(c, SB_EINVAL, "out->logits misaligned");
  return is_bf16(c) ? verify_impl<bf16_t>(c, seqs, tree, target_kv, out, S_(stream))
                    : verify_impl<float>(c, seqs, tree, target_kv, out, S_(stream));
}

}  // extern "C"

namespace {

// The verifier-derived signal of sb_accept / sb_accept_sample, when asked.
void reject_signal(sb_ctx* c, int n_seqs, const sb_tree& t,
                   const sb_accept_out& o, hipStream_t st) {
  if (o.r_reject == nullptr) return;
  const float eps = c->cfg.target.norm_eps;
  const float* g = static_cast<const float*>(c->dw.final_norm);
  if (is_bf16(c))
    launch_reject_signal<bf16_t>(tree_dims(c, n_seqs), t, o, c->row_lse,
                                 static_cast<const bf16_t*>(c->dw.lm_head), g,
                                 eps, c->dw.d2t, c->D.Vd, o.r_reject, st);
  else
    launch_reject_signal<float>(tree_dims(c, n_seqs), t, o, c->row_lse,
                                static_cast<const float*>(c->dw.lm_head), g,
                                eps, c->dw.d2t, c->D.Vd, o.r_reject, st);
}

}  // namespace

extern "C" {

int sb_accept(sb_ctx* c, int32_t n_seqs, const sb_tree* tree,
              const int32_t* argmax, sb_accept_out* out, void* stream) {
  int rc = check_common(c);
  if (rc) return rc;
  if (n_seqs < 1 || n_seqs > c->cfg.max_seqs)
    return fail(c, SB_ESHAPE, "n_seqs must be in 1..max_seqs");
  if ((rc = check_tree(c, tree))) return rc;
  if (bad_ptr(argmax, 4) || !out || bad_ptr(out->path, 4) ||
      bad_ptr(out->n_accepted, 4) || bad_ptr(out->bonus, 4) ||
      (out->r_reject && bad_ptr(out->r_reject, 4)))
    return fail(c, SB_EINVAL, "accept pointer NULL or misaligned");
  launch_accept(tree_dims(c, n_seqs), *tree, argmax, *out, S_(stream));
  reject_signal(c, n_seqs, *tree, *out, S_(stream));
  return hip_check(c, "sb_accept");
}

int sb_accept_sample(sb_ctx* c, int32_t n_seqs, const sb_tree* tree,
                     const float* logits, float temperature,
                     const float* u_accept, const float* u_bonus,
                     sb_accept_out* out, void* stream) {
  int rc = check_common(c);
  if (rc) return rc;
  if (n_seqs < 1 || n_seqs > c->cfg.max_seqs)
    return fail(c, SB_ESHAPE, "n_seqs must be in 1..max_seqs");
  if ((rc = check_tree(c, tree))) return rc;
  if (!(temperature > 0.f) || !(temperature < 3.0e38f))
    return fail(c, SB_EINVAL, "temperature must be positive and finite");
  if (bad_ptr(logits, 4) || bad_ptr(u_accept, 4) || bad_ptr(u_bonus, 4) ||
      !out || bad_ptr(out->path, 4) || bad_ptr(out->n_accepted, 4) ||
      bad_ptr(out->bonus, 4) || (out->r_reject && bad_ptr(out->r_reject, 4)))
    return fail(c, SB_EINVAL, "accept_sample pointer NULL or misaligned");
  if (c->D.V > sample_max_vocab())
    return fail(c, SB_ESHAPE, "sb_accept_sample supports vocab <= " +
                                  std::to_string(sample_max_vocab()));
  const hipStream_t st = S_(stream);
  const float inv_t = 1.0f / temperature;
  launch_node_stats(logits, c->D.V, inv_t, tree->n_nodes, n_seqs, c->D.budget,
                    c->node_stats, st);
  launch_accept_sample(tree_dims(c, n_seqs), *tree, logits, c->D.V, inv_t,
                       c->node_stats, u_accept, u_bonus, *out, st);
  reject_signal(c, n_seqs, *tree, *out, st);
  return hip_check(c, "sb_accept_sample");
}

}  // extern "C"

// Scratch of the allocation-free stochastic acceptance: the per-node
// softmax tile statistics that sb_accept_sample keeps in the workspace.
// Every GPU holds its own copy at its own address until the process ends.
constexpr size_t kNoAllocStats = 65536;   // float2 entries, 512 KiB
static __device__ __align__(256) float2 scratch[kNoAllocStats];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};   // device address of scratch per GPU

// Device address of this GPU's scratch, resolved once per device with the
// device current (host code never passes the array's own name).
int scratch_for_current_device(sb_ctx* c, float2** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(c, SB_EHIP, "sb_accept_sample_noalloc: hipGetDevice failed");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || ptr == nullptr)
      return fail(c, SB_EHIP,
                  std::string("sb_accept_sample_noalloc: hipGetSymbolAddress: ") +
                      hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = static_cast<float2*>(g_scratch_ptr[dev]);
  return SB_OK;
}

}  // namespace

extern "C" {

int sb_accept_sample_noalloc(sb_ctx* c, int32_t n_seqs, const sb_tree* tree,
                             const float* logits, float temperature,
                             const float* u_accept, const float* u_bonus,
                             sb_accept_out* out, void* stream) {
  if (!c) return SB_EINVAL;
  if (n_seqs < 1 || n_seqs > c->cfg.max_seqs)
    return fail(c, SB_ESHAPE, "n_seqs must be in 1..max_seqs");
  int rc = check_tree(c, tree);
  if (rc) return rc;
  if (!(temperature > 0.f) || !(temperature < 3.0e38f))
    return fail(c, SB_EINVAL, "temperature must be positive and finite");
  if (bad_ptr(logits, 4) || bad_ptr(u_accept, 4) || bad_ptr(u_bonus, 4) ||
      !out || bad_ptr(out->path, 4) || bad_ptr(out->n_accepted, 4) ||
      bad_ptr(out->bonus, 4) || (out->r_reject && bad_ptr(out->r_reject, 4)))
    return fail(c, SB_EINVAL, "accept_sample pointer NULL or misaligned");
  if (out->r_reject && !c->bound)
    return fail(c, SB_ESTATE,
                "r_reject needs a bound context (drafter weights)");
  if (c->D.V > sample_max_vocab())
    return fail(c, SB_ESHAPE, "sb_accept_sample_noalloc supports vocab <= " +
                                  std::to_string(sample_max_vocab()));
  const size_t need = (size_t)n_seqs * c->D.budget * sample_tiles(c->D.V);
  if (need > kNoAllocStats)
    return fail(c, SB_EBUDGET,
                "sb_accept_sample_noalloc: n_seqs * budget * ceil(vocab / "
                "16384) = " + std::to_string(need) + " exceeds its static "
                "scratch of " + std::to_string(kNoAllocStats) + " entries");
  float2* stats = nullptr;
  if ((rc = scratch_for_current_device(c, &stats))) return rc;
  const hipStream_t st = S_(stream);
  const float inv_t = 1.0f / temperature;
  launch_node_stats(logits, c->D.V, inv_t, tree->n_nodes, n_seqs, c->D.budget,
                    stats, st);
  launch_accept_sample(tree_dims(c, n_seqs), *tree, logits, c->D.V, inv_t,
                       stats, u_accept, u_bonus, *out, st);
  reject_signal(c, n_seqs, *tree, *out, st);
  return hip_check(c, "sb_accept_sample_noalloc");
}

int sb_adapt_push(sb_ctx* c, int32_t n_seqs, const sb_tree* tree,
                  const sb_accept_out* acc, sb_adapt_buffer* buf,
                  void* stream) {
  int rc = check_common(c);
  if (rc) return rc;
  if (c->D.adapt_cap < 1)
    return fail(c, SB_ESTATE, "head updates need cfg.adapt_cap >= 1");
  if (n_seqs < 1 || n_seqs > c->cfg.max_seqs)
    return fail(c, SB_ESHAPE, "n_seqs must be in 1..max_seqs");
  if ((rc = check_tree(c, tree))) return rc;
  if (!acc || bad_ptr(acc->path, 4) || bad_ptr(acc->n_accepted, 4) ||
      bad_ptr(acc->bonus, 4))
    return fail(c, SB_EINVAL, "accept out pointer NULL or misaligned");
  if (!buf || bad_ptr(buf->h, 4) || bad_ptr(buf->target, 4) ||
      bad_ptr(buf->count, 4))
    return fail(c, SB_EINVAL, "adapt buffer pointer NULL or misaligned");
  if (buf->cap != c->D.adapt_cap)
    return fail(c, SB_ESHAPE, "adapt buffer cap differs from cfg.adapt_cap");
  launch_adapt_push(tree_dims(c, n_seqs), *tree, *acc, buf->h, buf->target,
                    buf->count, buf->cap, S_(stream));
  return hip_check(c, "sb_adapt_push");
}

}  // extern "C"

namespace {

template <typename T>
int head_update_impl(sb_ctx* c, sb_adapt_buffer* buf, const void* lm_head0,
                     sb_head_weights* w, float lr, float kl_weight,
                     float* loss_out, hipStream_t st) {
  const Dims& D = c->D;
  const AdaptBufs& a = c->ad;
  const int cap = D.adapt_cap;
  T* A = static_cast<T*>(a.A);
  launch_adapt_prep<T>(buf->h, buf->count, cap,
                       static_cast<const float*>(c->dw.final_norm),
                       c->cfg.target.norm_eps, D.d, A, a.n, st);
  launch_gemm_xwt<T>(A, D.d, static_cast<const T*>(w->lm_head), D.Vd, D.d,
                     a.Z, (size_t)cap * D.Vd, a.n, cap, 1, st);
  launch_gemm_xwt<T>(A, D.d, static_cast<const T*>(lm_head0), D.Vd, D.d, a.Z0,
                     (size_t)cap * D.Vd, a.n, cap, 1, st);
  const int n_chunks = launch_vocab_partial(a.Z, a.n, cap, D.Vd, D.n_chunks_d,
                                            SB_TOPK, a.part, st);
  launch_vocab_partial(a.Z0, a.n, cap, D.Vd, D.n_chunks_d, 1, a.part0, st);
  launch_adapt_rows(a.Z, a.Z0, D.Vd, a.part, a.part0, n_chunks, a.n, cap,
                    buf->h, D.d, buf->target, c->dw.d2t, w->rank_w, w->rank_b,
                    kl_weight, a.psi, a.ds, a.loss, st);
  launch_lm_update<T>(static_cast<T*>(w->lm_head), D.Vd, D.d, a.Z, A, a.n, lr,
                      st);
  launch_rank_update(w->rank_w, w->rank_b, a.ds, buf->h, a.psi, D.d, a.n, lr,
                     a.loss, loss_out, buf->count, st);
  return hip_check(c, "sb_head_update");
}

}  // namespace

extern "C" {

int sb_head_update(sb_ctx* c, sb_adapt_buffer* buf, const void* lm_head0,
                   sb_head_weights* train, float lr, float kl_weight,
                   float* loss_out, void* stream) {
  int rc = check_common(c);
  if (rc) return rc;
  if (c->D.adapt_cap < 1)
    return fail(c, SB_ESTATE, "head updates need cfg.adapt_cap >= 1");
  if (!buf || bad_ptr(buf->h, 4) || bad_ptr(buf->target, 4) ||
      bad_ptr(buf->count, 4))
    return fail(c, SB_EINVAL, "adapt buffer pointer NULL or misaligned");
  if (buf->cap != c->D.adapt_cap)
    return fail(c, SB_ESHAPE, "adapt buffer cap differs from cfg.adapt_cap");
  if (!train || bad_ptr(train->lm_head, 16) || bad_ptr(train->rank_w, 4) ||
      bad_ptr(train->rank_b, 4) || bad_ptr(lm_head0, 16) ||
      (loss_out && bad_ptr(loss_out, 4)))
    return fail(c, SB_EINVAL, "head weights NULL or misaligned");
  if (train->lm_head == lm_head0 || train->lm_head == c->dw.lm_head)
    return fail(c, SB_EINVAL,
                "the training LM head must be its own copy (not the "
                "pre-deployment or the bound one)");
  if (!(lr >= 0.f) || !(kl_weight >= 0.f) || !(lr < 3.0e38f) ||
      !(kl_weight < 3.0e38f))
    return fail(c, SB_EINVAL, "lr and kl_weight must be finite and >= 0");
  return is_bf16(c) ? head_update_impl<bf16_t>(c, buf, lm_head0, train, lr,
                                                kl_weight, loss_out, S_(stream))
                    : head_update_impl<float>(c, buf, lm_head0, train, lr,
                                              kl_weight, loss_out, S_(stream));
}

int sb_commit(sb_ctx* c, sb_seqs* seqs, const sb_tree* tree,
              const sb_verify_out* verify, const sb_accept_out* acc,
              sb_kv* target_kv, sb_kv* draft_kv, void* stream) {
  int rc = check_common(c);
  if (rc) return rc;
  if ((rc = check_seqs(c, seqs)) || (rc = check_tree(c, tree)) ||
      (rc = check_kv(c, target_kv, c->D.L, "target_kv")) ||
      (rc = check_kv(c, draft_kv, c->D.LD, "draft_kv")))
    return rc;
  if (!verify || bad_ptr(verify->taps, 4) || !acc || bad_ptr(acc->path, 4) ||
      bad_ptr(acc->n_accepted, 4) || bad_ptr(acc->bonus, 4))
    return fail(c, SB_EINVAL, "commit pointer NULL or misaligned");
  return is_bf16(c) ? commit_impl<bf16_t>(c, seqs, tree, verify, acc, target_kv, draft_kv, S_(stream))
                    : commit_impl<float>(c, seqs, tree, verify, acc, target_kv, draft_kv, S_(stream));
}

int sb_prefill(sb_ctx* c, const sb_seqs* seqs, const int32_t* prompt,
               int32_t ld_prompt, const int32_t* lens, sb_kv* target_kv,
               sb_kv* draft_kv, void* stream) {
  int rc = check_common(c);
  if (rc) return rc;
  if ((rc = check_seqs(c, seqs)) || (rc = check_kv(c, target_kv, c->D.L, "target_kv")) ||
      (rc = check_kv(c, draft_kv, c->D.LD, "draft_kv")))
    return rc;
  if (bad_ptr(prompt, 4) || !lens) return fail(c, SB_EINVAL, "prompt or lens NULL");
  for (int s = 0; s < seqs->n_seqs; ++s) {
    if (lens[s] < 1 || lens[s] > ld_prompt)
      return fail(c, SB_ESHAPE, "prompt length out of range");
    if (lens[s] + 1 > c->cfg.max_pages * 16)
      return fail(c, SB_EBUDGET, "prompt does not fit max_pages");
  }
  return is_bf16(c) ? prefill_impl<bf16_t>(c, seqs, prompt, ld_prompt, lens, target_kv, draft_kv, S_(stream))
                    : prefill_impl<float>(c, seqs, prompt, ld_prompt, lens, target_kv, draft_kv, S_(stream));
}

}  // extern "C"

extern "C" {

int sb_set_length_bound(sb_ctx* c, int32_t max_T) {
  if (!c) return SB_EINVAL;
  if (max_T < 0) return fail(c, SB_EINVAL, "max_T must be >= 0");
  c->T_bound = max_T;
  return SB_OK;
}

int sb_set_debug(sb_ctx* c, int32_t on) {
  if (!c) return SB_EINVAL;
  if (!c->bound) return fail(c, SB_ESTATE, "context not bound (call sb_bind)");
  // kernels of earlier calls (on any stream) finish before the word is
  // cleared, so that none of them sets a bit after it
  if (hipDeviceSynchronize() != hipSuccess ||
      hipMemset(c->dev_status, 0, sizeof(int)) != hipSuccess)
    return fail(c, SB_EHIP, "clearing the debug status word failed");
  c->status_live = true;
  c->debug = on != 0;
  return SB_OK;
}

int sb_device_check(sb_ctx* c, void* stream) {
  if (!c) return SB_EINVAL;
  if (!c->bound) return fail(c, SB_ESTATE, "context not bound (call sb_bind)");
  if (!c->status_live) return SB_OK;   // no kernel has had the word
  int word = 0;
  if (hipStreamSynchronize(S_(stream)) != hipSuccess ||
      hipMemcpy(&word, c->dev_status, sizeof(int), hipMemcpyDeviceToHost) !=
          hipSuccess)
    return fail(c, SB_EHIP, "reading the debug status word failed");
  if (word == 0) return SB_OK;
  if (hipMemset(c->dev_status, 0, sizeof(int)) != hipSuccess)
    return fail(c, SB_EHIP, "clearing the debug status word failed");
  std::string msg = "out-of-range input clamped on the device:";
  if (word & kDevPage) msg += " page-table entry outside [0, n_pages)";
  if ((word & kDevPage) && (word & kDevToken)) msg += ";";
  if (word & kDevToken) msg += " token id outside [0, vocab)";
  return fail(c, SB_EDEVICE, msg);
}

int sb_set_bucket_override(sb_ctx* c, const int32_t* buckets) {
  if (!c) return SB_EINVAL;
  if (reinterpret_cast<uintptr_t>(buckets) % alignof(int32_t))
    return fail(c, SB_EINVAL, "bucket override must be 4-byte aligned");
  c->bucket_in = buckets;
  return SB_OK;
}

int sb_profile(sb_ctx* c, int32_t enable) {
  if (!c) return SB_EINVAL;
  if (enable) {
    c->recs.clear();
    c->ev_used = 0;
    c->prof_slots_used = 0;
  }
  c->prof = enable != 0;
  return SB_OK;
}

}  // extern "C"

namespace {

// Waits for the recorded events and fills the per-class and per-GEMM-group
// statistics (either output may be NULL).
int profile_collect(sb_ctx* c, sb_kernel_stat* out, sb_gemm_stat* gout) {
  if (out)
    for (int i = 0; i < SB_PROF_N; ++i) out[i] = sb_kernel_stat{0, 0.0, 0.0, 0.0};
  if (gout)
    for (int i = 0; i < SB_GEMM_N; ++i)
      gout[i] = sb_gemm_stat{0, 0, 0.0, 0.0, 0.0, 0.0};
  for (const auto& r : c->recs)
    if (hipEventSynchronize(r.b) != hipSuccess)
      return fail(c, SB_EHIP, "hipEventSynchronize failed");
  std::vector<int> rows(c->prof_slots_used);
  if (!rows.empty() &&
      hipMemcpy(rows.data(), c->prof_rows, rows.size() * sizeof(int),
                hipMemcpyDeviceToHost) != hipSuccess)
    return fail(c, SB_EHIP, "profiler row counts: hipMemcpy failed");
  for (const auto& r : c->recs) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess)
      return fail(c, SB_EHIP, "hipEventElapsedTime failed");
    double bytes = r.bytes, flops = r.flops;
    double rd = 0, wr = 0;
    const bool counted = r.group >= 0;
    if (counted) {
      const int m = r.slot >= 0 ? std::min(std::max(rows[r.slot], 0), r.m_cap)
                                : r.m_cap;
      rd = m > 0 ? r.w_bytes + m * r.in_row : 0.0;
      wr = m * r.out_row;
      bytes = rd + wr;
      flops = m * r.flops_row;
      if (gout) {
        sb_gemm_stat& g = gout[r.group];
        g.launches += 1;
        g.launches_with_rows += m > 0;
        g.total_ms += ms;
        g.bytes_read += rd;
        g.bytes_written += wr;
        g.flops += flops;
      }
    }
    if (out) {
      sb_kernel_stat& k = out[r.cls];
      k.launches += 1;
      k.total_ms += ms;
      k.bytes += bytes;
      k.flops += flops;
    }
  }
  return SB_OK;
}

}  // namespace

extern "C" {

int sb_profile_read(sb_ctx* c, sb_kernel_stat* out) {
  if (!c || !out) return SB_EINVAL;
  return profile_collect(c, out, nullptr);
}

int sb_profile_read_gemm(sb_ctx* c, sb_gemm_stat* out) {
  if (!c || !out) return SB_EINVAL;
  return profile_collect(c, nullptr, out);
}

}  // extern "C"
