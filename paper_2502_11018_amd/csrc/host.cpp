// Host side of the C ABI declared in include/griffin_verify.h: argument and
// tree validation, per-step metadata, weight packing, workspace ownership and
// the launch sequence of one verification pass.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include <functional>

#include "draft.h"
#include "griffin_internal.h"
#include "plan.h"
#include "sampling.h"
#include "griffin_verify.h"

using namespace griffin;
using namespace griffin_plan;

namespace {

constexpr int kMaxTree = 64;
constexpr int kTargetWaves = 1024;  // one streaming wave per SIMD on 256 CUs

int round_up(int x, int m) { return (x + m - 1) / m * m; }
int cdiv(int x, int m) { return (x + m - 1) / m; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Launch shape of one weight matrix (fixed at init; the packing follows it).
struct GemmPlan {
  int epi = 0, nb = 1, wn = 4, pf = 4;
  int tg = 1;       // 64-row tiles per workgroup
  int kslices = 1;  // K slices merged inside a workgroup (shape.splits / kslices output splits)
  int out_splits() const { return shape.splits / kslices; }
  int n_out = 0;   // output columns
  int rows = 0;    // weight rows (SwiGLU: 2 * n_out)
  int K = 0, ks = 0, ks_pad = 0;
  PackShape shape{};
  long long elems = 0;  // packed elements of one matrix (one expert)
};

// m_tiles: the most 64-row tiles a step of the context can have.  With
// several tiles (batched rows) the GEMMs approach the MFMA bound, and each
// weight fragment is shared between two 64-row tiles per workgroup:
//  * gate/up: every wave holds two gate and the matching two up blocks, so
//    each activation fragment read from LDS feeds four weight blocks (the
//    LDS reads, not HBM, bound these launches);
//  * wide_tiles (QKV, O and down): two 32-column blocks per wave with three
//    pipeline stages.
// Measured at 8 x 61 rows (Llama-3-8B shapes, per launch): gate/up 254 ->
// 222 us; with the wide form down 122 -> 113 us, O 56 -> 45 us, QKV about
// 70 -> 60 us.  The LM head gained little and keeps one tile per workgroup.
GemmPlan plan_gemm(int epi, int n_out, int K, int experts = 1, int m_tiles = 1, bool wide_tiles = false) {
  GemmPlan p;
  p.epi = epi;
  p.n_out = n_out;
  p.K = K;
  p.ks = cdiv(K, 64);
  if (m_tiles >= 2 && experts == 1 && epi == EPI_SWIGLU) {
    p.tg = 2;
    p.kslices = 1;
    p.pf = 3;
    p.nb = 4;
    p.wn = 4;
    p.rows = 2 * n_out;
    const int n_wgs = cdiv(cdiv(n_out, 32 * (p.nb / 2)), p.wn);
    p.ks_pad = p.ks;
    p.shape = PackShape{p.nb, p.wn, 1, p.ks, n_wgs, 1, n_out};
    p.elems = packed_elems(p.shape);
    return p;
  }
  if (m_tiles >= 2 && experts == 1 && epi == EPI_STORE && wide_tiles) {
    // two row tiles per workgroup, two column blocks per wave and three
    // pipeline stages: four blocks with two stages (the register budget's
    // other choice) wait a full memory latency at every step (long-context
    // step 27.1 -> 26.1 ms for O and down, 25.3 ms with QKV in this form)
    p.tg = 2;
    p.kslices = 1;
    p.pf = 3;
    p.nb = 2;
    p.wn = 4;
    p.rows = n_out;
    const int n_wgs = cdiv(cdiv(n_out, 32 * p.nb), p.wn);
    // K splits: about 256 workgroups in all (the grid holds round_up(n_wgs,
    // 8) workgroups per pair of row tiles), at least 4 K steps per split;
    // 512 measured slower for both matrices
    const int per_split = round_up(n_wgs, 8) * cdiv(m_tiles, 2);
    const int splits = std::max(1, std::min(16, std::min(p.ks / 4, 256 / per_split)));
    const int len = cdiv(p.ks, splits);
    p.ks_pad = len * splits;
    p.shape = PackShape{p.nb, p.wn, splits, len, n_wgs, 0, n_out};
    p.elems = packed_elems(p.shape);
    return p;
  }
  int splits = 1;
  if (epi == EPI_SWIGLU) {
    p.nb = 2;
    p.wn = 2;
    p.rows = 2 * n_out;
  } else {
    // the LM head streams two adjacent 32-row blocks per wave: half the
    // activation staging per weight byte, and its ~500 workgroups run in
    // one round at two per CU
    p.nb = epi == EPI_ARGMAX ? 2 : 1;
    p.wn = 4;
    p.rows = n_out;
  }
  const int n_blocks = cdiv(n_out, 32 * (epi == EPI_SWIGLU ? p.nb / 2 : p.nb));
  const int n_wgs = cdiv(n_blocks, p.wn);
  if (epi == EPI_STORE) {
    // split K so that the launch has ~kTargetWaves waves, preferring splits
    // that divide the K steps (little or no zero padding), and at most one
    // workgroup per CU: a launch just past a multiple of 256 workgroups
    // leaves some CUs twice the bytes to stream (measured on the draft's
    // 11008 x 8192 matrix: 2 splits, 172 workgroups, beat 3 and 4)
    const double want = (double)kTargetWaves / ((double)n_wgs * p.wn * experts);
    const int cap = std::max(1, 256 / (n_wgs * experts));
    double best_cost = 1e30;
    for (int s = 1; s <= std::max(1, p.ks / 2) && s <= 16 && s <= cap; ++s) {
      const int len = cdiv(p.ks, s);
      const double pad = (double)(len * s - p.ks) / p.ks;
      const double cost = std::fabs(std::log((double)s / std::max(want, 1.0))) + 8.0 * pad;
      if (cost < best_cost) {
        best_cost = cost;
        splits = s;
      }
    }
  }
  if (epi == EPI_STORE && experts == 1 && p.ks >= 16 * splits) {
    // long K ranges (the down projection): two waves per column block take
    // the two halves of each split's range and merge in LDS, eight waves per
    // workgroup, each with three stages in flight (down 34.3 -> 30.3 us per
    // launch with the non-temporal loads of this form; the shorter QKV and O
    // ranges measured slower so, with one stage in flight)
    p.kslices = 2;
    splits *= 2;
  }
  if (epi == EPI_SWIGLU && p.ks >= 4) {
    // one column block per wave gives too few waves to keep the matrix cores
    // of every SIMD busy with split-bf16 operands: two waves per column block
    // take the two K halves and merge in LDS
    p.kslices = 2;
    splits = 2;
  }
  const int len = cdiv(p.ks, splits);
  p.ks_pad = len * splits;
  p.pf = len >= 8 ? (p.kslices > 1 ? 3 : 4) : 2;
  p.shape = PackShape{p.nb, p.wn, splits, len, n_wgs, epi == EPI_SWIGLU ? 1 : 0, n_out};
  p.elems = packed_elems(p.shape);
  return p;
}

}  // namespace

struct griffin_ctx {
  griffin_model_desc d{};
  const uint16_t *embed = nullptr, *final_norm = nullptr;
  std::vector<const uint16_t*> attn_norm, mlp_norm, w_router;
  uint16_t *k_cache = nullptr, *v_cache = nullptr;
  hipStream_t stream = nullptr;

  int R = 0, Mpad = 0, qkv_n = 0, attn_w = 0, attn_splits = 1, attn_sp = 1, qblocks = 1;
  int comb_slots = 1;  // partial slots the merge reads this step (<= attn_sp)
  int E = 1, topk = 1;
  long long parts_elems = 0;

  // launch plans and packed weights (owned)
  GemmPlan p_qkv, p_o, p_gu, p_down, p_lm;
  int xd_ks = 0;  // K steps per tile of activations with K = d_model
  uint16_t* wpack = nullptr;
  std::vector<const uint16_t*> pk_qkv, pk_o, pk_gu, pk_down;
  const uint16_t* pk_lm = nullptr;

  std::vector<void*> allocs;
  float *x = nullptr, *parts = nullptr, *attn_po = nullptr, *attn_pml = nullptr;
  float *pmax = nullptr, *pmax2 = nullptr, *route_w = nullptr, *yslots = nullptr;
  double* rope_inv = nullptr;      // [head_dim / 2] rotary frequencies base^(-2j/dh), fp64
  float* margin = nullptr;         // [Mpad] top-2 logit margin of every row
  float* margin_host = nullptr;    // pinned copy for griffin_read_margins
  float* router_logits = nullptr;  // MoE: [n_layers][max_batch * max_tree][E] fp32, the last pass's
  uint16_t *xn = nullptr, *q = nullptr, *q_lo = nullptr, *o = nullptr, *act = nullptr, *xe = nullptr;
  TreeKV32 tree{};  // fp32 tree K/V of the layer being computed (reused by every layer)
  int32_t *pidx = nullptr, *pnan = nullptr, *pred = nullptr, *nan_row = nullptr, *result = nullptr;
  int32_t *route_ids = nullptr, *count = nullptr, *slot = nullptr;
  // stochastic acceptance: residual rows [max_batch][2][vocab], uniforms
  // [2][max_batch * max_tree] (accept, final), results
  char* samp_scratch = nullptr;  // sampled_scratch_bytes(max_batch, max_tree, vocab), zeroed
  float* samp_u = nullptr;      // [5][max_batch * max_tree]: u_accept, u_final, work order, step children, tokens
  float* samp_host = nullptr;   // pinned staging of samp_u
  int32_t* samp_result = nullptr;

  // metadata: one device buffer, double-buffered pinned staging
  char* meta_dev = nullptr;
  char* meta_host[2] = {nullptr, nullptr};
  hipEvent_t meta_ev[2] = {nullptr, nullptr};
  size_t meta_bytes = 0;
  size_t off_prefix = 0, off_nodes = 0, off_token = 0, off_pos = 0, off_parent = 0, off_depth = 0, off_anc = 0;
  size_t off_split = 0, off_nsplit = 0;
  int meta_cur = 0;
  StepMeta meta{};

  int32_t* result_host = nullptr;
  int32_t* pred_host = nullptr;
  // per-class launch timing (griffin_profile_*)
  uint32_t prof_mask = 0;

  // captured launch sequences of a pass, keyed by (batch, logits_out,
  // kv_only), and of a whole draft tree (also keyed by k, depth, n_total)
  struct GraphEntry {
    int batch;
    float* logits;
    bool kv_only;
    int tree_k, tree_depth, tree_n;  // 0: one pass
    int slots;                       // partial slots the merge reads
    hipGraphExec_t exec;
  };
  std::vector<GraphEntry> graphs;
  bool use_graphs = true;
  std::vector<hipEvent_t> prof_ev;     // pairs: start, stop
  std::vector<int> prof_cls;           // class of each pair
  size_t prof_used = 0;                // pairs recorded since the last read
  // GEMM launches time themselves on the device wall clock: slots of
  // (~start, end), zeroed when timing is enabled or read
  unsigned long long* prof_stamp = nullptr;
  std::vector<int> stamp_cls;          // class of each used slot
  double wall_khz = 0.0;               // device wall clock rate
  int batch = 0;
  bool stepped = false;
  // the accepted paths griffin_commit moves: the result buffer of the last
  // acceptance (greedy walk or stochastic) since the last step, else null
  const int32_t* accepted = nullptr;
  // A draft model's one-layer context replaces the token embedding by its
  // fusion module (front: writes x) and the final residual + norm by its
  // heads (back: writes xn); it runs no argmax or acceptance.
  std::function<int(griffin_ctx*, hipStream_t)> front;
  std::function<int(griffin_ctx*, const ResidualAdd&, hipStream_t)> back;
  // a pass that ends once the last layer has written the nodes' K/V (a
  // draft catching up on accepted tokens)
  bool kv_only = false;
  // GEMM operands: bf16 hi + lo activations (default) or the bf16 hi part alone
  bool act_bf16 = false;
  // griffin_read_features: rows of x to gather, staged through pinned memory
  int32_t* feat_rows = nullptr;
  int32_t* feat_rows_host = nullptr;
  hipEvent_t feat_ev = nullptr;
  std::string err;
};

namespace {

int set_err(griffin_ctx* c, int code, const std::string& msg) {
  if (c) c->err = msg;
  return code;
}

int hip_err(griffin_ctx* c, const char* what, hipError_t e) {
  return set_err(c, GRIFFIN_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(ctx, call)                                          \
  do {                                                              \
    hipError_t e_ = (call);                                         \
    if (e_ != hipSuccess) return hip_err((ctx), #call, e_);         \
  } while (0)

#define TRY(expr)                      \
  do {                                 \
    int rc_ = (expr);                  \
    if (rc_ != GRIFFIN_OK) return rc_; \
  } while (0)

template <typename T>
int dev_alloc(griffin_ctx* c, T** p, size_t count) {
  void* raw = nullptr;
  const size_t bytes = std::max<size_t>(count * sizeof(T), 256);
  hipError_t e = hipMalloc(&raw, bytes);
  if (e != hipSuccess) return set_err(c, GRIFFIN_ENOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
  c->allocs.push_back(raw);
  e = hipMemset(raw, 0, bytes);
  if (e != hipSuccess) return hip_err(c, "hipMemset", e);
  *p = static_cast<T*>(raw);
  return GRIFFIN_OK;
}

GemmArgs gemm_args(const GemmPlan& p, const uint16_t* X, int x_ks, const uint16_t* W, int m_tiles, bool xlo) {
  GemmArgs a{};
  a.epi = p.epi;
  a.nb = p.nb;
  a.wn = p.wn;
  a.pf = p.pf;
  a.n_wgs = p.shape.n_wgs;
  a.splits = p.shape.splits;
  a.kslices = p.kslices;
  a.tg = p.tg;
  a.len = p.shape.len;
  a.N = p.n_out;
  a.m_tiles = m_tiles;
  // each weight read once (one row tile): stream the LM head past the caches;
  // with several tiles their re-reads of a fragment are served by L2
  a.nt = p.epi == EPI_ARGMAX && m_tiles == 1 ? 1 : 0;
  a.X = X;
  a.x_ks = x_ks;
  a.xlo = xlo ? 1 : 0;
  a.W = W;
  return a;
}

// Event pair for one timed launch (grown on demand, reused after each read).
int prof_pair(griffin_ctx* c, int cls, hipEvent_t* a, hipEvent_t* b) {
  if (c->prof_used * 2 + 2 > c->prof_ev.size()) {
    for (int k = 0; k < 2; ++k) {
      hipEvent_t e;
      HIP_TRY(c, hipEventCreate(&e));
      c->prof_ev.push_back(e);
    }
    c->prof_cls.push_back(0);
  }
  c->prof_cls[c->prof_used] = cls;
  *a = c->prof_ev[2 * c->prof_used];
  *b = c->prof_ev[2 * c->prof_used + 1];
  ++c->prof_used;
  return GRIFFIN_OK;
}

constexpr size_t kStampSlots = 16384;

// A stamp slot for a timed GEMM launch of class cls (null when the class is
// not timed or the slots are used up; the launch then carries events only).
unsigned long long* stamp_slot(griffin_ctx* c, int cls) {
  if (!((c->prof_mask >> cls) & 1u) || !c->prof_stamp || c->stamp_cls.size() >= kStampSlots) return nullptr;
  c->stamp_cls.push_back(cls);
  return c->prof_stamp + 2 * (c->stamp_cls.size() - 1);
}

#define LAUNCH(cls, call)                                                   \
  do {                                                                      \
    hipEvent_t ev0_ = nullptr, ev1_ = nullptr;                              \
    const bool prof_ = (c->prof_mask >> (cls)) & 1u;                        \
    if (prof_) {                                                            \
      TRY(prof_pair(c, (cls), &ev0_, &ev1_));                               \
      HIP_TRY(c, hipEventRecord(ev0_, c->stream));                          \
    }                                                                       \
    HIP_TRY(c, call);                                                       \
    if (prof_) HIP_TRY(c, hipEventRecord(ev1_, c->stream));                 \
  } while (0)

int enqueue_pass(griffin_ctx* c, float* logits_out) {
  const griffin_model_desc& d = c->d;
  const int B = c->batch;
  const int rows = B * d.max_tree;
  const int Mpad = round_up(rows, 64);
  const int m_tiles = Mpad / 64;
  const long long ps = (long long)Mpad;  // rows per split slice of `parts`
  hipStream_t s = c->stream;
  const size_t layer_kv = (size_t)d.max_batch * d.n_kv_heads * d.kv_capacity * d.head_dim;
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d.head_dim));  // log2(e) / sqrt(dh)

  if (c->front)
    TRY(c->front(c, s));
  else
    LAUNCH(GRIFFIN_KC_NORM, launch_embed(c->embed, c->meta.token, Mpad, d.d_model, c->x, s));
  ResidualAdd none{};
  ResidualAdd add_down{};
  for (int l = 0; l < d.n_layers; ++l) {
    // ---- attention block
    Router clear{};  // MoE: this layer's expert counters start at zero
    if (c->E > 1) {
      clear.clear = c->count;
      clear.n_clear = c->E;
    }
    LAUNCH(GRIFFIN_KC_NORM, launch_residual_rmsnorm(c->x, l == 0 ? none : add_down, c->attn_norm[l], d.rms_eps,
                                                    Mpad, d.d_model, c->xn, c->xd_ks, s, clear));
    {
      GemmArgs a = gemm_args(c->p_qkv, c->xn, c->xd_ks, c->pk_qkv[l], m_tiles, !c->act_bf16);
      a.out = c->parts;
      a.ldo = c->qkv_n;
      a.out_split_stride = ps * c->qkv_n;
      a.stamp = stamp_slot(c, GRIFFIN_KC_QKV);
      LAUNCH(GRIFFIN_KC_QKV, launch_gemm(a, 1, s));
    }
    uint16_t* kc = c->k_cache + (size_t)l * layer_kv;
    uint16_t* vc = c->v_cache + (size_t)l * layer_kv;
    LAUNCH(GRIFFIN_KC_ROPE, launch_qkv_rope(c->parts, c->p_qkv.out_splits(), ps * c->qkv_n, c->meta, c->rope_inv,
                                            d.n_q_heads, d.n_kv_heads, d.head_dim, d.max_tree, B, d.kv_capacity,
                                            c->q, c->q_lo, kc, vc, c->tree, s));
    if (c->kv_only && l == d.n_layers - 1) return GRIFFIN_OK;
    {
      AttnArgs a{};
      a.q = c->q;
      a.q_lo = c->q_lo;
      a.k_cache = kc;
      a.v_cache = vc;
      a.part_o = c->attn_po;
      a.part_ml = c->attn_pml;
      a.meta = c->meta;
      a.Hq = d.n_q_heads;
      a.Hkv = d.n_kv_heads;
      a.dh = d.head_dim;
      a.kv_cap = d.kv_capacity;
      a.max_tree = d.max_tree;
      a.qblocks = c->qblocks;
      a.units = B * c->attn_splits;
      a.sp = c->attn_sp;
      a.batch = B;
      a.scale_log2 = scale_log2;
      LAUNCH(GRIFFIN_KC_ATTN, launch_attention(a, B, s));
    }
    LAUNCH(GRIFFIN_KC_MERGE, launch_attn_combine(c->attn_po, c->attn_pml, c->meta, d.n_q_heads, d.n_kv_heads,
                                                d.head_dim, c->comb_slots, c->attn_sp, c->qblocks * 32, d.max_tree,
                                                B, c->q, c->q_lo, c->tree, PrefixKV{kc, vc, d.kv_capacity},
                                                scale_log2, c->o, c->p_o.ks_pad, s));
    {
      GemmArgs a = gemm_args(c->p_o, c->o, c->p_o.ks_pad, c->pk_o[l], m_tiles, !c->act_bf16);
      a.out = c->parts;
      a.ldo = d.d_model;
      a.out_split_stride = ps * d.d_model;
      a.stamp = stamp_slot(c, GRIFFIN_KC_O);
      LAUNCH(GRIFFIN_KC_O, launch_gemm(a, 1, s));
    }
    ResidualAdd add_o{};
    add_o.parts = c->parts;
    add_o.n_parts = c->p_o.out_splits();
    add_o.part_stride = ps * d.d_model;
    Router route{};
    if (c->E > 1) {  // MoE: the MLP norm also routes every row
      route.w = c->w_router[l];
      route.n_experts = c->E;
      route.top_k = c->topk;
      route.n_nodes = c->meta.n_nodes;
      route.max_tree = d.max_tree;
      route.rows = rows;
      route.ids = c->route_ids;
      route.weights = c->route_w;
      route.logits = c->router_logits + (long long)l * rows * c->E;
      route.count = c->count;
      route.slot = c->slot;
      route.xe = c->xe;
      route.xe_ks = c->xd_ks;
      route.cap = Mpad;
      route.padded_rows = Mpad;
    }
    LAUNCH(GRIFFIN_KC_NORM, launch_residual_rmsnorm(c->x, add_o, c->mlp_norm[l], d.rms_eps, Mpad, d.d_model, c->xn,
                                                    c->xd_ks, s, route));

    // ---- MLP block
    if (c->E == 1) {
      GemmArgs g = gemm_args(c->p_gu, c->xn, c->xd_ks, c->pk_gu[l], m_tiles, !c->act_bf16);
      g.act = c->act;
      g.act_ks = c->p_down.ks_pad;
      g.stamp = stamp_slot(c, GRIFFIN_KC_GATE_UP);
      LAUNCH(GRIFFIN_KC_GATE_UP, launch_gemm(g, 1, s));
      GemmArgs dn = gemm_args(c->p_down, c->act, c->p_down.ks_pad, c->pk_down[l], m_tiles, !c->act_bf16);
      dn.out = c->parts;
      dn.ldo = d.d_model;
      dn.out_split_stride = ps * d.d_model;
      dn.stamp = stamp_slot(c, GRIFFIN_KC_DOWN);
      LAUNCH(GRIFFIN_KC_DOWN, launch_gemm(dn, 1, s));
      add_down = ResidualAdd{};
      add_down.parts = c->parts;
      add_down.n_parts = c->p_down.out_splits();
      add_down.part_stride = ps * d.d_model;
    } else {
      const int xe_tiles = Mpad / 64;  // the routing norm filled count, slot and the experts' tiles
      GemmArgs g = gemm_args(c->p_gu, c->xe, c->xd_ks, c->pk_gu[l], m_tiles, !c->act_bf16);
      g.x_etiles = xe_tiles;
      g.count = c->count;
      g.o_erows = Mpad;
      g.w_estride = c->p_gu.elems;
      g.act = c->act;
      g.act_ks = c->p_down.ks_pad;
      g.stamp = stamp_slot(c, GRIFFIN_KC_GATE_UP);
      LAUNCH(GRIFFIN_KC_GATE_UP, launch_gemm(g, c->E, s));
      GemmArgs dn = gemm_args(c->p_down, c->act, c->p_down.ks_pad, c->pk_down[l], m_tiles, !c->act_bf16);
      dn.x_etiles = xe_tiles;
      dn.count = c->count;
      dn.o_erows = Mpad;
      dn.w_estride = c->p_down.elems;
      dn.out = c->yslots;
      dn.ldo = d.d_model;
      dn.out_split_stride = (long long)c->E * Mpad * d.d_model;
      dn.stamp = stamp_slot(c, GRIFFIN_KC_DOWN);
      LAUNCH(GRIFFIN_KC_DOWN, launch_gemm(dn, c->E, s));
      add_down = ResidualAdd{};
      add_down.parts = c->yslots;
      add_down.slot = c->slot;
      add_down.slot_w = c->route_w;
      add_down.top_k = c->topk;
      add_down.n_parts = c->p_down.out_splits();
      add_down.part_stride = (long long)c->E * Mpad * d.d_model;
    }
  }
  // ---- final norm, LM head with fused per-wave argmax, reduction, acceptance
  if (c->back)
    TRY(c->back(c, add_down, s));
  else
    LAUNCH(GRIFFIN_KC_NORM, launch_residual_rmsnorm(c->x, add_down, c->final_norm, d.rms_eps, Mpad, d.d_model,
                                                    c->xn, c->xd_ks, s));
  const int lm_parts = c->p_lm.shape.n_wgs * c->p_lm.wn;
  {
    GemmArgs a = gemm_args(c->p_lm, c->xn, c->xd_ks, c->pk_lm, m_tiles, !c->act_bf16);
    a.pmax = c->pmax;
    a.pmax2 = c->pmax2;
    a.pidx = c->pidx;
    a.pnan = c->pnan;
    a.ld_part = lm_parts;
    a.logits = logits_out;
    a.ld_logits = d.vocab;
    a.logit_rows = rows;
    a.stamp = stamp_slot(c, GRIFFIN_KC_LM_HEAD);
    LAUNCH(GRIFFIN_KC_LM_HEAD, launch_gemm(a, 1, s));
  }
  if (c->front) return GRIFFIN_OK;  // a draft pass: the caller reads the logits
  LAUNCH(GRIFFIN_KC_OTHER, launch_argmax_reduce(c->pmax, c->pmax2, c->pidx, c->pnan, lm_parts, lm_parts, rows,
                                                c->pred, c->margin, c->nan_row, s));
  LAUNCH(GRIFFIN_KC_OTHER, launch_accept(c->meta, c->pred, c->nan_row, B, d.max_tree, d.max_depth, c->result, s));
  return GRIFFIN_OK;
}

// Enqueue a launch sequence: replay the HIP graph captured for its key when
// there is one (at most kMaxGraphs kept, captured on first use), otherwise
// launch kernel by kernel.  Every per-step input lives in device buffers whose
// addresses are fixed for the context, so a graph stays valid for its key.
// Per-class timing and the legacy null stream use the plain launches.
constexpr size_t kMaxGraphs = 8;

template <class Body>
int run_graph(griffin_ctx* c, const griffin_ctx::GraphEntry& key, Body body) {
  if (!c->use_graphs || c->prof_mask != 0 || c->stream == nullptr) return body();
  for (auto& g : c->graphs)
    if (g.batch == key.batch && g.logits == key.logits && g.kv_only == key.kv_only && g.tree_k == key.tree_k &&
        g.tree_depth == key.tree_depth && g.tree_n == key.tree_n && g.slots == key.slots) {
      HIP_TRY(c, hipGraphLaunch(g.exec, c->stream));
      return GRIFFIN_OK;
    }
  HIP_TRY(c, hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal));
  const int rc = body();
  hipGraph_t graph = nullptr;
  const hipError_t e = hipStreamEndCapture(c->stream, &graph);
  if (rc != GRIFFIN_OK) {
    if (graph) hipGraphDestroy(graph);
    return rc;
  }
  HIP_TRY(c, e);
  hipGraphExec_t exec = nullptr;
  const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  hipGraphDestroy(graph);
  HIP_TRY(c, ei);
  if (c->graphs.size() == kMaxGraphs) {
    hipGraphExecDestroy(c->graphs.front().exec);
    c->graphs.erase(c->graphs.begin());
  }
  griffin_ctx::GraphEntry g = key;
  g.exec = exec;
  c->graphs.push_back(g);
  HIP_TRY(c, hipGraphLaunch(exec, c->stream));
  return GRIFFIN_OK;
}

// One pass (batch, logits_out, kv_only from the context).
int run_pass(griffin_ctx* c, float* logits_out) {
  return run_graph(c, {c->batch, logits_out, c->kv_only, 0, 0, 0, c->comb_slots, nullptr},
                   [&]() { return enqueue_pass(c, logits_out); });
}

}  // namespace

// ---------------------------------------------------------------- draft model

struct griffin_draft {
  griffin_ctx* inner = nullptr;  // the decoder layer: a one-layer context with the draft's front and back
  int d = 0, e = 0;
  float ln_eps = 1e-5f;
  GemmPlan p_m, p_u, p_d, p_h;
  uint16_t *pk_m = nullptr, *pk_u = nullptr, *pk_d = nullptr, *pk_h = nullptr;
  const uint16_t *b_m, *ln_h_g, *ln_h_b, *ln_x_g, *ln_x_b, *b_u, *b_d, *b_p, *b_r;
  float *parts = nullptr, *h = nullptr, *feat_r = nullptr, *feat_p = nullptr, *root_feat = nullptr;
  float* node_feat = nullptr;  // [max_batch * max_tree][d]: griffin_draft_extend's features
  float* logits = nullptr;
  uint16_t *x_m = nullptr, *x_u = nullptr, *x_d = nullptr, *x_h = nullptr;
  int32_t* topk_tok = nullptr;
  float* topk_lp = nullptr;
  float* topk_work = nullptr;
  int32_t* topk_tok_host = nullptr;
  float* topk_lp_host = nullptr;
  // griffin_draft_tree's device-side expansion: candidate and pass-tree
  // state, the fixed metadata of every pass (host staging and device copy)
  // and the output rows
  int32_t *c_tok = nullptr, *c_node = nullptr, *n_cand = nullptr;
  double *c_score = nullptr, *n_score = nullptr;
  char* stage_host = nullptr;
  char* stage_dev = nullptr;
  int max_passes = 0;
  hipEvent_t stage_ev = nullptr;  // the staging buffer's last copy
  int32_t* out_dev = nullptr;   // [max_batch] node counts, then tokens, parents, scores [max_batch * max_tree]
  int32_t* out_host = nullptr;
  std::vector<void*> allocs;
};

namespace {

DraftArgs draft_args(griffin_draft* dc, griffin_ctx* c) {
  const griffin_model_desc& d = c->d;
  const int rows = c->batch * d.max_tree, mpad = round_up(rows, 64);
  DraftArgs a{};
  a.d = dc->d;
  a.tgf_dim = dc->e;
  a.rows = rows;
  a.mpad = mpad;
  a.max_tree = d.max_tree;
  a.ln_eps = dc->ln_eps;
  a.rms_eps = d.rms_eps;
  a.embed = c->embed;
  a.root_feat = dc->root_feat;
  a.node_feat = c->kv_only ? dc->node_feat : nullptr;
  a.feat_r = dc->feat_r;
  a.feat_p = dc->feat_p;
  a.h = dc->h;
  a.x = c->x;
  a.parts = dc->parts;
  a.n_parts_m = dc->p_m.out_splits();
  a.n_parts_u = dc->p_u.out_splits();
  a.n_parts_d = dc->p_d.out_splits();
  a.n_parts_h = dc->p_h.out_splits();
  a.stride_m = (long long)mpad * dc->d;
  a.stride_u = (long long)mpad * dc->e;
  a.stride_d = (long long)mpad * dc->d;
  a.stride_h = (long long)mpad * 2 * dc->d;
  a.x_m = dc->x_m;
  a.x_u = dc->x_u;
  a.x_d = dc->x_d;
  a.x_h = dc->x_h;
  a.xn = c->xn;
  a.ks_m = dc->p_m.ks_pad;
  a.ks_u = dc->p_u.ks_pad;
  a.ks_d = dc->p_d.ks_pad;
  a.ks_h = dc->p_h.ks_pad;
  a.xn_ks = c->xd_ks;
  a.b_m = dc->b_m;
  a.ln_h_g = dc->ln_h_g;
  a.ln_h_b = dc->ln_h_b;
  a.ln_x_g = dc->ln_x_g;
  a.ln_x_b = dc->ln_x_b;
  a.b_u = dc->b_u;
  a.b_d = dc->b_d;
  a.b_p = dc->b_p;
  a.b_r = dc->b_r;
  a.final_norm = c->final_norm;
  return a;
}

hipError_t draft_gemm(griffin_draft* dc, griffin_ctx* c, const GemmPlan& p, const uint16_t* X, const uint16_t* W,
                      int N, hipStream_t s) {
  const int mpad = round_up(c->batch * c->d.max_tree, 64);
  GemmArgs a = gemm_args(p, X, p.ks_pad, W, mpad / 64, !c->act_bf16);
  a.out = dc->parts;
  a.ldo = N;
  a.out_split_stride = (long long)mpad * N;
  return launch_gemm(a, 1, s);
}

}  // namespace

extern "C" {

size_t griffin_kv_cache_bytes(const griffin_model_desc* d) {
  if (!d) return 0;
  return (size_t)d->n_layers * d->max_batch * d->n_kv_heads * d->kv_capacity * d->head_dim * 2;
}

const char* griffin_status_str(int code) {
  switch (code) {
    case GRIFFIN_OK: return "ok";
    case GRIFFIN_EINVAL: return "invalid argument";
    case GRIFFIN_ESHAPE: return "unsupported model shape";
    case GRIFFIN_ETREE: return "malformed draft tree";
    case GRIFFIN_ETOKEN: return "token id out of range";
    case GRIFFIN_ECAPACITY: return "KV cache capacity exceeded";
    case GRIFFIN_EORDER: return "accept called before any step";
    case GRIFFIN_ENOMEM: return "out of memory";
    case GRIFFIN_EHIP: return "HIP runtime error";
    case GRIFFIN_ENUMERIC: return "NaN in logits";
    default: return "unknown status";
  }
}

const char* griffin_last_error(const griffin_ctx* ctx) { return ctx ? ctx->err.c_str() : ""; }

int griffin_tree_prepare(int32_t n, const int32_t* tokens, const int32_t* parents, int32_t prefix_len,
                         int32_t max_tree, int32_t max_depth, int32_t vocab, int32_t kv_capacity, int32_t* depth,
                         int32_t* pos, uint64_t* anc) {
  if (max_tree < 1 || max_tree > kMaxTree || vocab < 1 || max_depth < 0) return GRIFFIN_EINVAL;
  return prepare_tree(n, tokens, parents, prefix_len, max_tree, max_depth, vocab, kv_capacity, depth, pos, anc,
                      nullptr);
}

void griffin_verify_free(griffin_ctx* c) {
  if (!c) return;
  hipStreamSynchronize(c->stream);
  for (void* p : c->allocs) hipFree(p);
  for (int k = 0; k < 2; ++k) {
    if (c->meta_host[k]) hipHostFree(c->meta_host[k]);
    if (c->meta_ev[k]) hipEventDestroy(c->meta_ev[k]);
  }
  for (hipEvent_t e : c->prof_ev) hipEventDestroy(e);
  if (c->prof_stamp) hipFree(c->prof_stamp);
  for (auto& g : c->graphs) hipGraphExecDestroy(g.exec);
  if (c->result_host) hipHostFree(c->result_host);
  if (c->pred_host) hipHostFree(c->pred_host);
  if (c->margin_host) hipHostFree(c->margin_host);
  if (c->samp_host) hipHostFree(c->samp_host);
  if (c->feat_rows_host) hipHostFree(c->feat_rows_host);
  if (c->feat_ev) hipEventDestroy(c->feat_ev);
  delete c;
}

int griffin_verify_init(const griffin_model_desc* desc, const griffin_weights* w, void* k_cache, void* v_cache,
                        void* hip_stream, griffin_ctx** out) {
  if (!out) return GRIFFIN_EINVAL;
  *out = nullptr;
  if (!desc || !w || !k_cache || !v_cache) return GRIFFIN_EINVAL;
  std::string why;
  int rc = validate_desc(desc, &why);
  if (rc != GRIFFIN_OK) return rc;
  const griffin_model_desc& d = *desc;
  const bool moe = d.n_experts > 1;
  if (!w->embed || !w->lm_head || !w->final_norm || !w->attn_norm || !w->w_qkv || !w->w_o || !w->mlp_norm ||
      !w->w_gate_up || !w->w_down || (moe && !w->w_router))
    return GRIFFIN_EINVAL;
  if (!aligned16(w->embed) || !aligned16(w->lm_head) || !aligned16(w->final_norm) || !aligned16(k_cache) ||
      !aligned16(v_cache))
    return GRIFFIN_EINVAL;
  for (int l = 0; l < d.n_layers; ++l) {
    const void* ps[] = {w->attn_norm[l], w->w_qkv[l], w->w_o[l], w->mlp_norm[l], w->w_gate_up[l], w->w_down[l],
                        moe ? w->w_router[l] : w->w_qkv[l]};
    for (const void* p : ps)
      if (!p || !aligned16(p)) return GRIFFIN_EINVAL;
  }

  griffin_ctx* c = new (std::nothrow) griffin_ctx();
  if (!c) return GRIFFIN_ENOMEM;
  c->d = d;
  c->embed = static_cast<const uint16_t*>(w->embed);
  c->final_norm = static_cast<const uint16_t*>(w->final_norm);
  for (int l = 0; l < d.n_layers; ++l) {
    c->attn_norm.push_back(static_cast<const uint16_t*>(w->attn_norm[l]));
    c->mlp_norm.push_back(static_cast<const uint16_t*>(w->mlp_norm[l]));
    c->w_router.push_back(moe ? static_cast<const uint16_t*>(w->w_router[l]) : nullptr);
  }
  c->k_cache = static_cast<uint16_t*>(k_cache);
  c->v_cache = static_cast<uint16_t*>(v_cache);
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->E = moe ? d.n_experts : 1;
  c->topk = moe ? d.top_k : 1;

  c->R = d.max_batch * d.max_tree;
  c->Mpad = round_up(c->R, 64);
  c->qkv_n = (d.n_q_heads + 2 * d.n_kv_heads) * d.head_dim;
  c->attn_w = d.n_q_heads * d.head_dim;
  c->qblocks = cdiv(d.max_tree, 32);
  {
    // key splits: about 512 attention workgroups, at least two 32-key
    // blocks per split and at most 16 splits.  A grid of 512 or more runs
    // the kernel's two-workgroups-per-CU form; smaller ones (a single
    // sequence: 16 splits x 16 units) hold one wave per SIMD
    const int G = d.n_q_heads / d.n_kv_heads, nw = attn_waves(G);
    const int units = d.max_batch * d.n_kv_heads * cdiv(G, nw) * c->qblocks;
    const int by_par = cdiv(512, units);
    const int by_len = std::max(1, d.kv_capacity / 64);
    c->attn_splits = std::max(1, std::min(std::min(by_len, by_par), 16));
    // With several sequences a step has batch * attn_splits split units,
    // dealt to its sequences in proportion to their prefix lengths (a split
    // table in the step's metadata); one sequence holds at most twice the
    // even share (and 16), which bounds the slots the merge reads.  A
    // single-sequence context gives its sequence all attn_splits, no table.
    c->attn_sp = d.max_batch > 1 ? std::min(16, 2 * c->attn_splits) : c->attn_splits;
  }
  c->comb_slots = c->attn_sp;
  const int max_tiles = c->Mpad / 64;
  c->p_qkv = plan_gemm(EPI_STORE, c->qkv_n, d.d_model, 1, max_tiles, true);
  c->p_o = plan_gemm(EPI_STORE, d.d_model, c->attn_w, 1, max_tiles, true);
  c->p_gu = plan_gemm(EPI_SWIGLU, d.d_ff, d.d_model, c->E, max_tiles);
  c->p_down = plan_gemm(EPI_STORE, d.d_model, d.d_ff, c->E, max_tiles, true);
  c->p_lm = plan_gemm(EPI_ARGMAX, d.vocab, d.d_model, 1, max_tiles);
  c->xd_ks = std::max({c->p_qkv.ks_pad, c->p_gu.ks_pad, c->p_lm.ks_pad});
  const long long Mp = c->Mpad;
  const long long tiles = Mp / 64;
  c->parts_elems = Mp * std::max({(long long)c->p_qkv.out_splits() * c->qkv_n,
                                  (long long)c->p_o.out_splits() * d.d_model,
                                  (long long)c->p_down.out_splits() * d.d_model});
  const int qrows = c->qblocks * 32;

#define ALLOC(ptr, n)                              \
  do {                                             \
    int rc_ = dev_alloc(c, &(ptr), (size_t)(n));   \
    if (rc_ != GRIFFIN_OK) {                       \
      griffin_verify_free(c);                      \
      return rc_;                                  \
    }                                              \
  } while (0)

  // packed weights, one buffer: per layer qkv, o, gate/up (E experts), down (E experts); then the LM head
  const long long per_layer = c->p_qkv.elems + c->p_o.elems + (long long)c->E * (c->p_gu.elems + c->p_down.elems);
  ALLOC(c->wpack, per_layer * d.n_layers + c->p_lm.elems);
  ALLOC(c->x, Mp * d.d_model);
  ALLOC(c->xn, tiles * c->xd_ks * XPACK_STEP);
  ALLOC(c->parts, c->parts_elems);
  ALLOC(c->q, Mp * c->attn_w);
  ALLOC(c->q_lo, Mp * c->attn_w);
  ALLOC(c->tree.k, (long long)d.max_batch * d.n_kv_heads * d.max_tree * d.head_dim);
  ALLOC(c->tree.v, (long long)d.max_batch * d.n_kv_heads * d.max_tree * d.head_dim);
  ALLOC(c->o, tiles * c->p_o.ks_pad * XPACK_STEP);
  ALLOC(c->attn_po, (long long)d.max_batch * d.n_q_heads * c->attn_sp * qrows * d.head_dim);
  ALLOC(c->attn_pml, (long long)d.max_batch * d.n_q_heads * c->attn_sp * qrows * 2);
  ALLOC(c->act, (long long)c->E * tiles * c->p_down.ks_pad * XPACK_STEP);
  const long long lm_parts = (long long)c->p_lm.shape.n_wgs * c->p_lm.wn;
  ALLOC(c->pmax, Mp * lm_parts);
  ALLOC(c->pmax2, Mp * lm_parts);
  ALLOC(c->margin, Mp);
  ALLOC(c->pidx, Mp * lm_parts);
  ALLOC(c->pnan, Mp * lm_parts);
  ALLOC(c->pred, Mp);
  ALLOC(c->feat_rows, (long long)d.max_batch * d.max_tree);
  ALLOC(c->nan_row, Mp);
  ALLOC(c->result, (long long)d.max_batch * result_stride(d.max_depth));
  ALLOC(c->samp_scratch, sampled_scratch_bytes(d.max_batch, d.max_tree, d.vocab));
  ALLOC(c->samp_u, 5LL * d.max_batch * d.max_tree);
  ALLOC(c->samp_result, (long long)d.max_batch * result_stride(d.max_depth));
  ALLOC(c->rope_inv, d.head_dim / 2);
  if (moe) {
    ALLOC(c->route_ids, Mp * c->topk);
    ALLOC(c->route_w, Mp * c->topk);
    ALLOC(c->router_logits, (long long)d.n_layers * d.max_batch * d.max_tree * c->E);
    ALLOC(c->count, c->E);
    ALLOC(c->slot, Mp * c->topk);
    ALLOC(c->yslots, (long long)c->p_down.out_splits() * c->E * Mp * d.d_model);
    ALLOC(c->xe, (long long)c->E * tiles * c->xd_ks * XPACK_STEP);
  }
#undef ALLOC

  // pack the weight matrices (the caller's copies are not read after this)
  {
    uint16_t* dst = c->wpack;
    hipError_t e = hipSuccess;
    for (int l = 0; l < d.n_layers && e == hipSuccess; ++l) {
      c->pk_qkv.push_back(dst);
      e = launch_pack_weight(static_cast<const uint16_t*>(w->w_qkv[l]), c->qkv_n, d.d_model, c->p_qkv.shape, dst,
                             c->stream);
      dst += c->p_qkv.elems;
      c->pk_o.push_back(dst);
      if (e == hipSuccess)
        e = launch_pack_weight(static_cast<const uint16_t*>(w->w_o[l]), d.d_model, c->attn_w, c->p_o.shape, dst,
                               c->stream);
      dst += c->p_o.elems;
      c->pk_gu.push_back(dst);
      for (int x = 0; x < c->E && e == hipSuccess; ++x) {
        e = launch_pack_weight(static_cast<const uint16_t*>(w->w_gate_up[l]) + (size_t)x * 2 * d.d_ff * d.d_model,
                               2 * d.d_ff, d.d_model, c->p_gu.shape, dst, c->stream);
        dst += c->p_gu.elems;
      }
      c->pk_down.push_back(dst);
      for (int x = 0; x < c->E && e == hipSuccess; ++x) {
        e = launch_pack_weight(static_cast<const uint16_t*>(w->w_down[l]) + (size_t)x * d.d_model * d.d_ff,
                               d.d_model, d.d_ff, c->p_down.shape, dst, c->stream);
        dst += c->p_down.elems;
      }
    }
    c->pk_lm = dst;
    if (e == hipSuccess)
      e = launch_pack_weight(static_cast<const uint16_t*>(w->lm_head), d.vocab, d.d_model, c->p_lm.shape, dst,
                             c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) {
      griffin_verify_free(c);
      return GRIFFIN_EHIP;
    }
  }

  // rotary frequencies base^(-2j/dh) in fp64; the kernel forms the angle
  // pos * inv in fp64 and rounds its cosine and sine to fp32
  {
    const int half = d.head_dim / 2;
    std::vector<double> inv(half);
    for (int j = 0; j < half; ++j) inv[j] = std::pow(d.rope_base, -2.0 * j / d.head_dim);
    hipError_t e = hipMemcpy(c->rope_inv, inv.data(), inv.size() * sizeof(double), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      griffin_verify_free(c);
      return GRIFFIN_EHIP;
    }
  }

  // metadata layout (256-byte aligned sections)
  {
    size_t off = 0;
    auto take = [&](size_t bytes) {
      const size_t o = off;
      off += (bytes + 255) / 256 * 256;
      return o;
    };
    // the rows that depend on the tree's shape first, the rest (fixed for a
    // given batch, prefix and size) after them from off_prefix on
    c->off_anc = take(sizeof(uint64_t) * Mp);
    c->off_token = take(sizeof(int32_t) * Mp);
    c->off_parent = take(sizeof(int32_t) * Mp);
    c->off_prefix = take(sizeof(int32_t) * d.max_batch);
    c->off_nodes = take(sizeof(int32_t) * d.max_batch);
    c->off_pos = take(sizeof(int32_t) * Mp);
    c->off_depth = take(sizeof(int32_t) * Mp);
    c->off_split = take(4 * sizeof(int32_t) * d.max_batch * c->attn_splits);
    c->off_nsplit = take(sizeof(int32_t) * d.max_batch);
    c->meta_bytes = off;
    hipError_t e = hipMalloc((void**)&c->meta_dev, c->meta_bytes);
    if (e != hipSuccess) {
      griffin_verify_free(c);
      return GRIFFIN_ENOMEM;
    }
    c->allocs.push_back(c->meta_dev);
    hipMemset(c->meta_dev, 0, c->meta_bytes);
    for (int k = 0; k < 2; ++k) {
      if (hipHostMalloc((void**)&c->meta_host[k], c->meta_bytes, hipHostMallocDefault) != hipSuccess ||
          hipEventCreateWithFlags(&c->meta_ev[k], hipEventDisableTiming) != hipSuccess) {
        griffin_verify_free(c);
        return GRIFFIN_ENOMEM;
      }
      memset(c->meta_host[k], 0, c->meta_bytes);
    }
    c->meta.anc = reinterpret_cast<const uint64_t*>(c->meta_dev + c->off_anc);
    c->meta.prefix_len = reinterpret_cast<const int32_t*>(c->meta_dev + c->off_prefix);
    c->meta.n_nodes = reinterpret_cast<const int32_t*>(c->meta_dev + c->off_nodes);
    c->meta.token = reinterpret_cast<const int32_t*>(c->meta_dev + c->off_token);
    c->meta.pos = reinterpret_cast<const int32_t*>(c->meta_dev + c->off_pos);
    c->meta.parent = reinterpret_cast<const int32_t*>(c->meta_dev + c->off_parent);
    c->meta.depth = reinterpret_cast<const int32_t*>(c->meta_dev + c->off_depth);
    c->meta.split_tab = d.max_batch > 1 ? reinterpret_cast<const int4*>(c->meta_dev + c->off_split) : nullptr;
    c->meta.n_split = reinterpret_cast<const int32_t*>(c->meta_dev + c->off_nsplit);
  }
  if (hipHostMalloc((void**)&c->result_host, sizeof(int32_t) * d.max_batch * result_stride(d.max_depth),
                    hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->pred_host, sizeof(int32_t) * Mp, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->margin_host, sizeof(float) * Mp, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->samp_host, sizeof(float) * 5 * d.max_batch * d.max_tree, hipHostMallocDefault) !=
          hipSuccess ||
      hipHostMalloc((void**)&c->feat_rows_host, sizeof(int32_t) * d.max_batch * d.max_tree, hipHostMallocDefault) !=
          hipSuccess ||
      hipEventCreateWithFlags(&c->feat_ev, hipEventDisableTiming) != hipSuccess) {
    griffin_verify_free(c);
    return GRIFFIN_ENOMEM;
  }
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    griffin_verify_free(c);
    return GRIFFIN_EHIP;
  }
  *out = c;
  return GRIFFIN_OK;
}

int griffin_verify_step(griffin_ctx* c, int32_t batch, const int32_t* prefix_len, const int32_t* n_nodes,
                        const int32_t* tokens, const int32_t* parents, float* logits_out) {
  if (!c) return GRIFFIN_EINVAL;
  const griffin_model_desc& d = c->d;
  if (batch < 1 || batch > d.max_batch || !prefix_len || !n_nodes || !tokens || !parents)
    return set_err(c, GRIFFIN_EINVAL, "bad batch or null host array");
  if (logits_out && !aligned16(logits_out)) return set_err(c, GRIFFIN_EINVAL, "logits_out not 16-byte aligned");
  // validate everything before touching any buffer
  for (int b = 0; b < batch; ++b) {
    std::string why;
    const int rc = prepare_tree(n_nodes[b], tokens + (size_t)b * d.max_tree, parents + (size_t)b * d.max_tree,
                                prefix_len[b], d.max_tree, d.max_depth, d.vocab, d.kv_capacity, nullptr, nullptr,
                                nullptr, &why);
    if (rc != GRIFFIN_OK) return set_err(c, rc, "sequence " + std::to_string(b) + ": " + why);
  }
  // fill the staging buffer not used by the previous step's copy
  const int k = c->meta_cur ^ 1;
  HIP_TRY(c, hipEventSynchronize(c->meta_ev[k]));
  char* h = c->meta_host[k];
  memset(h, 0, c->meta_bytes);
  auto* h_anc = reinterpret_cast<uint64_t*>(h + c->off_anc);
  auto* h_prefix = reinterpret_cast<int32_t*>(h + c->off_prefix);
  auto* h_nodes = reinterpret_cast<int32_t*>(h + c->off_nodes);
  auto* h_token = reinterpret_cast<int32_t*>(h + c->off_token);
  auto* h_pos = reinterpret_cast<int32_t*>(h + c->off_pos);
  auto* h_parent = reinterpret_cast<int32_t*>(h + c->off_parent);
  auto* h_depth = reinterpret_cast<int32_t*>(h + c->off_depth);
  for (int b = 0; b < batch; ++b) {
    const int n = n_nodes[b];
    const size_t r0 = (size_t)b * d.max_tree;
    h_prefix[b] = prefix_len[b];
    h_nodes[b] = n;
    prepare_tree(n, tokens + r0, parents + r0, prefix_len[b], d.max_tree, d.max_depth, d.vocab, d.kv_capacity,
                 h_depth + r0, h_pos + r0, h_anc + r0, nullptr);
    for (int i = 0; i < n; ++i) {
      h_token[r0 + i] = tokens[r0 + i];
      h_parent[r0 + i] = i == 0 ? 0 : parents[r0 + i];
    }
  }
  attn_split_plan(batch, prefix_len, n_nodes, c->attn_splits, c->attn_sp,
                  reinterpret_cast<int32_t*>(h + c->off_split), reinterpret_cast<int32_t*>(h + c->off_nsplit));
  c->comb_slots = c->meta.split_tab ? merge_slots(reinterpret_cast<const int32_t*>(h + c->off_nsplit), batch, c->attn_sp)
                                    : c->attn_sp;
  HIP_TRY(c, hipMemcpyAsync(c->meta_dev, h, c->meta_bytes, hipMemcpyHostToDevice, c->stream));
  HIP_TRY(c, hipEventRecord(c->meta_ev[k], c->stream));
  c->meta_cur = k;
  c->batch = batch;
  c->stepped = false;
  c->accepted = nullptr;
  const int rc = run_pass(c, logits_out);
  if (rc != GRIFFIN_OK) return rc;
  c->stepped = true;
  return GRIFFIN_OK;
}

int griffin_commit(griffin_ctx* c) {
  if (!c) return GRIFFIN_EINVAL;
  if (!c->stepped) return set_err(c, GRIFFIN_EORDER, "no verification step has been enqueued");
  if (!c->accepted)
    return set_err(c, GRIFFIN_EORDER, "no griffin_accept or griffin_accept_sampled since the last step");
  const griffin_model_desc& d = c->d;
  const long long layer_kv = (long long)d.max_batch * d.n_kv_heads * d.kv_capacity * d.head_dim;
  HIP_TRY(c, launch_commit(c->accepted, d.max_depth, c->meta, c->batch, d.n_layers, d.n_kv_heads, d.head_dim,
                           d.kv_capacity, layer_kv, c->k_cache, c->v_cache, c->stream));
  return GRIFFIN_OK;
}

int griffin_set_activation_precision(griffin_ctx* c, int32_t bf16_only) {
  if (!c) return GRIFFIN_EINVAL;
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  c->act_bf16 = bf16_only != 0;
  for (auto& g : c->graphs) hipGraphExecDestroy(g.exec);  // captured launches carry the GEMM variant
  c->graphs.clear();
  return GRIFFIN_OK;
}

int griffin_set_graphs(griffin_ctx* c, int32_t enable) {
  if (!c) return GRIFFIN_EINVAL;
  c->use_graphs = enable != 0;
  return GRIFFIN_OK;
}

int griffin_accept(griffin_ctx* c, int32_t* accept_len, int32_t* tokens_out, int32_t* path_nodes) {
  if (!c) return GRIFFIN_EINVAL;
  if (!c->stepped) return set_err(c, GRIFFIN_EORDER, "no verification step has been enqueued");
  const griffin_model_desc& d = c->d;
  const int st = result_stride(d.max_depth);
  HIP_TRY(c, hipMemcpyAsync(c->result_host, c->result, sizeof(int32_t) * c->batch * st, hipMemcpyDeviceToHost,
                            c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  c->accepted = c->result;
  bool nan = false;
  for (int b = 0; b < c->batch; ++b) {
    const int32_t* r = c->result_host + (size_t)b * st;
    if (accept_len) accept_len[b] = r[0];
    nan |= r[1] != 0;
    if (tokens_out) memcpy(tokens_out + (size_t)b * (d.max_depth + 1), r + 2, sizeof(int32_t) * (d.max_depth + 1));
    if (path_nodes && d.max_depth > 0)
      memcpy(path_nodes + (size_t)b * d.max_depth, r + 3 + d.max_depth, sizeof(int32_t) * d.max_depth);
  }
  if (nan) return set_err(c, GRIFFIN_ENUMERIC, "NaN in the logits of a tree node");
  return GRIFFIN_OK;
}

int griffin_accept_sampled(griffin_ctx* c, const float* logits, const float* q_draft, const float* u_accept,
                           const float* u_final, float temperature, int32_t* accept_len, int32_t* tokens_out,
                           int32_t* path_nodes) {
  if (!c) return GRIFFIN_EINVAL;
  if (!logits || !u_accept || !u_final)
    return set_err(c, GRIFFIN_EINVAL, "logits and both uniform arrays are required");
  if (!(temperature > 0.f) || !std::isfinite(temperature))
    return set_err(c, GRIFFIN_EINVAL, "temperature must be finite and > 0");
  if (!c->stepped) return set_err(c, GRIFFIN_EORDER, "no verification step has been enqueued");
  const griffin_model_desc& d = c->d;
  const int rows = c->batch * d.max_tree;
  for (int r = 0; r < rows; ++r)
    if (!(u_accept[r] >= 0.f && u_accept[r] < 1.f) || !(u_final[r] >= 0.f && u_final[r] < 1.f))
      return set_err(c, GRIFFIN_EINVAL, "uniforms must lie in [0, 1)");
  std::vector<int32_t> order, step_child, step_token;
  std::vector<int> rows_with;
  const char* mh = c->meta_host[c->meta_cur];
  sampled_plan(c->batch, d.max_tree, reinterpret_cast<const int32_t*>(mh + c->off_nodes),
               reinterpret_cast<const int32_t*>(mh + c->off_parent), reinterpret_cast<const int32_t*>(mh + c->off_token),
               order, rows_with, step_child, step_token);
  // one copy from pinned staging (the previous call's copy ended at its synchronisation)
  memcpy(c->samp_host, u_accept, sizeof(float) * rows);
  memcpy(c->samp_host + rows, u_final, sizeof(float) * rows);
  memcpy(c->samp_host + 2 * rows, order.data(), sizeof(int32_t) * order.size());
  memcpy(c->samp_host + 3 * rows, step_child.data(), sizeof(int32_t) * step_child.size());
  memcpy(c->samp_host + 4 * rows, step_token.data(), sizeof(int32_t) * step_token.size());
  HIP_TRY(c, hipMemcpyAsync(c->samp_u, c->samp_host, sizeof(float) * 5 * rows, hipMemcpyHostToDevice, c->stream));
  const float* ua = c->samp_u;
  const float* uf = c->samp_u + rows;
  SampledArgs a{};
  a.n_nodes = c->meta.n_nodes;
  a.token = c->meta.token;
  a.parent = c->meta.parent;
  a.logits = logits;
  a.q = q_draft;
  a.u_accept = ua;
  a.u_final = uf;
  a.order = reinterpret_cast<const int32_t*>(c->samp_u + 2 * rows);
  a.step_child = reinterpret_cast<const int32_t*>(c->samp_u + 3 * rows);
  a.step_token = reinterpret_cast<const int32_t*>(c->samp_u + 4 * rows);
  a.scratch = c->samp_scratch;
  a.result = c->samp_result;
  a.inv_t = 1.f / temperature;
  a.batch = c->batch;
  a.scratch_batch = d.max_batch;
  a.max_tree = d.max_tree;
  a.max_depth = d.max_depth;
  a.vocab = d.vocab;
  HIP_TRY(c, launch_sampled_accept(a, rows_with.data(), (int)rows_with.size() - 1, c->stream));
  const int st = result_stride(d.max_depth);
  HIP_TRY(c, hipMemcpyAsync(c->result_host, c->samp_result, sizeof(int32_t) * c->batch * st, hipMemcpyDeviceToHost,
                            c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  c->accepted = c->samp_result;
  bool nan = false;
  for (int b = 0; b < c->batch; ++b) {
    const int32_t* r = c->result_host + (size_t)b * st;
    if (accept_len) accept_len[b] = r[0];
    nan |= r[1] != 0;
    if (tokens_out) memcpy(tokens_out + (size_t)b * (d.max_depth + 1), r + 2, sizeof(int32_t) * (d.max_depth + 1));
    if (path_nodes && d.max_depth > 0)
      memcpy(path_nodes + (size_t)b * d.max_depth, r + 3 + d.max_depth, sizeof(int32_t) * d.max_depth);
  }
  if (nan) return set_err(c, GRIFFIN_ENUMERIC, "NaN in the logits of a visited tree node");
  return GRIFFIN_OK;
}

int griffin_read_predictions(griffin_ctx* c, int32_t* pred) {
  if (!c || !pred) return GRIFFIN_EINVAL;
  if (!c->stepped) return set_err(c, GRIFFIN_EORDER, "no verification step has been enqueued");
  const int rows = c->batch * c->d.max_tree;
  HIP_TRY(c, hipMemcpyAsync(c->pred_host, c->pred, sizeof(int32_t) * rows, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  const int32_t* nodes = reinterpret_cast<const int32_t*>(c->meta_host[c->meta_cur] + c->off_nodes);
  for (int r = 0; r < rows; ++r) {
    const int b = r / c->d.max_tree, i = r % c->d.max_tree;
    pred[r] = i < nodes[b] ? c->pred_host[r] : -1;
  }
  return GRIFFIN_OK;
}

int griffin_read_margins(griffin_ctx* c, float* margin) {
  if (!c || !margin) return GRIFFIN_EINVAL;
  if (!c->stepped) return set_err(c, GRIFFIN_EORDER, "no verification step has been enqueued");
  const int rows = c->batch * c->d.max_tree;
  HIP_TRY(c, hipMemcpyAsync(c->margin_host, c->margin, sizeof(float) * rows, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  const int32_t* nodes = reinterpret_cast<const int32_t*>(c->meta_host[c->meta_cur] + c->off_nodes);
  for (int r = 0; r < rows; ++r) {
    const int b = r / c->d.max_tree, i = r % c->d.max_tree;
    margin[r] = i < nodes[b] ? c->margin_host[r] : -1.f;
  }
  return GRIFFIN_OK;
}

int griffin_read_router_logits(griffin_ctx* c, float* out) {
  if (!c || !out) return GRIFFIN_EINVAL;
  if (c->E == 1) return set_err(c, GRIFFIN_EINVAL, "the model has no router (n_experts = 1)");
  if (!c->stepped) return set_err(c, GRIFFIN_EORDER, "no verification step has been enqueued");
  const griffin_model_desc& d = c->d;
  const int rows = c->batch * d.max_tree;
  // the pass writes layer l's rows at l * rows * E (rows of this step's batch)
  const size_t n = (size_t)d.n_layers * rows * c->E;
  HIP_TRY(c, hipMemcpyAsync(out, c->router_logits, sizeof(float) * n, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  const int32_t* nodes = reinterpret_cast<const int32_t*>(c->meta_host[c->meta_cur] + c->off_nodes);
  for (int l = 0; l < d.n_layers; ++l)
    for (int r = 0; r < rows; ++r)
      if (r % d.max_tree >= nodes[r / d.max_tree])
        std::fill(out + ((size_t)l * rows + r) * c->E, out + ((size_t)l * rows + r + 1) * c->E, 0.f);
  return GRIFFIN_OK;
}

int griffin_read_features(griffin_ctx* c, int32_t batch, int32_t n, const int32_t* nodes, float* out) {
  if (!c || !nodes || !out) return GRIFFIN_EINVAL;
  if (!c->stepped) return set_err(c, GRIFFIN_EORDER, "no verification step has been enqueued");
  if (batch < 1 || batch > c->batch || n < 1 || n > c->d.max_tree)
    return set_err(c, GRIFFIN_EINVAL, "batch must be in [1, the last step's batch] and n in [1, max_tree]");
  const int32_t* n_nodes = reinterpret_cast<const int32_t*>(c->meta_host[c->meta_cur] + c->off_nodes);
  HIP_TRY(c, hipEventSynchronize(c->feat_ev));  // the previous call's upload has left the staging buffer
  for (int b = 0; b < batch; ++b)
    for (int j = 0; j < n; ++j) {
      const int node = nodes[(size_t)b * n + j];
      if (node < -1 || node >= n_nodes[b])
        return set_err(c, GRIFFIN_ETREE, "sequence " + std::to_string(b) + ": node " + std::to_string(node) +
                                             " is not a node of the last step");
      c->feat_rows_host[(size_t)b * n + j] = node < 0 ? -1 : b * c->d.max_tree + node;
    }
  HIP_TRY(c, hipMemcpyAsync(c->feat_rows, c->feat_rows_host, sizeof(int32_t) * batch * n, hipMemcpyHostToDevice,
                            c->stream));
  HIP_TRY(c, hipEventRecord(c->feat_ev, c->stream));
  HIP_TRY(c, launch_gather_rows(c->x, c->d.d_model, c->feat_rows, batch * n, out, c->stream));
  return GRIFFIN_OK;
}

int griffin_profile_enable(griffin_ctx* c, uint32_t class_mask) {
  if (!c) return GRIFFIN_EINVAL;
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  c->prof_mask = class_mask & ((1u << GRIFFIN_KC_COUNT) - 1);
  c->prof_used = 0;
  c->stamp_cls.clear();
  if (c->prof_mask && !c->prof_stamp) {
    int dev = 0, khz = 0;
    HIP_TRY(c, hipGetDevice(&dev));
    HIP_TRY(c, hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev));
    if (khz <= 0) return set_err(c, GRIFFIN_EHIP, "device wall clock rate unavailable");
    c->wall_khz = khz;
    void* p = nullptr;
    if (hipMalloc(&p, kStampSlots * 2 * sizeof(unsigned long long)) != hipSuccess)
      return set_err(c, GRIFFIN_ENOMEM, "launch timing slots");
    c->prof_stamp = static_cast<unsigned long long*>(p);
  }
  if (c->prof_stamp)
    HIP_TRY(c, hipMemsetAsync(c->prof_stamp, 0, kStampSlots * 2 * sizeof(unsigned long long), c->stream));
  return GRIFFIN_OK;
}

int griffin_profile_read(griffin_ctx* c, double* ms, int64_t* launches) {
  if (!c || !ms || !launches) return GRIFFIN_EINVAL;
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  for (int k = 0; k < GRIFFIN_KC_COUNT; ++k) {
    ms[k] = 0.0;
    launches[k] = 0;
  }
  // classes timed on the device clock replace their event intervals
  uint32_t stamped = 0;
  for (int k : c->stamp_cls) stamped |= 1u << k;
  for (size_t i = 0; i < c->prof_used; ++i) {
    if ((stamped >> c->prof_cls[i]) & 1u) continue;
    float t = 0.f;
    HIP_TRY(c, hipEventElapsedTime(&t, c->prof_ev[2 * i], c->prof_ev[2 * i + 1]));
    ms[c->prof_cls[i]] += t;
    launches[c->prof_cls[i]] += 1;
  }
  if (!c->stamp_cls.empty()) {
    std::vector<unsigned long long> st(2 * c->stamp_cls.size());
    HIP_TRY(c, hipMemcpy(st.data(), c->prof_stamp, st.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost));
    for (size_t i = 0; i < c->stamp_cls.size(); ++i) {
      if (st[2 * i] == 0 || st[2 * i + 1] == 0) continue;  // a launch whose workgroups all returned early
      const unsigned long long t0 = ~st[2 * i], t1 = st[2 * i + 1];
      ms[c->stamp_cls[i]] += t1 > t0 ? (double)(t1 - t0) / c->wall_khz : 0.0;
      launches[c->stamp_cls[i]] += 1;
    }
    HIP_TRY(c, hipMemsetAsync(c->prof_stamp, 0, st.size() * sizeof(unsigned long long), c->stream));
    HIP_TRY(c, hipStreamSynchronize(c->stream));
  }
  c->stamp_cls.clear();
  c->prof_used = 0;
  return GRIFFIN_OK;
}

int griffin_accept_walk(void* hip_stream, int32_t batch, int32_t max_tree, int32_t max_depth, int32_t vocab,
                        const int32_t* n_nodes, const int32_t* tokens, const int32_t* parents, const int32_t* pred,
                        int32_t* accept_len, int32_t* tokens_out, int32_t* path_nodes) {
  if (batch < 1 || max_tree < 1 || max_tree > kMaxTree || max_depth < 0 || max_depth >= max_tree || vocab < 1 ||
      !n_nodes || !tokens || !parents || !pred)
    return GRIFFIN_EINVAL;
  const int rows = batch * max_tree;
  std::vector<uint64_t> anc(rows, 0);
  std::vector<int32_t> tok(rows, 0), par(rows, 0), dep(rows, 0), pos(rows, 0), nodes(batch), zero(batch, 0);
  for (int b = 0; b < batch; ++b) {
    const size_t r0 = (size_t)b * max_tree;
    const int rc = prepare_tree(n_nodes[b], tokens + r0, parents + r0, 0, max_tree, max_depth, vocab,
                                1 << 30, dep.data() + r0, pos.data() + r0, anc.data() + r0, nullptr);
    if (rc != GRIFFIN_OK) return rc;
    nodes[b] = n_nodes[b];
    for (int i = 0; i < n_nodes[b]; ++i) {
      tok[r0 + i] = tokens[r0 + i];
      par[r0 + i] = i == 0 ? 0 : parents[r0 + i];
      if (pred[r0 + i] < 0 || pred[r0 + i] >= vocab) return GRIFFIN_ETOKEN;
    }
  }
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const int st = result_stride(max_depth);
  char* dev = nullptr;
  const size_t n_anc = sizeof(uint64_t) * rows, n_int = sizeof(int32_t) * rows;
  const size_t total = n_anc + 6 * n_int + sizeof(int32_t) * 2 * batch + sizeof(int32_t) * batch * st + 1024;
  if (hipMalloc((void**)&dev, total) != hipSuccess) return GRIFFIN_ENOMEM;
  char* p = dev;
  auto carve = [&](size_t bytes) {
    char* q = p;
    p += (bytes + 255) / 256 * 256;
    return q;
  };
  StepMeta m{};
  uint64_t* d_anc = reinterpret_cast<uint64_t*>(carve(n_anc));
  int32_t* d_tok = reinterpret_cast<int32_t*>(carve(n_int));
  int32_t* d_par = reinterpret_cast<int32_t*>(carve(n_int));
  int32_t* d_dep = reinterpret_cast<int32_t*>(carve(n_int));
  int32_t* d_pred = reinterpret_cast<int32_t*>(carve(n_int));
  int32_t* d_nan = reinterpret_cast<int32_t*>(carve(n_int));
  int32_t* d_nodes = reinterpret_cast<int32_t*>(carve(sizeof(int32_t) * batch));
  int32_t* d_res = reinterpret_cast<int32_t*>(carve(sizeof(int32_t) * batch * st));
  int rc = GRIFFIN_OK;
  std::vector<int32_t> res((size_t)batch * st);
  hipError_t e = hipSuccess;
  if (p > dev + total) {
    rc = GRIFFIN_ENOMEM;
    goto done;
  }
  m.anc = d_anc;
  m.token = d_tok;
  m.parent = d_par;
  m.depth = d_dep;
  m.n_nodes = d_nodes;
  m.pos = d_dep;
  m.prefix_len = d_nodes;
  if ((e = hipMemcpyAsync(d_anc, anc.data(), n_anc, hipMemcpyHostToDevice, s)) != hipSuccess ||
      (e = hipMemcpyAsync(d_tok, tok.data(), n_int, hipMemcpyHostToDevice, s)) != hipSuccess ||
      (e = hipMemcpyAsync(d_par, par.data(), n_int, hipMemcpyHostToDevice, s)) != hipSuccess ||
      (e = hipMemcpyAsync(d_dep, dep.data(), n_int, hipMemcpyHostToDevice, s)) != hipSuccess ||
      (e = hipMemcpyAsync(d_pred, pred, n_int, hipMemcpyHostToDevice, s)) != hipSuccess ||
      (e = hipMemsetAsync(d_nan, 0, n_int, s)) != hipSuccess ||
      (e = hipMemcpyAsync(d_nodes, nodes.data(), sizeof(int32_t) * batch, hipMemcpyHostToDevice, s)) != hipSuccess ||
      (e = launch_accept(m, d_pred, d_nan, batch, max_tree, max_depth, d_res, s)) != hipSuccess ||
      (e = hipMemcpyAsync(res.data(), d_res, sizeof(int32_t) * batch * st, hipMemcpyDeviceToHost, s)) !=
          hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess) {
    rc = GRIFFIN_EHIP;
    goto done;
  }
  for (int b = 0; b < batch; ++b) {
    const int32_t* r = res.data() + (size_t)b * st;
    if (accept_len) accept_len[b] = r[0];
    if (tokens_out) memcpy(tokens_out + (size_t)b * (max_depth + 1), r + 2, sizeof(int32_t) * (max_depth + 1));
    if (path_nodes && max_depth > 0)
      memcpy(path_nodes + (size_t)b * max_depth, r + 3 + max_depth, sizeof(int32_t) * max_depth);
  }
done:
  hipStreamSynchronize(s);
  hipFree(dev);
  return rc;
}

// The stochastic walk for trees given directly.  Its device memory (staged
// inputs, kernel scratch, result) is one block: hipMalloc'ed for this call
// when `fixed` is null, else the caller's fixed block of `fixed_bytes`.
static int sampled_walk(void* hip_stream, int32_t batch, int32_t max_tree, int32_t max_depth, int32_t vocab,
                        const int32_t* n_nodes, const int32_t* tokens, const int32_t* parents, const float* logits,
                        const float* q_draft, const float* u_accept, const float* u_final, float temperature,
                        int32_t* accept_len, int32_t* tokens_out, int32_t* path_nodes, char* fixed,
                        size_t fixed_bytes) {
  if (batch < 1 || max_tree < 1 || max_tree > kMaxTree || max_depth < 0 || max_depth >= max_tree || vocab < 1 ||
      !n_nodes || !tokens || !parents || !logits || !u_accept || !u_final)
    return GRIFFIN_EINVAL;
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return GRIFFIN_EINVAL;
  const int rows = batch * max_tree;
  const int st = result_stride(max_depth);
  // staging, one copy: tokens [rows], parents [rows], n_nodes [batch], u_accept [rows],
  // u_final [rows] (float bits), work order, step children, step tokens [<= rows each]
  const size_t n_stage = sizeof(int32_t) * (7 * (size_t)rows + batch);
  const size_t n_scratch = sampled_scratch_bytes(batch, max_tree, vocab);
  const size_t total = n_stage + n_scratch + sizeof(int32_t) * batch * st + 3 * 256;
  if (fixed && total > fixed_bytes) return GRIFFIN_ENOMEM;  // before any device work
  std::vector<uint64_t> anc(rows, 0);
  std::vector<int32_t> dep(rows, 0), pos(rows, 0);
  std::vector<int32_t> stage(7 * (size_t)rows + batch, 0);
  int32_t* tok = stage.data();
  int32_t* par = tok + rows;
  int32_t* nodes = par + rows;
  float* uu = reinterpret_cast<float*>(nodes + batch);
  for (int b = 0; b < batch; ++b) {
    const size_t r0 = (size_t)b * max_tree;
    const int rc = prepare_tree(n_nodes[b], tokens + r0, parents + r0, 0, max_tree, max_depth, vocab,
                                1 << 30, dep.data() + r0, pos.data() + r0, anc.data() + r0, nullptr);
    if (rc != GRIFFIN_OK) return rc;
    nodes[b] = n_nodes[b];
    for (int i = 0; i < n_nodes[b]; ++i) {
      tok[r0 + i] = tokens[r0 + i];
      par[r0 + i] = i == 0 ? 0 : parents[r0 + i];
    }
  }
  for (int r = 0; r < rows; ++r) {
    if (!(u_accept[r] >= 0.f && u_accept[r] < 1.f) || !(u_final[r] >= 0.f && u_final[r] < 1.f))
      return GRIFFIN_EINVAL;
    uu[r] = u_accept[r];
    uu[rows + r] = u_final[r];
  }
  std::vector<int32_t> order, step_child, step_token;
  std::vector<int> rows_with;
  sampled_plan(batch, max_tree, nodes, par, tok, order, rows_with, step_child, step_token);
  int32_t* plan = reinterpret_cast<int32_t*>(uu + 2 * rows);
  std::copy(order.begin(), order.end(), plan);
  std::copy(step_child.begin(), step_child.end(), plan + rows);
  std::copy(step_token.begin(), step_token.end(), plan + 2 * rows);
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  char* dev = fixed;
  if (!dev && hipMalloc((void**)&dev, total) != hipSuccess) return GRIFFIN_ENOMEM;
  char* p = dev;
  auto carve = [&](size_t bytes) {
    char* q = p;
    p += (bytes + 255) / 256 * 256;
    return q;
  };
  int32_t* d_stage = reinterpret_cast<int32_t*>(carve(n_stage));
  char* d_scratch = carve(n_scratch);
  int32_t* d_out = reinterpret_cast<int32_t*>(carve(sizeof(int32_t) * batch * st));
  int rc = GRIFFIN_OK;
  std::vector<int32_t> res((size_t)batch * st);
  hipError_t e = hipSuccess;
  SampledArgs a{};
  a.n_nodes = d_stage + 2 * rows;
  a.token = d_stage;
  a.parent = d_stage + rows;
  a.logits = logits;
  a.q = q_draft;
  a.u_accept = reinterpret_cast<const float*>(d_stage + 2 * rows + batch);
  a.u_final = a.u_accept + rows;
  a.order = d_stage + 4 * rows + batch;
  a.step_child = a.order + rows;
  a.step_token = a.order + 2 * rows;
  a.scratch = d_scratch;
  a.result = d_out;
  a.inv_t = 1.f / temperature;
  a.batch = batch;
  a.scratch_batch = batch;
  a.max_tree = max_tree;
  a.max_depth = max_depth;
  a.vocab = vocab;
  if (p > dev + total) {
    rc = GRIFFIN_ENOMEM;
    goto done;
  }
  if ((e = hipMemcpyAsync(d_stage, stage.data(), n_stage, hipMemcpyHostToDevice, s)) != hipSuccess ||
      (e = launch_sampled_accept(a, rows_with.data(), (int)rows_with.size() - 1, s)) != hipSuccess ||
      (e = hipMemcpyAsync(res.data(), d_out, sizeof(int32_t) * batch * st, hipMemcpyDeviceToHost, s)) !=
          hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess) {
    rc = GRIFFIN_EHIP;
    goto done;
  }
  for (int b = 0; b < batch; ++b) {
    const int32_t* r = res.data() + (size_t)b * st;
    if (accept_len) accept_len[b] = r[0];
    if (r[1] != 0) rc = GRIFFIN_ENUMERIC;
    if (tokens_out) memcpy(tokens_out + (size_t)b * (max_depth + 1), r + 2, sizeof(int32_t) * (max_depth + 1));
    if (path_nodes && max_depth > 0)
      memcpy(path_nodes + (size_t)b * max_depth, r + 3 + max_depth, sizeof(int32_t) * max_depth);
  }
done:
  hipStreamSynchronize(s);
  if (!fixed) hipFree(dev);
  return rc;
}

int griffin_accept_sampled_walk(void* hip_stream, int32_t batch, int32_t max_tree, int32_t max_depth, int32_t vocab,
                                const int32_t* n_nodes, const int32_t* tokens, const int32_t* parents,
                                const float* logits, const float* q_draft, const float* u_accept,
                                const float* u_final, float temperature, int32_t* accept_len, int32_t* tokens_out,
                                int32_t* path_nodes) {
  return sampled_walk(hip_stream, batch, max_tree, max_depth, vocab, n_nodes, tokens, parents, logits, q_draft,
                      u_accept, u_final, temperature, accept_len, tokens_out, path_nodes, nullptr, 0);
}

int griffin_accept_sampled_walk_noalloc(void* hip_stream, int32_t batch, int32_t max_tree, int32_t max_depth,
                                        int32_t vocab, const int32_t* n_nodes, const int32_t* tokens,
                                        const int32_t* parents, const float* logits, const float* q_draft,
                                        const float* u_accept, const float* u_final, float temperature,
                                        int32_t* accept_len, int32_t* tokens_out, int32_t* path_nodes) {
  void* block = nullptr;
  size_t bytes = 0;
  if (static_scratch(&block, &bytes) != hipSuccess) return GRIFFIN_EHIP;
  return sampled_walk(hip_stream, batch, max_tree, max_depth, vocab, n_nodes, tokens, parents, logits, q_draft,
                      u_accept, u_final, temperature, accept_len, tokens_out, path_nodes, static_cast<char*>(block),
                      bytes);
}


void griffin_draft_free(griffin_draft* dc) {
  if (!dc) return;
  if (dc->inner) griffin_verify_free(dc->inner);
  for (void* p : dc->allocs) hipFree(p);
  if (dc->topk_tok_host) hipHostFree(dc->topk_tok_host);
  if (dc->topk_lp_host) hipHostFree(dc->topk_lp_host);
  if (dc->stage_host) hipHostFree(dc->stage_host);
  if (dc->stage_ev) hipEventDestroy(dc->stage_ev);
  if (dc->out_host) hipHostFree(dc->out_host);
  delete dc;
}

constexpr int kDraftMaxVocab = 64 * 8192;
constexpr int kDraftMaxDim = 8192;

int griffin_draft_init(const griffin_model_desc* desc, int32_t tgf_dim, float ln_eps, const griffin_draft_weights* w,
                       const void* embed, const void* lm_head, const void* final_norm, void* k_cache, void* v_cache,
                       void* hip_stream, griffin_draft** out) {
  if (!out) return GRIFFIN_EINVAL;
  *out = nullptr;
  if (!desc || !w || !embed || !lm_head || !final_norm || tgf_dim < 1 || !(ln_eps > 0.f)) return GRIFFIN_EINVAL;
  if (desc->n_experts != 1) return GRIFFIN_ESHAPE;  // the draft's decoder layer is dense
  if (desc->vocab > kDraftMaxVocab) return GRIFFIN_ESHAPE;  // the top-k's slice count
  if (desc->d_model > kDraftMaxDim) return GRIFFIN_ESHAPE;   // rows held in registers
  const void* ptrs[] = {w->w_m, w->b_m, w->ln_h_g, w->ln_h_b, w->ln_x_g, w->ln_x_b, w->w_u, w->b_u, w->w_d,
                        w->b_d, w->w_p, w->b_p, w->w_r, w->b_r, w->attn_norm, w->w_qkv, w->w_o, w->mlp_norm,
                        w->w_gate_up, w->w_down};
  for (const void* p : ptrs)
    if (!p) return GRIFFIN_EINVAL;
  griffin_model_desc ld = *desc;
  ld.n_layers = 1;
  griffin_weights lw{};
  lw.embed = embed;
  lw.lm_head = lm_head;
  lw.final_norm = final_norm;
  lw.attn_norm = &w->attn_norm;
  lw.w_qkv = &w->w_qkv;
  lw.w_o = &w->w_o;
  lw.mlp_norm = &w->mlp_norm;
  lw.w_gate_up = &w->w_gate_up;
  lw.w_down = &w->w_down;
  const void* no_router = nullptr;
  lw.w_router = &no_router;
  auto* dc = new griffin_draft();
  int rc = griffin_verify_init(&ld, &lw, k_cache, v_cache, hip_stream, &dc->inner);
  if (rc != GRIFFIN_OK) {
    delete dc;
    return rc;
  }
  griffin_ctx* c = dc->inner;
  const int d = desc->d_model, e = tgf_dim;
  dc->d = d;
  dc->e = e;
  dc->ln_eps = ln_eps;
  dc->b_m = static_cast<const uint16_t*>(w->b_m);
  dc->ln_h_g = static_cast<const uint16_t*>(w->ln_h_g);
  dc->ln_h_b = static_cast<const uint16_t*>(w->ln_h_b);
  dc->ln_x_g = static_cast<const uint16_t*>(w->ln_x_g);
  dc->ln_x_b = static_cast<const uint16_t*>(w->ln_x_b);
  dc->b_u = static_cast<const uint16_t*>(w->b_u);
  dc->b_d = static_cast<const uint16_t*>(w->b_d);
  dc->b_p = static_cast<const uint16_t*>(w->b_p);
  dc->b_r = static_cast<const uint16_t*>(w->b_r);
  const int rows = desc->max_batch * desc->max_tree, mpad = round_up(rows, 64), tiles = mpad / 64;
  dc->p_m = plan_gemm(EPI_STORE, d, 2 * d, 1, tiles);
  dc->p_u = plan_gemm(EPI_STORE, e, 2 * d, 1, tiles);
  dc->p_d = plan_gemm(EPI_STORE, d, e, 1, tiles);
  dc->p_h = plan_gemm(EPI_STORE, 2 * d, d, 1, tiles);
  long long parts = 0;
  for (const GemmPlan* p : {&dc->p_m, &dc->p_u, &dc->p_d, &dc->p_h})
    parts = std::max(parts, (long long)p->out_splits() * mpad * p->n_out);
  auto alloc = [&](void** p, size_t bytes) {
    if (hipMalloc(p, std::max<size_t>(bytes, 256)) != hipSuccess) return false;
    dc->allocs.push_back(*p);
    return hipMemset(*p, 0, std::max<size_t>(bytes, 256)) == hipSuccess;
  };
  bool ok = alloc((void**)&dc->pk_m, 2 * dc->p_m.elems) && alloc((void**)&dc->pk_u, 2 * dc->p_u.elems) &&
            alloc((void**)&dc->pk_d, 2 * dc->p_d.elems) && alloc((void**)&dc->pk_h, 2 * dc->p_h.elems) &&
            alloc((void**)&dc->parts, 4 * parts) && alloc((void**)&dc->h, 4LL * mpad * d) &&
            alloc((void**)&dc->feat_r, 4LL * rows * d) && alloc((void**)&dc->feat_p, 4LL * mpad * d) &&
            alloc((void**)&dc->root_feat, 4LL * desc->max_batch * d) &&
            alloc((void**)&dc->node_feat, 4LL * rows * d) &&
            alloc((void**)&dc->logits, 4LL * rows * desc->vocab) &&
            alloc((void**)&dc->x_m, 2LL * tiles * dc->p_m.ks_pad * XPACK_STEP) &&
            alloc((void**)&dc->x_u, 2LL * tiles * dc->p_u.ks_pad * XPACK_STEP) &&
            alloc((void**)&dc->x_d, 2LL * tiles * dc->p_d.ks_pad * XPACK_STEP) &&
            alloc((void**)&dc->x_h, 2LL * tiles * dc->p_h.ks_pad * XPACK_STEP) &&
            alloc((void**)&dc->topk_tok, 4LL * rows * 16) && alloc((void**)&dc->topk_lp, 4LL * rows * 16) &&
            alloc((void**)&dc->topk_work, draft_topk_work_bytes(rows, desc->vocab)) &&
            hipHostMalloc((void**)&dc->topk_tok_host, 4LL * rows * 16, hipHostMallocDefault) == hipSuccess &&
            hipHostMalloc((void**)&dc->topk_lp_host, 4LL * rows * 16, hipHostMallocDefault) == hipSuccess;
  dc->max_passes = std::min(desc->max_tree, desc->max_depth + 1);
  const size_t tail = c->meta_bytes - c->off_prefix, out_words = desc->max_batch + 3LL * rows;
  ok = ok && alloc((void**)&dc->c_tok, 4LL * desc->max_batch * DRAFT_SEL_MAX) &&
       alloc((void**)&dc->c_node, 4LL * desc->max_batch * DRAFT_SEL_MAX) &&
       alloc((void**)&dc->c_score, 8LL * desc->max_batch * DRAFT_SEL_MAX) &&
       alloc((void**)&dc->n_cand, 4LL * rows) && alloc((void**)&dc->n_score, 8LL * rows) &&
       alloc((void**)&dc->stage_dev, tail * dc->max_passes) && alloc((void**)&dc->out_dev, 4 * out_words) &&
       hipHostMalloc((void**)&dc->stage_host, c->meta_bytes + tail * dc->max_passes, hipHostMallocDefault) ==
           hipSuccess &&
       hipHostMalloc((void**)&dc->out_host, 4 * out_words, hipHostMallocDefault) == hipSuccess &&
       hipEventCreateWithFlags(&dc->stage_ev, hipEventDisableTiming) == hipSuccess;
  if (!ok) {
    griffin_draft_free(dc);
    return GRIFFIN_ENOMEM;
  }
  // pack the four matrices; the heads as one [2d][d] matrix (predict rows, then regress rows)
  uint16_t* heads = nullptr;
  hipError_t he = hipMalloc((void**)&heads, 2LL * 2 * d * d);
  hipStream_t s = c->stream;
  if (he == hipSuccess)
    he = hipMemcpyAsync(heads, w->w_p, 2LL * d * d, hipMemcpyDeviceToDevice, s);
  if (he == hipSuccess)
    he = hipMemcpyAsync(heads + (size_t)d * d, w->w_r, 2LL * d * d, hipMemcpyDeviceToDevice, s);
  if (he == hipSuccess)
    he = launch_pack_weight(static_cast<const uint16_t*>(w->w_m), d, 2 * d, dc->p_m.shape, dc->pk_m, s);
  if (he == hipSuccess)
    he = launch_pack_weight(static_cast<const uint16_t*>(w->w_u), e, 2 * d, dc->p_u.shape, dc->pk_u, s);
  if (he == hipSuccess)
    he = launch_pack_weight(static_cast<const uint16_t*>(w->w_d), d, e, dc->p_d.shape, dc->pk_d, s);
  if (he == hipSuccess) he = launch_pack_weight(heads, 2 * d, d, dc->p_h.shape, dc->pk_h, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (heads) hipFree(heads);
  if (he != hipSuccess) {
    griffin_draft_free(dc);
    return GRIFFIN_EHIP;
  }
  c->front = [dc](griffin_ctx* cc, hipStream_t st) -> int {
    const DraftArgs a = draft_args(dc, cc);
    const int d2 = dc->d;
    HIP_TRY(cc, launch_draft_front(a, cc->meta, 0, st));
    HIP_TRY(cc, draft_gemm(dc, cc, dc->p_m, dc->x_m, dc->pk_m, d2, st));
    HIP_TRY(cc, launch_draft_front(a, cc->meta, 1, st));
    HIP_TRY(cc, draft_gemm(dc, cc, dc->p_u, dc->x_u, dc->pk_u, dc->e, st));
    HIP_TRY(cc, launch_draft_front(a, cc->meta, 2, st));
    HIP_TRY(cc, draft_gemm(dc, cc, dc->p_d, dc->x_d, dc->pk_d, d2, st));
    HIP_TRY(cc, launch_draft_front(a, cc->meta, 3, st));
    return GRIFFIN_OK;
  };
  c->back = [dc](griffin_ctx* cc, const ResidualAdd& add, hipStream_t st) -> int {
    const DraftArgs a = draft_args(dc, cc);
    HIP_TRY(cc, launch_draft_head(a, cc->meta, add, 0, st));
    HIP_TRY(cc, draft_gemm(dc, cc, dc->p_h, dc->x_h, dc->pk_h, 2 * dc->d, st));
    HIP_TRY(cc, launch_draft_head(a, cc->meta, add, 1, st));
    return GRIFFIN_OK;
  };
  *out = dc;
  return GRIFFIN_OK;
}

griffin_ctx* griffin_draft_context(griffin_draft* dc) { return dc ? dc->inner : nullptr; }

int griffin_draft_step(griffin_draft* dc, int32_t batch, const int32_t* prefix_len, const int32_t* n_nodes,
                       const int32_t* tokens, const int32_t* parents, const float* root_features, int32_t k,
                       int32_t* topk_tokens, float* topk_logp) {
  if (!dc) return GRIFFIN_EINVAL;
  griffin_ctx* c = dc->inner;
  const griffin_model_desc& d = c->d;
  if (!root_features || !topk_tokens || !topk_logp || k < 1 || k > 16 || k > d.vocab || batch < 1 ||
      batch > d.max_batch)
    return set_err(c, GRIFFIN_EINVAL, "bad draft step arguments");
  HIP_TRY(c, hipMemcpyAsync(dc->root_feat, root_features, sizeof(float) * batch * dc->d, hipMemcpyDeviceToDevice,
                            c->stream));
  TRY(griffin_verify_step(c, batch, prefix_len, n_nodes, tokens, parents, dc->logits));
  const int rows = batch * d.max_tree;
  HIP_TRY(c, launch_draft_topk(dc->logits, d.vocab, d.vocab, c->meta, rows, d.max_tree, k, dc->topk_tok,
                               dc->topk_lp, dc->topk_work, c->stream));
  HIP_TRY(c, hipMemcpyAsync(dc->topk_tok_host, dc->topk_tok, sizeof(int32_t) * rows * k, hipMemcpyDeviceToHost,
                            c->stream));
  HIP_TRY(c, hipMemcpyAsync(dc->topk_lp_host, dc->topk_lp, sizeof(float) * rows * k, hipMemcpyDeviceToHost,
                            c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  memcpy(topk_tokens, dc->topk_tok_host, sizeof(int32_t) * rows * k);
  memcpy(topk_logp, dc->topk_lp_host, sizeof(float) * rows * k);
  c->stepped = false;  // a draft pass has no acceptance result
  return GRIFFIN_OK;
}

int griffin_draft_extend(griffin_draft* dc, int32_t batch, const int32_t* prefix_len, const int32_t* n_tokens,
                         const int32_t* tokens, const float* features) {
  if (!dc) return GRIFFIN_EINVAL;
  griffin_ctx* c = dc->inner;
  const griffin_model_desc& d = c->d;
  const int T = d.max_tree;
  if (!prefix_len || !n_tokens || !tokens || !features || batch < 1 || batch > d.max_batch)
    return set_err(c, GRIFFIN_EINVAL, "bad draft extend arguments");
  std::vector<int32_t> par((size_t)batch * T, -1);
  for (int b = 0; b < batch; ++b) {
    if (n_tokens[b] < 1 || n_tokens[b] > T || n_tokens[b] - 1 > d.max_depth)
      return set_err(c, GRIFFIN_ETREE, "n_tokens must be in [1, min(max_tree, max_depth + 1)]");
    for (int i = 1; i < n_tokens[b]; ++i) par[(size_t)b * T + i] = i - 1;  // a chain: node i at prefix_len + i
  }
  HIP_TRY(c, hipMemcpyAsync(dc->node_feat, features, sizeof(float) * batch * T * dc->d, hipMemcpyDeviceToDevice,
                            c->stream));
  c->kv_only = true;
  const int rc = griffin_verify_step(c, batch, prefix_len, n_tokens, tokens, par.data(), nullptr);
  c->kv_only = false;
  c->stepped = false;  // nothing to accept or commit: the chain's K/V already sit at their positions
  return rc;
}

int griffin_draft_tree(griffin_draft* dc, int32_t batch, const int32_t* prefix_len, const int32_t* root_tokens,
                       const float* root_features, int32_t k, int32_t depth, int32_t n_total, int32_t* n_nodes_out,
                       int32_t* tokens_out, int32_t* parents_out, float* scores_out) {
  if (!dc) return GRIFFIN_EINVAL;
  griffin_ctx* c = dc->inner;
  const griffin_model_desc& d = c->d;
  const int T = d.max_tree;
  if (!prefix_len || !root_tokens || !root_features || !n_nodes_out || !tokens_out || !parents_out || batch < 1 ||
      batch > d.max_batch || k < 1 || k > 16 || k > d.vocab || depth < 1 || n_total < 1)
    return set_err(c, GRIFFIN_EINVAL, "bad draft tree arguments");
  if (1 + (long long)k * (depth - 1) > T || depth - 1 > d.max_depth)
    return set_err(c, GRIFFIN_ETREE, "1 + k * (depth - 1) expanded nodes must fit max_tree and max_depth");
  if (n_total + 1 > T) return set_err(c, GRIFFIN_ETREE, "n_total + 1 must fit max_tree");
  // Pass t's tree has 1 + k t nodes: the root, then k nodes per depth (node
  // i >= 1 at depth 1 + (i - 1) / k), whichever candidates they hold, so
  // every pass's sizes, positions and attention split table are known here;
  // only the tokens, parents and ancestor masks come from the device.
  auto depth_of = [k](int i) { return i == 0 ? 0 : 1 + (i - 1) / k; };
  const int n_last = 1 + k * (depth - 1);
  {
    std::vector<int32_t> tok(n_last, 0), par(n_last, -1);
    for (int i = 1; i < n_last; ++i) par[i] = depth_of(i) == 1 ? 0 : 1 + k * (depth_of(i) - 2);
    for (int b = 0; b < batch; ++b) {
      tok[0] = root_tokens[b];
      std::string why;
      const int rc = prepare_tree(n_last, tok.data(), par.data(), prefix_len[b], T, d.max_depth, d.vocab,
                                  d.kv_capacity, nullptr, nullptr, nullptr, &why);
      if (rc != GRIFFIN_OK) return set_err(c, rc, "sequence " + std::to_string(b) + ": " + why);
    }
  }
  const size_t mb = c->meta_bytes, tail = mb - c->off_prefix;
  HIP_TRY(c, hipEventSynchronize(dc->stage_ev));  // the previous call's copies out of the staging buffer
  char* h0 = dc->stage_host;
  memset(h0, 0, mb + tail * (depth - 1));
  std::vector<int32_t> nn(batch);
  for (int t = 0; t < depth; ++t) {
    // h + off_x addresses field x of pass t's metadata (fields from off_prefix on, for t > 0)
    char* h = t == 0 ? h0 : h0 + mb + tail * (t - 1) - c->off_prefix;
    auto* prefix = reinterpret_cast<int32_t*>(h + c->off_prefix);
    auto* nodes = reinterpret_cast<int32_t*>(h + c->off_nodes);
    auto* pos = reinterpret_cast<int32_t*>(h + c->off_pos);
    auto* dep = reinterpret_cast<int32_t*>(h + c->off_depth);
    for (int b = 0; b < batch; ++b) {
      nn[b] = 1 + k * t;
      prefix[b] = prefix_len[b];
      nodes[b] = nn[b];
      for (int i = 0; i < nn[b]; ++i) {
        dep[(size_t)b * T + i] = depth_of(i);
        pos[(size_t)b * T + i] = prefix_len[b] + depth_of(i);
      }
      if (t == 0) {
        reinterpret_cast<int32_t*>(h + c->off_token)[(size_t)b * T] = root_tokens[b];
        reinterpret_cast<int32_t*>(h + c->off_parent)[(size_t)b * T] = 0;
        reinterpret_cast<uint64_t*>(h + c->off_anc)[(size_t)b * T] = 1ull;
      }
    }
    attn_split_plan(batch, prefix_len, nn.data(), c->attn_splits, c->attn_sp,
                    reinterpret_cast<int32_t*>(h + c->off_split), reinterpret_cast<int32_t*>(h + c->off_nsplit));
  }
  HIP_TRY(c, hipMemcpyAsync(c->meta_dev, h0, mb, hipMemcpyHostToDevice, c->stream));
  if (depth > 1)
    HIP_TRY(c, hipMemcpyAsync(dc->stage_dev, h0 + mb, tail * (depth - 1), hipMemcpyHostToDevice, c->stream));
  HIP_TRY(c, hipEventRecord(dc->stage_ev, c->stream));
  HIP_TRY(c, hipMemcpyAsync(dc->root_feat, root_features, sizeof(float) * batch * dc->d, hipMemcpyDeviceToDevice,
                            c->stream));
  c->batch = batch;
  c->stepped = false;
  c->accepted = nullptr;
  const int rows = batch * T, MT = d.max_batch * T;
  DraftSelectArgs sa{};
  sa.k = k;
  sa.depth = depth;
  sa.n_total = n_total;
  sa.max_tree = T;
  sa.topk_tok = dc->topk_tok;
  sa.topk_lp = dc->topk_lp;
  sa.c_tok = dc->c_tok;
  sa.c_node = dc->c_node;
  sa.c_score = dc->c_score;
  sa.n_cand = dc->n_cand;
  sa.n_score = dc->n_score;
  sa.m_token = reinterpret_cast<int32_t*>(c->meta_dev + c->off_token);
  sa.m_parent = reinterpret_cast<int32_t*>(c->meta_dev + c->off_parent);
  sa.m_anc = reinterpret_cast<uint64_t*>(c->meta_dev + c->off_anc);
  sa.tail_dst = reinterpret_cast<uint4*>(c->meta_dev + c->off_prefix);
  sa.o_nodes = dc->out_dev;
  sa.o_tok = dc->out_dev + d.max_batch;
  sa.o_par = sa.o_tok + MT;
  sa.o_score = reinterpret_cast<float*>(sa.o_par + MT);
  // the whole expansion, every pass with its top-k and selection, is one graph
  // the passes' split plans differ, so the merge reads every slot
  c->comb_slots = c->attn_sp;
  TRY(run_graph(c, {batch, dc->logits, false, k, depth, n_total, c->comb_slots, nullptr}, [&]() -> int {
    for (int t = 0; t < depth; ++t) {
      TRY(enqueue_pass(c, dc->logits));
      HIP_TRY(c, launch_draft_topk(dc->logits, d.vocab, d.vocab, c->meta, rows, T, k, dc->topk_tok, dc->topk_lp,
                                   dc->topk_work, c->stream));
      sa.t = t;
      const bool more = t + 1 < depth;
      sa.tail_src = more ? reinterpret_cast<const uint4*>(dc->stage_dev + tail * t) : nullptr;
      sa.tail_words = more ? (int)(tail / 16) : 0;
      HIP_TRY(c, launch_draft_select(sa, batch, c->stream));
    }
    return GRIFFIN_OK;
  }));
  HIP_TRY(c, hipMemcpyAsync(dc->out_host, dc->out_dev, sizeof(int32_t) * (d.max_batch + 3LL * MT),
                            hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  const int32_t* o_tok = dc->out_host + d.max_batch;
  const int32_t* o_par = o_tok + MT;
  const float* o_score = reinterpret_cast<const float*>(o_par + MT);
  for (int b = 0; b < batch; ++b) {
    const int n = dc->out_host[b];
    n_nodes_out[b] = n;
    memcpy(tokens_out + (size_t)b * T, o_tok + (size_t)b * T, sizeof(int32_t) * n);
    memcpy(parents_out + (size_t)b * T, o_par + (size_t)b * T, sizeof(int32_t) * n);
    if (scores_out) memcpy(scores_out + (size_t)b * T, o_score + (size_t)b * T, sizeof(float) * n);
  }
  return GRIFFIN_OK;
}

}  // extern "C"
