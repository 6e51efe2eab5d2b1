// Internal interfaces between the host library (host.cpp) and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace griffin {

// Per-step metadata, device resident, one row per (sequence, node slot):
// row r = b * max_tree + i.  Built on the host from the trees and uploaded in
// one copy per step.
struct StepMeta {
  const int32_t* prefix_len;  // [B]
  const int32_t* n_nodes;     // [B]
  const int32_t* token;       // [R] token id (0 for absent nodes)
  const int32_t* pos;         // [R] rotary position prefix_len + depth
  const int32_t* parent;      // [R]
  const int32_t* depth;       // [R]
  const uint64_t* anc;        // [R] ancestor-or-self bitmask over node ids
  const int4* split_tab;      // [units] prefix-attention work: (b | split << 16, splits of b,
                              // prefix_len[b], n_nodes[b]); x < 0: no work
  const int32_t* n_split;     // [B] key splits of each sequence
};

enum GemmEpilogue : int {
  EPI_STORE = 0,    // fp32 out[split][row][n]
  EPI_SWIGLU = 1,   // packed bf16 act[row][n] = silu(gate) * up (one gate + one up block per wave)
  EPI_ARGMAX = 2,   // per (row, wave column group) max/argmax/NaN count; optional fp32 logits
};

// Shape of a packed weight matrix: the launch it is packed for.  A stream is
// one wave's slice: (split, wg, wave) -> NB blocks of 32 rows for `len`
// 64-wide K steps starting at split * len.
struct PackShape {
  int nb, wn, splits, len, n_wgs;
  int swiglu;   // 1: rows [0, n_out) are gate rows, [n_out, 2 n_out) up rows; a wave's blocks
                // [0, nb/2) are gate blocks, block b + nb/2 the up rows of block b
  int n_out;    // SwiGLU output columns (d_ff)
};

__host__ __device__ inline long long packed_elems(const PackShape& p) {
  return (long long)p.len * p.n_wgs * p.splits * p.wn * p.nb * 2048;
}

// Activations feeding a GEMM are stored as split bf16 (hi + lo planes) in
// fragment order.  Per 64-row tile and 64-wide K step there is one block of
// XPACK_STEP elements: plane (hi, lo), 32-row half mb, piece j = (k % 32) / 8,
// lane r + 32 g (r = m % 32, g = (k % 64) / 32), 8 values.  xpack_off gives
// the offset of the hi value of (row m, column k) in a layout whose tiles hold
// ks steps; the lo value sits XPACK_LO elements further.
constexpr int XPACK_STEP = 8192;
constexpr int XPACK_LO = 4096;
__host__ __device__ inline long long xpack_off(long long m, int k, int ks) {
  const long long tile = m >> 6;
  const int mb = (int)((m >> 5) & 1), r = (int)(m & 31);
  const int s = k >> 6, kk = k & 63, g = kk >> 5, j = (kk >> 3) & 3, e = kk & 7;
  return (tile * ks + s) * XPACK_STEP + mb * 2048 + j * 512 + (r + 32 * g) * 8 + e;
}

struct GemmArgs {
  int epi, nb, wn, pf;       // kernel variant
  int n_wgs, splits, len;    // launch shape (matches the weight packing): splits = K slices
  int kslices;               // K slices merged inside one workgroup (output splits = splits / kslices)
  int tg;                    // 64-row tiles per workgroup sharing each weight fragment (1 or 4)
  int N;                     // output columns (SwiGLU: d_ff)
  int m_tiles;               // 64-row activation tiles
  const uint16_t* X;         // packed activations
  int x_ks;                  // K steps per activation tile
  int xlo;                   // 1: activations as bf16 hi + lo (fp32-grade); 0: the bf16 hi part alone
  int nt;                    // LM head: 1 = non-temporal weight loads (one row tile: each weight read once)
  int x_etiles;              // MoE: activation tiles per expert (0 for dense)
  const int32_t* count;      // MoE: [E] valid rows per expert; NULL = m_tiles * 64
  const uint16_t* W;         // packed weights (+ e * w_estride)
  long long w_estride;
  int o_erows;               // output row = e * o_erows + tile row
  // EPI_STORE
  float* out;
  long long out_split_stride;
  int ldo;
  // EPI_SWIGLU
  uint16_t* act;             // packed activations of the next GEMM
  int act_ks;
  // EPI_ARGMAX
  float* pmax;
  float* pmax2;              // second largest value of the same columns (top-2 margin)
  int32_t* pidx;
  int32_t* pnan;
  int ld_part;
  float* logits;             // optional fp32 [rows][ld_logits], rows < logit_rows
  long long ld_logits;
  int logit_rows;
  // per-launch timing (null when not timed): [0] = ~(earliest workgroup
  // start), [1] = latest wave end, device wall clock; both start at 0
  unsigned long long* stamp;
};

// Residual update folded into the normalisation kernel:
// x[r] += sum_s parts[s][r]           (dense, K-split partial sums), or
// x[r] += sum_k w[r][k] * parts[slot[r][k]]   (MoE expert outputs)
struct ResidualAdd {
  const float* parts;
  int n_parts;
  long long part_stride;     // elements between splits
  const int32_t* slot;       // MoE: [rows][top_k] slot of each kept expert output, NULL for dense
  const float* slot_w;       // MoE: [rows][top_k] renormalised router weights
  int top_k;
};

// MoE routing folded into the RMSNorm before the experts: from the normed fp32
// row h = RMSNorm(x) * gain, router logits h . w_e (fp32), softmax over the
// experts, the top_k kept (ties to the lower id) with renormalised weights.
// w == NULL: no routing.
struct Router {
  const uint16_t* w;         // [n_experts][d] bf16
  int n_experts, top_k;
  const int32_t* n_nodes;    // [B]: rows of absent nodes get id -1
  int max_tree, rows;        // live row slots B * max_tree (padding rows beyond are left alone)
  int32_t* ids;              // [rows][top_k]
  float* weights;            // [rows][top_k]
  float* logits;             // [rows][n_experts], the fp32 router logits (diagnostic)
  // Dispatch of the routed rows to the experts' GEMM operands (count non-null):
  // each row takes place = atomicAdd(count[e], 1) for each kept expert e, in
  // arrival order (a row's expert output does not depend on its place), sets
  // slot[r][k] = e * cap + place and copies its packed operand to row `place`
  // of expert e's tiles xe (xe_ks K steps per tile).  Absent rows and the
  // padding rows up to padded_rows get slot -1.  count starts at zero.
  int32_t* count;            // [n_experts]
  int32_t* slot;             // [padded_rows][top_k]
  uint16_t* xe;              // [n_experts][cap / 64 tiles] packed split bf16
  int xe_ks, cap, padded_rows;
  // Counters this launch sets to zero (the next routed norm's), or null; may
  // be given without routing (w null).
  int32_t* clear;
  int n_clear;
};

// fp32 copies of the tree nodes' K (after rotation) and V for the layer being
// computed, written by qkv_rope next to the bf16 cache entries and read by the
// attention merge, which adds each node's own ancestors in fp32:
//   k, v: [B][Hkv][max_tree][dh]
struct TreeKV32 {
  float* k;
  float* v;
};

// One layer's prefix cache (bf16): K [max_batch][Hkv][kv_cap][dh], V in
// 32-slot transposed tiles [max_batch][Hkv][kv_cap / 32][dh][32].
struct PrefixKV {
  const uint16_t* k;
  const uint16_t* v;
  int kv_cap;
};

struct AttnArgs {
  const uint16_t* q;         // bf16 [R][Hq][dh]
  const uint16_t* q_lo;      // bf16 residual q - bf16(q), same layout
  const uint16_t* k_cache;   // this layer: [max_batch][Hkv][cap][dh]
  const uint16_t* v_cache;   // this layer: [max_batch][Hkv][cap / 32][dh][32]
  float* part_o;             // [B][Hq][sp][qrows][dh]
  float* part_ml;            // [B][Hq][sp][qrows][2]
  StepMeta meta;
  int Hq, Hkv, dh, kv_cap, max_tree, qblocks, batch;
  int units;                 // entries of meta.split_tab
  int sp;                    // split slots per (sequence, head) in the partials (<= 16)
  float scale_log2;          // log2(e) / sqrt(dh)
};

// launchers (return hipGetLastError())
hipError_t launch_gemm(const GemmArgs& a, int experts, hipStream_t s);
hipError_t launch_pack_weight(const uint16_t* src, int rows, int K, const PackShape& p, uint16_t* dst,
                              hipStream_t s);
hipError_t launch_embed(const uint16_t* embed, const int32_t* token, int rows, int d, float* x, hipStream_t s);
hipError_t launch_residual_rmsnorm(float* x, const ResidualAdd& add, const uint16_t* gain, float eps,
                                   int rows, int d, uint16_t* xn, int xn_ks, hipStream_t s,
                                   const Router& route = Router{});
// inv_freq: [dh / 2] fp64 rotary frequencies base^(-2j/dh)
hipError_t launch_qkv_rope(const float* qkv_parts, int n_parts, long long part_stride, StepMeta meta,
                           const double* inv_freq, int Hq, int Hkv, int dh, int max_tree, int batch, int kv_cap,
                           uint16_t* q_out, uint16_t* q_lo, uint16_t* k_cache_l, uint16_t* v_cache_l, TreeKV32 tree,
                           hipStream_t s);
hipError_t launch_attention(const AttnArgs& a, int batch, hipStream_t s);
constexpr int ATTN_RING = 4;  // 32-key K/V blocks in flight per attention workgroup
int attn_waves(int group);    // waves (query heads) per attention workgroup
hipError_t launch_attn_combine(const float* part_o, const float* part_ml, StepMeta meta, int Hq, int Hkv, int dh,
                               int slots, int sp, int qrows, int max_tree, int batch, const uint16_t* q,
                               const uint16_t* q_lo, TreeKV32 tree, PrefixKV prefix, float scale_log2,
                               uint16_t* o_out, int o_ks, hipStream_t s);
hipError_t launch_argmax_reduce(const float* pmax, const float* pmax2, const int32_t* pidx, const int32_t* pnan,
                                int n_tiles, int ld_part, int rows, int32_t* pred, float* margin, int32_t* nan_row,
                                hipStream_t s);
hipError_t launch_commit(const int32_t* result, int max_depth, StepMeta meta, int batch, int n_layers, int Hkv,
                         int dh, int kv_cap, long long layer_kv, uint16_t* k_cache, uint16_t* v_cache,
                         hipStream_t s);
// out[j] = row rows[j] of x ([*][d] fp32), or zeros where rows[j] < 0; n rows.
hipError_t launch_gather_rows(const float* x, int d, const int32_t* rows, int n, float* out, hipStream_t s);
hipError_t launch_accept(StepMeta meta, const int32_t* pred, const int32_t* nan_row, int batch,
                         int max_tree, int max_depth, int32_t* result, hipStream_t s);
// Per-expert row lists (count[e], slot[row][k]) and the gather of the routed
// rows' packed activations into each expert's tiles, in one launch.

// Result block written by the acceptance kernel, per sequence b:
// [0] accept_len, [1] nan flag, [2 .. 2+max_depth] tokens_out (max_depth+1),
// [3+max_depth .. 3+2*max_depth) path.
__host__ __device__ inline int result_stride(int max_depth) { return 3 + 2 * max_depth; }

}  // namespace griffin
