// GRIFFIN-style draft model: the kernels around its decoder layer.
//
// The draft (Sec. 4.2) fuses an input feature F with the token embedding e in
// Token-Guided Fusion, runs one decoder layer, and splits the result in the
// Token-Enhanced Head:
//   h = [F, e] W_m + b_m;  z = [LN(h), LN(e)] W_u + b_u;  o = SiLU(z) W_d + b_d + h
//   y = decoder layer(o);  F^P = y W_p + b_p;  F^R = y W_r + b_r
//   logits = RMSNorm(F^P) (the target's final norm) times the target's LM head
// The four matrices go through the library's GEMM (split-K partials, fp32);
// the kernels here sum those partials in split order, add biases, normalise
// and write the next GEMM's split-bf16 operand.  Rows are b * max_tree + i;
// rows of absent nodes get zero operands.  A node's input feature is its
// parent's regress feature from the previous draft pass (the root's is the
// caller's), unless the caller gives every node's feature (a draft catching
// up on accepted tokens with the target's features).

#include "device_common.h"
#include "draft.h"
#include "griffin_internal.h"

namespace griffin {

constexpr int DT = 256;   // threads per workgroup of the elementwise kernels
constexpr int DR = 1024;  // threads per workgroup of the per-row reductions (LayerNorm, RMSNorm)

__device__ __forceinline__ bool draft_live(const StepMeta& m, int r, int rows, int max_tree) {
  return r < rows && (r % max_tree) < m.n_nodes[r / max_tree];
}

__device__ __forceinline__ void put_split(uint16_t* dst, long long off, float v) {
  const uint16_t hi = f32_to_bf16(v);
  dst[off] = hi;
  dst[off + XPACK_LO] = f32_to_bf16(v - bf16_to_f32(hi));
}

__device__ __forceinline__ float sum_parts(const float* parts, int n, long long stride, long long at) {
  float s = 0.f;
  for (int p = 0; p < n; ++p) s += parts[p * stride + at];
  return s;
}

__device__ __forceinline__ float dblock_sum(float v, float* red) { return block_sum(v, red); }

// [F, e] of every row as the operand of W_m (K = 2d).
__global__ __launch_bounds__(DT) void draft_in_kernel(DraftArgs a, StepMeta meta) {  // grid (rows, y)
  const int r = blockIdx.x, d = a.d;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  const int b = r / a.max_tree, i = r % a.max_tree;
  const float* f = a.node_feat ? a.node_feat + (long long)min(r, a.rows - 1) * d
                  : i == 0    ? a.root_feat + (long long)b * d
                              : a.feat_r + ((long long)b * a.max_tree + meta.parent[min(r, a.rows - 1)]) * d;
  const uint16_t* e = a.embed + (long long)meta.token[min(r, a.rows - 1)] * d;
  for (int k = blockIdx.y * DT + threadIdx.x; k < 2 * d; k += gridDim.y * DT) {
    const float v = !live ? 0.f : (k < d ? f[k] : bf16_to_f32(e[k - d]));
    put_split(a.x_m, xpack_off(r, k, a.ks_m), v);
  }
}

// Per-row reductions hold a row in registers: RV values per thread.
constexpr int RV = 8;  // d <= DR * RV

// acc[j] += the split-K partials of column threadIdx.x + j * DR of the row at
// `at`, in split order; four splits' loads are issued together.
__device__ __forceinline__ void add_parts(float (&acc)[RV], const float* parts, int n, long long stride, long long at,
                                          int d) {
  for (int p0 = 0; p0 < n; p0 += 4) {
    float t[4][RV];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int j = 0; j < RV; ++j) {
        const int k = threadIdx.x + j * DR;
        t[u][j] = p0 + u < n && k < d ? parts[(p0 + u) * stride + at + k] : 0.f;
      }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int j = 0; j < RV; ++j) acc[j] += t[u][j];
  }
}

// Two block-wide sums at once (fixed order).
__device__ __forceinline__ float2 block_sum2(float x, float y, float* red /* >= 32 floats */) {
  x = wave_sum(x);
  y = wave_sum(y);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    red[w] = x;
    red[16 + w] = y;
  }
  __syncthreads();
  float sx = 0.f, sy = 0.f;
  for (int i = 0; i < nw; ++i) {
    sx += red[i];
    sy += red[16 + i];
  }
  return make_float2(sx, sy);
}

// h = sum of the W_m partials + b_m (kept), then [LN(h), LN(e)] as the
// operand of W_u (K = 2d).
__global__ __launch_bounds__(DR) void draft_fuse_kernel(DraftArgs a, StepMeta meta) {
  __shared__ float red[32];
  const int r = blockIdx.x, d = a.d;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  const uint16_t* e = a.embed + (long long)meta.token[min(r, a.rows - 1)] * d;
  float hv[RV], ev[RV];
#pragma unroll
  for (int j = 0; j < RV; ++j) {
    const int k = threadIdx.x + j * DR;
    hv[j] = 0.f;
    ev[j] = k < d ? bf16_to_f32(e[k]) : 0.f;
  }
  if (live) add_parts(hv, a.parts, a.n_parts_m, a.stride_m, (long long)r * d, d);
  float sh = 0.f, se = 0.f;
#pragma unroll
  for (int j = 0; j < RV; ++j) {
    const int k = threadIdx.x + j * DR;
    if (k < d) {
      hv[j] = live ? hv[j] + bf16_to_f32(a.b_m[k]) : 0.f;
      a.h[(long long)r * d + k] = hv[j];
      sh += hv[j];
      se += ev[j];
    }
  }
  const float2 mean = block_sum2(sh, se, red);
  const float mh = mean.x / d, me = mean.y / d;
  float vh = 0.f, ve = 0.f;
#pragma unroll
  for (int j = 0; j < RV; ++j)
    if (threadIdx.x + j * DR < d) {
      vh += (hv[j] - mh) * (hv[j] - mh);
      ve += (ev[j] - me) * (ev[j] - me);
    }
  const float2 var = block_sum2(vh, ve, red);
  const float rh = rsqrtf(var.x / d + a.ln_eps), re = rsqrtf(var.y / d + a.ln_eps);
#pragma unroll
  for (int j = 0; j < RV; ++j) {
    const int k = threadIdx.x + j * DR;
    if (k < d) {
      const float lh = (hv[j] - mh) * rh * bf16_to_f32(a.ln_h_g[k]) + bf16_to_f32(a.ln_h_b[k]);
      const float le = (ev[j] - me) * re * bf16_to_f32(a.ln_x_g[k]) + bf16_to_f32(a.ln_x_b[k]);
      put_split(a.x_u, xpack_off(r, k, a.ks_u), live ? lh : 0.f);
      put_split(a.x_u, xpack_off(r, d + k, a.ks_u), live ? le : 0.f);
    }
  }
}

// SiLU(sum of the W_u partials + b_u) as the operand of W_d (K = tgf_dim).
__global__ __launch_bounds__(DT) void draft_silu_kernel(DraftArgs a, StepMeta meta) {
  const int r = blockIdx.x, e = a.tgf_dim;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  for (int k = blockIdx.y * DT + threadIdx.x; k < e; k += gridDim.y * DT) {
    float v = 0.f;
    if (live) {
      const float z = sum_parts(a.parts, a.n_parts_u, a.stride_u, (long long)r * e + k) + bf16_to_f32(a.b_u[k]);
      v = z / (1.f + expf(-z));
    }
    put_split(a.x_d, xpack_off(r, k, a.ks_d), v);
  }
}

// o = sum of the W_d partials + b_d + h: the decoder layer's input x.
__global__ __launch_bounds__(DT) void draft_out_kernel(DraftArgs a, StepMeta meta) {
  const int r = blockIdx.x, d = a.d;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  for (int k = blockIdx.y * DT + threadIdx.x; k < d; k += gridDim.y * DT) {
    const long long at = (long long)r * d + k;
    a.x[at] = live ? sum_parts(a.parts, a.n_parts_d, a.stride_d, at) + bf16_to_f32(a.b_d[k]) + a.h[at] : 0.f;
  }
}

// y = x + the decoder layer's last residual (down-projection partials), as
// the operand of [W_p; W_r] (K = d).
__global__ __launch_bounds__(DT) void draft_head_in_kernel(DraftArgs a, StepMeta meta, ResidualAdd add) {
  const int r = blockIdx.x, d = a.d;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  for (int k = blockIdx.y * DT + threadIdx.x; k < d; k += gridDim.y * DT) {
    const long long at = (long long)r * d + k;
    const float y = live ? a.x[at] + sum_parts(add.parts, add.n_parts, add.part_stride, at) : 0.f;
    put_split(a.x_h, xpack_off(r, k, a.ks_h), y);
  }
}

// F^P and F^R from the head partials; F^R is kept for the next pass, and
// RMSNorm(F^P) times the final norm's gain becomes the LM head's operand.
__global__ __launch_bounds__(DR) void draft_head_out_kernel(DraftArgs a, StepMeta meta) {
  __shared__ float red[32];
  const int r = blockIdx.x, d = a.d;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  float pv[RV], qv[RV];
#pragma unroll
  for (int j = 0; j < RV; ++j) pv[j] = qv[j] = 0.f;
  if (live) {
    add_parts(pv, a.parts, a.n_parts_h, a.stride_h, (long long)r * 2 * d, d);
    add_parts(qv, a.parts, a.n_parts_h, a.stride_h, (long long)r * 2 * d + d, d);
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < RV; ++j) {
    const int k = threadIdx.x + j * DR;
    if (k < d) {
      pv[j] = live ? pv[j] + bf16_to_f32(a.b_p[k]) : 0.f;
      a.feat_p[(long long)r * d + k] = pv[j];
      if (live) a.feat_r[(long long)r * d + k] = qv[j] + bf16_to_f32(a.b_r[k]);
      ss += pv[j] * pv[j];
    }
  }
  const float inv = rsqrtf(block_sum2(ss, 0.f, red).x / d + a.rms_eps);
#pragma unroll
  for (int j = 0; j < RV; ++j) {
    const int k = threadIdx.x + j * DR;
    if (k < d) put_split(a.xn, xpack_off(r, k, a.xn_ks), live ? pv[j] * inv * bf16_to_f32(a.final_norm[k]) : 0.f);
  }
}

// Top-k tokens (value descending, lower id first on ties) and their
// log-probabilities log softmax.  Two launches, so that a handful of rows
// still fills the chip: first every (row, vocabulary slice) workgroup holds
// its slice in registers (32 logits a thread) and writes the slice's k best
// candidates in order plus its maximum and sum of exp; then one wave per row
// combines the slices' log-sum-exp and merges their sorted lists.
constexpr int DK = 16;       // largest k
constexpr int TS = 256;      // threads per slice workgroup
constexpr int TE = 32;       // logits per thread
constexpr int SLICE_MAX = TS * TE;
constexpr int MAX_SLICES = 64;
constexpr int PART_WORDS = 2 * DK + 2;  // values, ids, maximum, sum of exp

__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

__host__ __device__ __forceinline__ int topk_slices(int V) { return (V + SLICE_MAX - 1) / SLICE_MAX; }
__host__ __device__ __forceinline__ int topk_slice_len(int V) {
  const int s = topk_slices(V);
  return ((V + s - 1) / s + 3) & ~3;
}

template <bool VEC>
__global__ __launch_bounds__(TS) void draft_topk_slice_kernel(const float* logits, long long ld, int V, StepMeta meta,
                                                             int rows, int max_tree, int k, float* part) {
  __shared__ float wv[2][TS / 64], red[16];
  __shared__ int wi[2][TS / 64];
  const int r = blockIdx.x, slice = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (!draft_live(meta, r, rows, max_tree)) return;  // uniform
  const int len = topk_slice_len(V), lo = slice * len, hi = min(V, lo + len);
  const float* lg = logits + (long long)r * ld;
  float x[TE];
  unsigned taken = 0;  // bit j: element j is outside the slice or already chosen
  auto id_of = [&](int j) { return VEC ? lo + 4 * (tid + (j >> 2) * TS) + (j & 3) : lo + tid + j * TS; };
  if (VEC) {
    const float4* l4 = reinterpret_cast<const float4*>(lg + lo);
#pragma unroll
    for (int q = 0; q < TE / 4; ++q) {
      const int at = lo + 4 * (tid + q * TS);
      const float4 v = at < hi ? l4[tid + q * TS] : make_float4(0.f, 0.f, 0.f, 0.f);
      x[4 * q] = v.x;
      x[4 * q + 1] = v.y;
      x[4 * q + 2] = v.z;
      x[4 * q + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < TE; ++j) {
      const int at = lo + tid + j * TS;
      x[j] = at < hi ? lg[at] : 0.f;
    }
  }
#pragma unroll
  for (int j = 0; j < TE; ++j)
    if (id_of(j) >= hi) taken |= 1u << j;
  // the slice's maximum and sum of exp (fixed order)
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < TE; ++j)
    if (!(taken >> j & 1)) m = fmaxf(m, x[j]);
  m = wave_max(m);
  __syncthreads();
  if (lane == 0) red[wave] = m;
  __syncthreads();
  float M = red[0];
  for (int w = 1; w < TS / 64; ++w) M = fmaxf(M, red[w]);
  float e = 0.f;
  if (M > -INFINITY) {
#pragma unroll
    for (int j = 0; j < TE; ++j)
      if (!(taken >> j & 1)) e += expf(x[j] - M);
  }
  const float S = block_sum(e, red);
  float* out = part + ((long long)r * gridDim.y + slice) * PART_WORDS;
  if (tid == 0) {
    out[2 * DK] = M;
    out[2 * DK + 1] = S;
  }
  // k rounds of a block-wide argmax; the owner of the winner drops it
  float bv = -INFINITY;
  int bi = 0x7fffffff, bj = -1;
  auto rescan = [&]() {
    bv = -INFINITY;
    bi = 0x7fffffff;
    bj = -1;
#pragma unroll
    for (int j = 0; j < TE; ++j)
      if (!(taken >> j & 1) && better(x[j], id_of(j), bv, bi)) {
        bv = x[j];
        bi = id_of(j);
        bj = j;
      }
  };
  rescan();
  for (int round = 0; round < k; ++round) {
    float v = bv;
    int i = bi;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(v, o, 64);
      const int oi = __shfl_xor(i, o, 64);
      if (better(ov, oi, v, i)) {
        v = ov;
        i = oi;
      }
    }
    const int buf = round & 1;  // two buffers: round r + 2 writes after every reader of round r passed round r + 1's barrier
    if (lane == 0) {
      wv[buf][wave] = v;
      wi[buf][wave] = i;
    }
    __syncthreads();
    float gv = wv[buf][0];
    int gi = wi[buf][0];
    for (int w = 1; w < TS / 64; ++w)
      if (better(wv[buf][w], wi[buf][w], gv, gi)) {
        gv = wv[buf][w];
        gi = wi[buf][w];
      }
    if (tid == 0) {
      out[round] = gv;
      out[DK + round] = __int_as_float(gi);
    }
    if (bj >= 0 && bi == gi) {  // ids are unique: this thread held the winner
      taken |= 1u << bj;
      rescan();
    }
  }
}

__global__ __launch_bounds__(64) void draft_topk_merge_kernel(const float* part, int nslice, StepMeta meta, int rows,
                                                             int max_tree, int k, int32_t* tok_out, float* logp_out) {
  __shared__ float cv[MAX_SLICES * DK];
  __shared__ int ci[MAX_SLICES * DK];
  const int r = blockIdx.x, lane = threadIdx.x;
  if (!draft_live(meta, r, rows, max_tree)) return;  // uniform
  const float* pr = part + (long long)r * nslice * PART_WORDS;
  const float Ms = lane < nslice ? pr[lane * PART_WORDS + 2 * DK] : -INFINITY;
  const float Ss = lane < nslice ? pr[lane * PART_WORDS + 2 * DK + 1] : 0.f;
  const float M = wave_max(Ms);
  const float lse = M + logf(wave_sum(Ms > -INFINITY ? Ss * expf(Ms - M) : 0.f));
  for (int q = lane; q < nslice * k; q += 64) {
    cv[q] = pr[(q / k) * PART_WORDS + q % k];
    ci[q] = __float_as_int(pr[(q / k) * PART_WORDS + DK + q % k]);
  }
  __syncthreads();
  int head = 0;  // this lane's slice: next candidate of its sorted list
  for (int round = 0; round < k; ++round) {
    float v = lane < nslice && head < k ? cv[lane * k + head] : -INFINITY;
    int i = lane < nslice && head < k ? ci[lane * k + head] : 0x7fffffff, w = lane;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(v, o, 64);
      const int oi = __shfl_xor(i, o, 64), ow = __shfl_xor(w, o, 64);
      if (better(ov, oi, v, i)) {
        v = ov;
        i = oi;
        w = ow;
      }
    }
    if (lane == 0) {
      tok_out[(long long)r * k + round] = i;
      logp_out[(long long)r * k + round] = v - lse;
    }
    if (lane == w) ++head;
  }
}

hipError_t launch_draft_front(const DraftArgs& a, const StepMeta& meta, int stage, hipStream_t s) {
  const dim3 g(a.mpad);
  switch (stage) {
    case 0: hipLaunchKernelGGL(draft_in_kernel, dim3(a.mpad, 8), dim3(DT), 0, s, a, meta); break;
    case 1: hipLaunchKernelGGL(draft_fuse_kernel, g, dim3(DR), 0, s, a, meta); break;
    case 2: hipLaunchKernelGGL(draft_silu_kernel, dim3(a.mpad, 16), dim3(DT), 0, s, a, meta); break;
    case 3: hipLaunchKernelGGL(draft_out_kernel, dim3(a.mpad, 8), dim3(DT), 0, s, a, meta); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_draft_head(const DraftArgs& a, const StepMeta& meta, const ResidualAdd& add, int stage,
                             hipStream_t s) {
  if (add.slot != nullptr) return hipErrorInvalidValue;  // dense decoder layer only
  if (stage == 0)
    hipLaunchKernelGGL(draft_head_in_kernel, dim3(a.mpad, 8), dim3(DT), 0, s, a, meta, add);
  else
    hipLaunchKernelGGL(draft_head_out_kernel, dim3(a.mpad), dim3(DR), 0, s, a, meta);
  return hipGetLastError();
}

size_t draft_topk_work_bytes(int rows, int V) {
  return sizeof(float) * (size_t)rows * topk_slices(V) * PART_WORDS;
}

hipError_t launch_draft_topk(const float* logits, long long ld, int V, const StepMeta& meta, int rows, int max_tree,
                             int k, int32_t* tok, float* logp, float* work, hipStream_t s) {
  if (k < 1 || k > DK || V < k || topk_slices(V) > MAX_SLICES) return hipErrorInvalidValue;
  const int ns = topk_slices(V);
  if ((V & 3) == 0 && (ld & 3) == 0)  // 16-byte aligned rows and slices
    hipLaunchKernelGGL(draft_topk_slice_kernel<true>, dim3(rows, ns), dim3(TS), 0, s, logits, ld, V, meta, rows,
                       max_tree, k, work);
  else
    hipLaunchKernelGGL(draft_topk_slice_kernel<false>, dim3(rows, ns), dim3(TS), 0, s, logits, ld, V, meta, rows,
                       max_tree, k, work);
  hipLaunchKernelGGL(draft_topk_merge_kernel, dim3(rows), dim3(64), 0, s, work, ns, meta, rows, max_tree, k, tok,
                     logp);
  return hipGetLastError();
}

// ------------------------------------------------------------ tree expansion

// Ranking key of a candidate score: NaN counts as the lowest score.
__device__ __forceinline__ double sel_key(double s) { return s != s ? -INFINITY : s; }
// Candidate a (score sa) ranks before candidate b: higher score, then lower index.
__device__ __forceinline__ bool sel_before(double sa, int a, double sb, int b) {
  return sa > sb || (sa == sb && a < b);
}

constexpr int SEL_T = 1024;  // one thread per candidate of the last pass (four waves per SIMD)
constexpr int SEL_U = 16;    // candidates compared per batch of LDS reads

// Rank of candidate q (key s) among the n candidates keyed sc[0, n): how many
// rank before it.  The reads are batched so that their LDS latencies overlap.
__device__ __forceinline__ int sel_rank(const double* sc, int n, double s, int q) {
  int rk = 0, o = 0;
  for (; o + SEL_U <= n; o += SEL_U) {
    double v[SEL_U];
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) v[u] = sc[o + u];
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) rk += sel_before(v[u], o + u, s, q);
  }
  for (; o < n; ++o) rk += sel_before(sc[o], o, s, q);
  return rk;
}

__global__ __launch_bounds__(SEL_T) void draft_select_kernel(DraftSelectArgs a) {
  __shared__ double sc[DRAFT_SEL_MAX];  // ranking keys of the candidates
  __shared__ int slot[DRAFT_SEL_MAX];   // last pass: output row - 1 of a kept candidate, else -1
  __shared__ int dep[DRAFT_SEL_MAX];    // last pass: depth of a candidate
  __shared__ int kept[64], kdep[64];    // last pass: kept candidates by rank, their depths
  const int b = blockIdx.x, tid = threadIdx.x, k = a.k, T = a.max_tree, t = a.t;
  // the frontier of pass t: the root, or the k nodes the previous pass added
  const int f0 = t == 0 ? 0 : 1 + k * (t - 1), nf = (t == 0 ? 1 : k) * k;
  const int c0 = t == 0 ? 0 : k + k * k * (t - 1);  // index of the first fresh candidate
  const long long cb = (long long)b * DRAFT_SEL_MAX, nb = (long long)b * T;
  for (int q = tid; q < nf; q += SEL_T) {
    const int r = f0 + q / k;
    const long long at = (nb + r) * k + q % k;
    const double s = (r == 0 ? 0.0 : a.n_score[nb + r]) + (double)a.topk_lp[at];
    a.c_tok[cb + c0 + q] = a.topk_tok[at];
    a.c_node[cb + c0 + q] = r;
    a.c_score[cb + c0 + q] = s;
    sc[c0 + q] = sel_key(s);
  }
  if (t + 1 < a.depth) {
    __syncthreads();
    // the k best fresh candidates become pass-tree nodes 1 + k t + rank
    for (int q = tid; q < nf; q += SEL_T) {
      const int rk = sel_rank(sc + c0, nf, sc[c0 + q], q);
      if (rk < k) {
        const int node = 1 + k * t + rk, r = f0 + q / k;
        a.n_cand[nb + node] = c0 + q;
        a.n_score[nb + node] = a.c_score[cb + c0 + q];
        a.m_token[nb + node] = a.c_tok[cb + c0 + q];
        a.m_parent[nb + node] = r;
        a.m_anc[nb + node] = a.m_anc[nb + r] | (1ull << node);
      }
    }
    for (int w = b * SEL_T + tid; w < a.tail_words; w += gridDim.x * SEL_T) a.tail_dst[w] = a.tail_src[w];
    return;
  }
  // last pass: the n_total best of all candidates, numbered by depth, then rank
  const int nc = c0 + nf, keep = min(nc, a.n_total);
  for (int q = tid; q < nc; q += SEL_T) {
    if (q < c0) sc[q] = sel_key(a.c_score[cb + q]);
    dep[q] = q < k ? 1 : 2 + (q - k) / (k * k);
    slot[q] = -1;
  }
  __syncthreads();
  for (int q = tid; q < nc; q += SEL_T) {
    const int rk = sel_rank(sc, nc, sc[q], q);
    if (rk < keep) {  // ranks are distinct
      kept[rk] = q;
      kdep[rk] = dep[q];
    }
  }
  __syncthreads();
  if (tid < keep) {
    const int dq = kdep[tid];
    int at = 0;
    for (int j = 0; j < keep; ++j) at += kdep[j] < dq || (kdep[j] == dq && j < tid);
    slot[kept[tid]] = at;
  }
  __syncthreads();
  if (tid < keep) {
    const int q = kept[tid], at = slot[q];
    const int r = a.c_node[cb + q];
    const int pc = r == 0 ? -1 : a.n_cand[nb + r];
    a.o_tok[nb + at + 1] = a.c_tok[cb + q];
    a.o_par[nb + at + 1] = pc < 0 ? 0 : slot[pc] + 1;
    a.o_score[nb + at + 1] = (float)a.c_score[cb + q];
  }
  if (tid == 0) {
    a.o_nodes[b] = 1 + keep;
    a.o_tok[nb] = a.m_token[nb];
    a.o_par[nb] = -1;
    a.o_score[nb] = 0.f;
  }
}

hipError_t launch_draft_select(const DraftSelectArgs& a, int batch, hipStream_t s) {
  if (a.k < 1 || a.k > DK || a.t < 0 || a.t >= a.depth || a.max_tree > 64 || 1 + a.k * (a.depth - 1) > a.max_tree ||
      a.k * (1 + a.k * (a.depth - 1)) > DRAFT_SEL_MAX || a.n_total < 1 || a.n_total > 63 || batch < 1)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(draft_select_kernel, dim3(batch), dim3(SEL_T), 0, s, a);
  return hipGetLastError();
}

}  // namespace griffin
