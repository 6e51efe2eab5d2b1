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
// caller's).

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
  const float* f = i == 0 ? a.root_feat + (long long)b * d
                          : a.feat_r + ((long long)b * a.max_tree + meta.parent[min(r, a.rows - 1)]) * d;
  const uint16_t* e = a.embed + (long long)meta.token[min(r, a.rows - 1)] * d;
  for (int k = blockIdx.y * DT + threadIdx.x; k < 2 * d; k += gridDim.y * DT) {
    const float v = !live ? 0.f : (k < d ? f[k] : bf16_to_f32(e[k - d]));
    put_split(a.x_m, xpack_off(r, k, a.ks_m), v);
  }
}

// h = sum of the W_m partials + b_m (kept), then [LN(h), LN(e)] as the
// operand of W_u (K = 2d).
__global__ __launch_bounds__(DR) void draft_fuse_kernel(DraftArgs a, StepMeta meta) {
  __shared__ float red[16];
  const int r = blockIdx.x, d = a.d;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  float* h = a.h + (long long)r * d;
  const uint16_t* e = a.embed + (long long)meta.token[min(r, a.rows - 1)] * d;
  float sh = 0.f, se = 0.f;
  for (int k = threadIdx.x; k < d; k += DR) {
    const float v = live ? sum_parts(a.parts, a.n_parts_m, a.stride_m, (long long)r * d + k) + bf16_to_f32(a.b_m[k])
                         : 0.f;
    h[k] = v;
    sh += v;
    se += bf16_to_f32(e[k]);
  }
  const float mh = dblock_sum(sh, red) / d, me = dblock_sum(se, red) / d;
  float vh = 0.f, ve = 0.f;
  for (int k = threadIdx.x; k < d; k += DR) {
    const float dh = h[k] - mh, de = bf16_to_f32(e[k]) - me;
    vh += dh * dh;
    ve += de * de;
  }
  const float rh = rsqrtf(dblock_sum(vh, red) / d + a.ln_eps), re = rsqrtf(dblock_sum(ve, red) / d + a.ln_eps);
  for (int k = threadIdx.x; k < d; k += DR) {
    const float lh = (h[k] - mh) * rh * bf16_to_f32(a.ln_h_g[k]) + bf16_to_f32(a.ln_h_b[k]);
    const float le = (bf16_to_f32(e[k]) - me) * re * bf16_to_f32(a.ln_x_g[k]) + bf16_to_f32(a.ln_x_b[k]);
    put_split(a.x_u, xpack_off(r, k, a.ks_u), live ? lh : 0.f);
    put_split(a.x_u, xpack_off(r, d + k, a.ks_u), live ? le : 0.f);
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
  __shared__ float red[16];
  const int r = blockIdx.x, d = a.d;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  float* fp = a.feat_p + (long long)r * d;
  float* fr = a.feat_r + (long long)r * d;
  float ss = 0.f;
  for (int k = threadIdx.x; k < d; k += DR) {
    const long long at = (long long)r * 2 * d + k;
    const float p = live ? sum_parts(a.parts, a.n_parts_h, a.stride_h, at) + bf16_to_f32(a.b_p[k]) : 0.f;
    const float q = live ? sum_parts(a.parts, a.n_parts_h, a.stride_h, at + d) + bf16_to_f32(a.b_r[k]) : 0.f;
    fp[k] = p;
    if (live) fr[k] = q;
    ss += p * p;
  }
  const float inv = rsqrtf(dblock_sum(ss, red) / d + a.rms_eps);
  for (int k = threadIdx.x; k < d; k += DR)
    put_split(a.xn, xpack_off(r, k, a.xn_ks), live ? fp[k] * inv * bf16_to_f32(a.final_norm[k]) : 0.f);
}

// Top-k tokens (value descending, lower id first on ties) and their
// log-probabilities log softmax, one workgroup per live row.  One pass over
// the row with several 16-byte loads in flight per thread: every thread keeps
// a sorted list of its best DK candidates and a running maximum and sum of
// exp (rescaled when the maximum grows); then k rounds of a block-wide argmax
// over the list heads pick the winners (ties: lower id).
constexpr int DK = 16;
constexpr int TK = 1024;  // threads per row
constexpr int TK_LOADS = 4;

__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

struct TopList {
  float v[DK];
  int i[DK];
  float m, s;  // running maximum, sum of exp(x - m)

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int j = 0; j < DK; ++j) {
      v[j] = -INFINITY;
      i[j] = 0x7fffffff;
    }
    m = -INFINITY;
    s = 0.f;
  }
  __device__ __forceinline__ void add(float x, int id) {
    const float mn = fmaxf(m, x);
    s = (mn == m ? s : s * expf(m - mn)) + (x > -INFINITY ? expf(x - mn) : 0.f);
    m = mn;
    if (better(x, id, v[DK - 1], i[DK - 1])) {  // insert, keeping the list sorted
      float cv = x;
      int ci = id;
#pragma unroll
      for (int j = 0; j < DK; ++j) {
        const bool b = better(cv, ci, v[j], i[j]);
        const float tv = v[j];
        const int ti = i[j];
        v[j] = b ? cv : tv;
        i[j] = b ? ci : ti;
        cv = b ? tv : cv;
        ci = b ? ti : ci;
      }
    }
  }
};

__global__ __launch_bounds__(TK) void draft_topk_kernel(const float* logits, long long ld, int V, StepMeta meta,
                                                       int rows, int max_tree, int k, int32_t* tok_out,
                                                       float* logp_out) {
  __shared__ float wv[TK / 64], wm[TK / 64], wsum[TK / 64];
  __shared__ int wi[TK / 64], ww[TK / 64];
  __shared__ int win_thread;
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (!draft_live(meta, r, rows, max_tree)) return;  // uniform
  const float* lg = logits + (long long)r * ld;
  TopList L;
  L.init();
  if ((V & 3) == 0) {
    const float4* l4 = reinterpret_cast<const float4*>(lg);
    const int n4 = V >> 2;
    for (int base = tid; base < n4; base += TK * TK_LOADS) {
      float4 x[TK_LOADS];
#pragma unroll
      for (int u = 0; u < TK_LOADS; ++u) {
        const int at = base + u * TK;
        x[u] = at < n4 ? l4[at] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      }
#pragma unroll
      for (int u = 0; u < TK_LOADS; ++u) {
        const int id = 4 * (base + u * TK);
        L.add(x[u].x, id);
        L.add(x[u].y, id + 1);
        L.add(x[u].z, id + 2);
        L.add(x[u].w, id + 3);
      }
    }
  } else {
    for (int v = tid; v < V; v += TK) L.add(lg[v], v);
  }
  // log-sum-exp over the row (fixed order: waves, then the waves' results)
  float M = wave_max(L.m);
  float S = wave_sum(L.m > -INFINITY ? L.s * expf(L.m - M) : 0.f);
  if (lane == 0) {
    wm[wave] = M;
    wsum[wave] = S;
  }
  __syncthreads();
  float gm = -INFINITY;
  for (int w = 0; w < TK / 64; ++w) gm = fmaxf(gm, wm[w]);
  float gs = 0.f;
  for (int w = 0; w < TK / 64; ++w) gs += wm[w] > -INFINITY ? wsum[w] * expf(wm[w] - gm) : 0.f;
  const float lse = gm + logf(gs);
  for (int round = 0; round < k; ++round) {
    // wave argmax of the list heads, then across the waves
    float bv = L.v[0];
    int bi = L.i[0], bt = tid;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int oi = __shfl_xor(bi, o, 64), ot = __shfl_xor(bt, o, 64);
      if (better(ov, oi, bv, bi)) {
        bv = ov;
        bi = oi;
        bt = ot;
      }
    }
    __syncthreads();  // the previous round's readers of wv/wi/ww are done
    if (lane == 0) {
      wv[wave] = bv;
      wi[wave] = bi;
      ww[wave] = bt;
    }
    __syncthreads();
    if (tid == 0) {
      float gv = wv[0];
      int gi = wi[0], gt = ww[0];
      for (int w = 1; w < TK / 64; ++w)
        if (better(wv[w], wi[w], gv, gi)) {
          gv = wv[w];
          gi = wi[w];
          gt = ww[w];
        }
      tok_out[(long long)r * k + round] = gi;
      logp_out[(long long)r * k + round] = gv - lse;
      win_thread = gt;
    }
    __syncthreads();
    if (tid == win_thread) {  // pop the head
#pragma unroll
      for (int j = 0; j < DK - 1; ++j) {
        L.v[j] = L.v[j + 1];
        L.i[j] = L.i[j + 1];
      }
      L.v[DK - 1] = -INFINITY;
      L.i[DK - 1] = 0x7fffffff;
    }
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

hipError_t launch_draft_topk(const float* logits, long long ld, int V, const StepMeta& meta, int rows, int max_tree,
                             int k, int32_t* tok, float* logp, hipStream_t s) {
  if (k < 1 || k > DK || V < k) return hipErrorInvalidValue;
  if ((V & 3) == 0 && (ld & 3) != 0) return hipErrorInvalidValue;  // rows must stay 16-byte aligned
  hipLaunchKernelGGL(draft_topk_kernel, dim3(rows), dim3(TK), 0, s, logits, ld, V, meta, rows, max_tree, k, tok,
                     logp);
  return hipGetLastError();
}

}  // namespace griffin
