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

constexpr int DT = 256;  // threads per workgroup

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
__global__ __launch_bounds__(DT) void draft_in_kernel(DraftArgs a, StepMeta meta) {
  const int r = blockIdx.x, d = a.d;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  const int b = r / a.max_tree, i = r % a.max_tree;
  const float* f = i == 0 ? a.root_feat + (long long)b * d
                          : a.feat_r + ((long long)b * a.max_tree + meta.parent[min(r, a.rows - 1)]) * d;
  const uint16_t* e = a.embed + (long long)meta.token[min(r, a.rows - 1)] * d;
  for (int k = threadIdx.x; k < 2 * d; k += DT) {
    const float v = !live ? 0.f : (k < d ? f[k] : bf16_to_f32(e[k - d]));
    put_split(a.x_m, xpack_off(r, k, a.ks_m), v);
  }
}

// h = sum of the W_m partials + b_m (kept), then [LN(h), LN(e)] as the
// operand of W_u (K = 2d).
__global__ __launch_bounds__(DT) void draft_fuse_kernel(DraftArgs a, StepMeta meta) {
  __shared__ float red[16];
  const int r = blockIdx.x, d = a.d;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  float* h = a.h + (long long)r * d;
  const uint16_t* e = a.embed + (long long)meta.token[min(r, a.rows - 1)] * d;
  float sh = 0.f, se = 0.f;
  for (int k = threadIdx.x; k < d; k += DT) {
    const float v = live ? sum_parts(a.parts, a.n_parts_m, a.stride_m, (long long)r * d + k) + bf16_to_f32(a.b_m[k])
                         : 0.f;
    h[k] = v;
    sh += v;
    se += bf16_to_f32(e[k]);
  }
  const float mh = dblock_sum(sh, red) / d, me = dblock_sum(se, red) / d;
  float vh = 0.f, ve = 0.f;
  for (int k = threadIdx.x; k < d; k += DT) {
    const float dh = h[k] - mh, de = bf16_to_f32(e[k]) - me;
    vh += dh * dh;
    ve += de * de;
  }
  const float rh = rsqrtf(dblock_sum(vh, red) / d + a.ln_eps), re = rsqrtf(dblock_sum(ve, red) / d + a.ln_eps);
  for (int k = threadIdx.x; k < d; k += DT) {
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
__global__ __launch_bounds__(DT) void draft_head_out_kernel(DraftArgs a, StepMeta meta) {
  __shared__ float red[16];
  const int r = blockIdx.x, d = a.d;
  const bool live = draft_live(meta, r, a.rows, a.max_tree);
  float* fp = a.feat_p + (long long)r * d;
  float* fr = a.feat_r + (long long)r * d;
  float ss = 0.f;
  for (int k = threadIdx.x; k < d; k += DT) {
    const long long at = (long long)r * 2 * d + k;
    const float p = live ? sum_parts(a.parts, a.n_parts_h, a.stride_h, at) + bf16_to_f32(a.b_p[k]) : 0.f;
    const float q = live ? sum_parts(a.parts, a.n_parts_h, a.stride_h, at + d) + bf16_to_f32(a.b_r[k]) : 0.f;
    fp[k] = p;
    if (live) fr[k] = q;
    ss += p * p;
  }
  const float inv = rsqrtf(dblock_sum(ss, red) / d + a.rms_eps);
  for (int k = threadIdx.x; k < d; k += DT)
    put_split(a.xn, xpack_off(r, k, a.xn_ks), live ? fp[k] * inv * bf16_to_f32(a.final_norm[k]) : 0.f);
}

// Top-k tokens (value descending, lower id first on ties) and their
// log-probabilities log softmax, one workgroup per live row.  Every thread
// keeps a sorted list of its best DK candidates; k rounds of a block-wide
// argmax over the list heads pick the winners.
constexpr int DK = 16;

__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

__global__ __launch_bounds__(DT) void draft_topk_kernel(const float* logits, long long ld, int V, StepMeta meta,
                                                       int rows, int max_tree, int k, int32_t* tok_out,
                                                       float* logp_out) {
  __shared__ float sv[DT];
  __shared__ int si[DT], st[DT];
  __shared__ float red[16];
  const int r = blockIdx.x, tid = threadIdx.x;
  if (!draft_live(meta, r, rows, max_tree)) return;  // uniform
  const float* lg = logits + (long long)r * ld;
  float bv[DK];
  int bi[DK];
#pragma unroll
  for (int j = 0; j < DK; ++j) {
    bv[j] = -INFINITY;
    bi[j] = 0x7fffffff;
  }
  float mx = -INFINITY;
  for (int v = tid; v < V; v += DT) {
    const float x = lg[v];
    mx = fmaxf(mx, x);
    if (better(x, v, bv[DK - 1], bi[DK - 1])) {  // insert, keeping the list sorted
      float cv = x;
      int ci = v;
#pragma unroll
      for (int j = 0; j < DK; ++j) {
        if (better(cv, ci, bv[j], bi[j])) {
          const float tv = bv[j];
          const int ti = bi[j];
          bv[j] = cv;
          bi[j] = ci;
          cv = tv;
          ci = ti;
        }
      }
    }
  }
  // log-sum-exp over the row (fixed order)
  mx = wave_max(mx);
  __syncthreads();
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  float M = -INFINITY;
  for (int w = 0; w < DT / 64; ++w) M = fmaxf(M, red[w]);
  float s = 0.f;
  for (int v = tid; v < V; v += DT) s += expf(lg[v] - M);
  const float lse = M + logf(dblock_sum(s, red));
  int head = 0;
  for (int round = 0; round < k; ++round) {
    sv[tid] = head < DK ? bv[0] : -INFINITY;
    si[tid] = head < DK ? bi[0] : 0x7fffffff;
    st[tid] = tid;
    __syncthreads();
    for (int off = DT / 2; off > 0; off >>= 1) {
      if (tid < off && better(sv[tid + off], si[tid + off], sv[tid], si[tid])) {
        sv[tid] = sv[tid + off];
        si[tid] = si[tid + off];
        st[tid] = st[tid + off];
      }
      __syncthreads();
    }
    const int win = st[0];
    if (tid == 0) {
      tok_out[(long long)r * k + round] = si[0];
      logp_out[(long long)r * k + round] = sv[0] - lse;
    }
    __syncthreads();
    if (tid == win) {  // pop the head
#pragma unroll
      for (int j = 0; j < DK - 1; ++j) {
        bv[j] = bv[j + 1];
        bi[j] = bi[j + 1];
      }
      bv[DK - 1] = -INFINITY;
      bi[DK - 1] = 0x7fffffff;
      ++head;
    }
  }
}

hipError_t launch_draft_front(const DraftArgs& a, const StepMeta& meta, int stage, hipStream_t s) {
  const dim3 g(a.mpad);
  switch (stage) {
    case 0: hipLaunchKernelGGL(draft_in_kernel, g, dim3(DT), 0, s, a, meta); break;
    case 1: hipLaunchKernelGGL(draft_fuse_kernel, g, dim3(DT), 0, s, a, meta); break;
    case 2: hipLaunchKernelGGL(draft_silu_kernel, dim3(a.mpad, 4), dim3(DT), 0, s, a, meta); break;
    case 3: hipLaunchKernelGGL(draft_out_kernel, dim3(a.mpad, 2), dim3(DT), 0, s, a, meta); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_draft_head(const DraftArgs& a, const StepMeta& meta, const ResidualAdd& add, int stage,
                             hipStream_t s) {
  if (add.slot != nullptr) return hipErrorInvalidValue;  // dense decoder layer only
  if (stage == 0)
    hipLaunchKernelGGL(draft_head_in_kernel, dim3(a.mpad, 2), dim3(DT), 0, s, a, meta, add);
  else
    hipLaunchKernelGGL(draft_head_out_kernel, dim3(a.mpad), dim3(DT), 0, s, a, meta);
  return hipGetLastError();
}

hipError_t launch_draft_topk(const float* logits, long long ld, int V, const StepMeta& meta, int rows, int max_tree,
                             int k, int32_t* tok, float* logp, hipStream_t s) {
  if (k < 1 || k > DK || V < k) return hipErrorInvalidValue;
  hipLaunchKernelGGL(draft_topk_kernel, dim3(rows), dim3(DT), 0, s, logits, ld, V, meta, rows, max_tree, k, tok,
                     logp);
  return hipGetLastError();
}

}  // namespace griffin
