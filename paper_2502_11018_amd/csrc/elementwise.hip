// Row-wise kernels of the verify pass: embedding gather, residual update +
// RMSNorm, rotary embedding + tree K/V write, vocab argmax reduction, the
// acceptance walk and the MoE router.  All reductions use fixed orders, so
// repeated runs give identical bits.

#include "device_common.h"
#include "griffin_internal.h"

namespace griffin {

// ------------------------------------------------------------- embedding ----
// x[r][:] = E[token[r]][:] as fp32; one workgroup per row.
__global__ __launch_bounds__(256) void embed_kernel(const uint16_t* __restrict__ E, const int32_t* token,
                                                    int d, float* __restrict__ x) {
  const int r = blockIdx.x;
  const uint16_t* src = E + (long long)token[r] * d;
  float* dst = x + (long long)r * d;
  for (int j = threadIdx.x * 4; j < d; j += blockDim.x * 4) {
    const uint2 v = *reinterpret_cast<const uint2*>(src + j);
    *reinterpret_cast<float4*>(dst + j) =
        make_float4(bf16_to_f32(v.x & 0xffff), bf16_to_f32(v.x >> 16), bf16_to_f32(v.y & 0xffff),
                    bf16_to_f32(v.y >> 16));
  }
}

hipError_t launch_embed(const uint16_t* embed, const int32_t* token, int rows, int d, float* x, hipStream_t s) {
  hipLaunchKernelGGL(embed_kernel, dim3(rows), dim3(256), 0, s, embed, token, d, x);
  return hipGetLastError();
}

// ------------------------------------------------ residual update + RMSNorm ----
// x[r] += (split partial sums | weighted MoE expert outputs); then
// xn[r] = bf16(x[r] * rsqrt(mean(x[r]^2) + eps) * gain).
// 1024 threads per row, each owning GPT float4 groups of the row.  The number
// of dense partials NP is a template parameter so that every load of the row
// is issued before the first one is waited on (no branches between loads);
// NP < 0 selects the MoE form (per-row expert slots).
constexpr int RN_THREADS = 1024;  // measured against 256 and 512 (one row per workgroup either way)
constexpr int RN_SPLITS = 16;  // K-split partials per residual update

__device__ __forceinline__ void add4(float4& a, const float4& p) {
  a.x += p.x; a.y += p.y; a.z += p.z; a.w += p.w;
}

// The router epilogue of the norm kernel (Router): this thread's GPT groups
// of 4 normed values h, 8 experts per reduction round.
constexpr int ROUTE_EC = 8;  // experts per reduction round of the router epilogue

// Router weights of this thread's elements for experts e0 .. e0 + 7 (zero
// past n_experts), loaded early so that their latency overlaps the norm.
template <int GPT>
__device__ __forceinline__ void route_load(const Router& rt, int e0, int d, const int (&gi)[GPT],
                                           uint2 (&ww)[ROUTE_EC][GPT]) {
#pragma unroll
  for (int q = 0; q < ROUTE_EC; ++q)
#pragma unroll
    for (int u = 0; u < GPT; ++u)
      ww[q][u] = e0 + q < rt.n_experts ? *reinterpret_cast<const uint2*>(rt.w + (long long)(e0 + q) * d + 4 * gi[u])
                                       : make_uint2(0u, 0u);
}

// Sum 8 values over the 64 lanes of a wave with 10 shuffles: each exchange
// halves the values a lane carries; lane l ends with the sum of value
// (l >> 3) & 7 (as the 3 bits of lane l's positions 32, 16, 8 select it).
__device__ __forceinline__ float wave_sum8(const float (&v)[8]) {
  const int lane = threadIdx.x & 63;
  float a4[4];
  const bool h32 = lane & 32;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float send = h32 ? v[i] : v[i + 4], keep = h32 ? v[i + 4] : v[i];
    a4[i] = keep + __shfl_xor(send, 32, 64);
  }
  float a2[2];
  const bool h16 = lane & 16;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float send = h16 ? a4[i] : a4[i + 2], keep = h16 ? a4[i + 2] : a4[i];
    a2[i] = keep + __shfl_xor(send, 16, 64);
  }
  const bool h8 = lane & 8;
  float a1 = (h8 ? a2[1] : a2[0]) + __shfl_xor(h8 ? a2[0] : a2[1], 8, 64);
  a1 += __shfl_xor(a1, 4, 64);
  a1 += __shfl_xor(a1, 2, 64);
  a1 += __shfl_xor(a1, 1, 64);
  return a1;  // lane l: value index 4 * [l & 32] + 2 * [l & 16] + [l & 8]
}

template <int GPT>
__device__ __forceinline__ void route_row(const Router& rt, int r, const float4 (&h)[GPT], const int (&gi)[GPT],
                                          const bool (&ok)[GPT], int d, const uint2 (&w0)[ROUTE_EC][GPT]) {
  constexpr int EC = ROUTE_EC;
  __shared__ float part[RN_THREADS / 64][EC];
  __shared__ float logit[64];
  __shared__ int dest[4];  // dispatch: the row's place (expert tile row) for each kept expert
  __shared__ int kept[4];  // kept experts by rank, and their unnormalised probabilities
  __shared__ float kept_p[4];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int b = r / rt.max_tree, i = r % rt.max_tree;
  if (r >= rt.rows) {  // padding row (uniform)
    if (rt.count && r < rt.padded_rows && tid < rt.top_k) rt.slot[r * rt.top_k + tid] = -1;
    return;
  }
  if (i >= rt.n_nodes[b]) {  // absent node (uniform)
    if (tid < rt.top_k) {
      rt.ids[r * rt.top_k + tid] = -1;
      rt.weights[r * rt.top_k + tid] = 0.f;
      if (rt.count) rt.slot[r * rt.top_k + tid] = -1;
    }
    return;
  }
  for (int e0 = 0; e0 < rt.n_experts; e0 += EC) {
    uint2 wl[EC][GPT];
    if (e0 == 0) {
#pragma unroll
      for (int q = 0; q < EC; ++q)
#pragma unroll
        for (int u = 0; u < GPT; ++u) wl[q][u] = w0[q][u];
    } else {
      route_load<GPT>(rt, e0, d, gi, wl);
    }
    float acc[EC];
#pragma unroll
    for (int q = 0; q < EC; ++q) {
      acc[q] = 0.f;
#pragma unroll
      for (int u = 0; u < GPT; ++u)
        if (ok[u]) {
          const uint2 ww = wl[q][u];
          acc[q] += h[u].x * bf16_to_f32(ww.x & 0xffff) + h[u].y * bf16_to_f32(ww.x >> 16) +
                    h[u].z * bf16_to_f32(ww.y & 0xffff) + h[u].w * bf16_to_f32(ww.y >> 16);
        }
    }
    const float wsum = wave_sum8(acc);
    __syncthreads();
    if ((lane & 7) == 0) part[w][((lane >> 5) & 1) * 4 + ((lane >> 4) & 1) * 2 + ((lane >> 3) & 1)] = wsum;
    __syncthreads();
    if (tid < EC && e0 + tid < rt.n_experts) {
      float t = 0.f;
      for (int k = 0; k < RN_THREADS / 64; ++k) t += part[k][tid];  // fixed order
      logit[e0 + tid] = t;
    }
  }
  __syncthreads();
  if (tid < rt.n_experts) rt.logits[(long long)r * rt.n_experts + tid] = logit[tid];
  if (tid < 4) {  // every kept slot defined, whatever the logits hold
    kept[tid] = 0;
    kept_p[tid] = 0.f;
  }
  __syncthreads();
  if (tid < 64) {  // wave 0: softmax and top-k, one lane per expert
    const int n = rt.n_experts;
    const float lg = tid < n ? logit[tid] : -INFINITY;
    const float mx = wave_max(lg);
    const float p = tid < n ? __expf(lg - mx) : -1.f;  // unnormalised probability; -1 is never kept
    // place of this expert in (probability descending, id ascending)
    int rank = 0;
    for (int e = 0; e < n; ++e) {
      const float pe = __shfl(p, e, 64);
      rank += pe > p || (pe == p && e < tid);
    }
    if (tid < n && rank < rt.top_k) {
      kept[rank] = tid;
      kept_p[rank] = p;
    }
  }
  __syncthreads();
  if (tid < rt.top_k) {
    float tot = 0.f;
    for (int k = 0; k < rt.top_k; ++k) tot += kept_p[k];  // rank order
    const int e = min(max(kept[tid], 0), rt.n_experts - 1);
    rt.ids[r * rt.top_k + tid] = e;
    rt.weights[r * rt.top_k + tid] = kept_p[tid] / tot;
    if (rt.count) {
      const int place = __hip_atomic_fetch_add(rt.count + e, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // place < cap unless NaN logits kept one expert twice (then dropped)
      const int row = place < rt.cap ? e * rt.cap + place : -1;
      rt.slot[r * rt.top_k + tid] = row;
      dest[tid] = row;
    }
  }
  if (rt.count) {  // the row's packed operand to its place in each kept expert's tiles (uniform branch)
    __syncthreads();
    for (int k = 0; k < rt.top_k; ++k) {
      const int row = dest[k];
      if (row < 0) continue;  // uniform
#pragma unroll
      for (int u = 0; u < GPT; ++u)
        if (ok[u]) {
          const Hilo2 p0 = pack_hilo2(h[u].x, h[u].y), p1 = pack_hilo2(h[u].z, h[u].w);
          uint16_t* dst = rt.xe + xpack_off(row, 4 * gi[u], rt.xe_ks);
          *reinterpret_cast<uint2*>(dst) = make_uint2(p0.hi, p1.hi);
          *reinterpret_cast<uint2*>(dst + XPACK_LO) = make_uint2(p0.lo, p1.lo);
        }
    }
  }
}

template <int NP, int GPT>
__global__ __launch_bounds__(RN_THREADS) void residual_rmsnorm_kernel(float* __restrict__ x, ResidualAdd add,
                                                                      const uint16_t* __restrict__ gain,
                                                                      float eps, int d,
                                                                      uint16_t* __restrict__ xn, int xn_ks,
                                                                      Router rt) {
  __shared__ float red[16];
  const int r = blockIdx.x;
  if (rt.clear && r == 0 && threadIdx.x < rt.n_clear) rt.clear[threadIdx.x] = 0;
  float* __restrict__ xr = x + (long long)r * d;
  const float* __restrict__ parts = add.parts;
  const int groups = d >> 2;
  int gi[GPT];
  bool ok[GPT];
  float4 v[GPT];
#pragma unroll
  for (int u = 0; u < GPT; ++u) {
    const int g = threadIdx.x + u * RN_THREADS;
    ok[u] = g < groups;
    gi[u] = ok[u] ? g : groups - 1;  // clamped: loads stay unconditional
    v[u] = reinterpret_cast<const float4*>(xr)[gi[u]];
  }
  uint2 gg[GPT];  // gains, in flight with the row
#pragma unroll
  for (int u = 0; u < GPT; ++u) gg[u] = *reinterpret_cast<const uint2*>(gain + 4 * gi[u]);
  uint2 w0[ROUTE_EC][GPT];  // MoE: the first router weights, in flight during the norm
  if (rt.w) route_load<GPT>(rt, 0, d, gi, w0);
  if constexpr (NP > 0) {
    // dense: K-split partial sums, all loaded first, added in split order
    float4 p[NP][GPT];
#pragma unroll
    for (int s = 0; s < NP; ++s)
#pragma unroll
      for (int u = 0; u < GPT; ++u)
        p[s][u] = reinterpret_cast<const float4*>(parts + s * add.part_stride + (long long)r * d)[gi[u]];
#pragma unroll
    for (int s = 0; s < NP; ++s)
#pragma unroll
      for (int u = 0; u < GPT; ++u) add4(v[u], p[s][u]);
  } else if constexpr (NP < 0) {
    // MoE: kept experts in rank order, each the sum of its K-split partials
    for (int k = 0; k < add.top_k; ++k) {
      const int sl = add.slot[r * add.top_k + k];
      if (sl < 0) continue;
      const float w = add.slot_w[r * add.top_k + k];
      float4 y[GPT];
#pragma unroll
      for (int u = 0; u < GPT; ++u) y[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int s = 0; s < add.n_parts; ++s) {
        const float4* ps = reinterpret_cast<const float4*>(parts + s * add.part_stride + (long long)sl * d);
#pragma unroll
        for (int u = 0; u < GPT; ++u) add4(y[u], ps[gi[u]]);
      }
#pragma unroll
      for (int u = 0; u < GPT; ++u) {
        v[u].x += w * y[u].x; v[u].y += w * y[u].y; v[u].z += w * y[u].z; v[u].w += w * y[u].w;
      }
    }
  }
  if constexpr (NP != 0) {
#pragma unroll
    for (int u = 0; u < GPT; ++u)
      if (ok[u]) reinterpret_cast<float4*>(xr)[gi[u]] = v[u];
  }
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < GPT; ++u)
    ss += ok[u] ? v[u].x * v[u].x + v[u].y * v[u].y + v[u].z * v[u].z + v[u].w * v[u].w : 0.f;
  const float tot = block_sum(ss, red);
  const float rs = rsqrtf(tot / (float)d + eps);
#pragma unroll
  for (int u = 0; u < GPT; ++u) {
    if (ok[u]) {
      const float4 a = v[u];
      const Hilo2 p0 = pack_hilo2(a.x * rs * bf16_to_f32(gg[u].x & 0xffff), a.y * rs * bf16_to_f32(gg[u].x >> 16));
      const Hilo2 p1 = pack_hilo2(a.z * rs * bf16_to_f32(gg[u].y & 0xffff), a.w * rs * bf16_to_f32(gg[u].y >> 16));
      uint16_t* dst = xn + xpack_off(r, 4 * gi[u], xn_ks);  // fragment-packed split-bf16 GEMM operand
      *reinterpret_cast<uint2*>(dst) = make_uint2(p0.hi, p1.hi);
      *reinterpret_cast<uint2*>(dst + XPACK_LO) = make_uint2(p0.lo, p1.lo);
    }
  }
  if (rt.w) {  // MoE: route the row from its normed fp32 values (uniform branch)
    float4 h[GPT];
#pragma unroll
    for (int u = 0; u < GPT; ++u)
      h[u] = make_float4(v[u].x * rs * bf16_to_f32(gg[u].x & 0xffff), v[u].y * rs * bf16_to_f32(gg[u].x >> 16),
                         v[u].z * rs * bf16_to_f32(gg[u].y & 0xffff), v[u].w * rs * bf16_to_f32(gg[u].y >> 16));
    route_row<GPT>(rt, r, h, gi, ok, d, w0);
  }
}

template <int NP>
static hipError_t launch_rn(float* x, const ResidualAdd& add, const uint16_t* gain, float eps, int rows, int d,
                            uint16_t* xn, int xn_ks, hipStream_t s, const Router& rt) {
  const int gpt = (d / 4 + RN_THREADS - 1) / RN_THREADS;  // float4 groups per thread
#define GRIFFIN_RN_LAUNCH(G)                                                                                    \
  hipLaunchKernelGGL((residual_rmsnorm_kernel<NP, G>), dim3(rows), dim3(RN_THREADS), 0, s, x, add, gain, eps, d, \
                     xn, xn_ks, rt)
  if (gpt <= 1) GRIFFIN_RN_LAUNCH(1);
  else if (gpt <= 2) GRIFFIN_RN_LAUNCH(2);
  else if (gpt <= 4) GRIFFIN_RN_LAUNCH(4);
  else GRIFFIN_RN_LAUNCH(8);
#undef GRIFFIN_RN_LAUNCH
  return hipGetLastError();
}

hipError_t launch_residual_rmsnorm(float* x, const ResidualAdd& add, const uint16_t* gain, float eps, int rows,
                                   int d, uint16_t* xn, int xn_ks, hipStream_t s, const Router& rt) {
  if (d % 4 != 0 || d > 32 * RN_THREADS || d > 32768 || add.n_parts > RN_SPLITS) return hipErrorInvalidValue;
  if (rt.w && (rt.n_experts < 1 || rt.n_experts > 64 || rt.top_k < 1 || rt.top_k > 4)) return hipErrorInvalidValue;
  if (rt.count && (!rt.w || !rt.slot || !rt.xe || rt.padded_rows < rows || rt.cap < rt.padded_rows))
    return hipErrorInvalidValue;
  if (rt.clear && (rt.n_clear < 0 || rt.n_clear > RN_THREADS)) return hipErrorInvalidValue;
  if (add.parts == nullptr) return launch_rn<0>(x, add, gain, eps, rows, d, xn, xn_ks, s, rt);
  if (add.slot != nullptr) return launch_rn<-1>(x, add, gain, eps, rows, d, xn, xn_ks, s, rt);
  switch (add.n_parts) {
#define GRIFFIN_RN_CASE(n) \
  case n: return launch_rn<n>(x, add, gain, eps, rows, d, xn, xn_ks, s, rt);
    GRIFFIN_RN_CASE(1) GRIFFIN_RN_CASE(2) GRIFFIN_RN_CASE(3) GRIFFIN_RN_CASE(4) GRIFFIN_RN_CASE(5)
    GRIFFIN_RN_CASE(6) GRIFFIN_RN_CASE(7) GRIFFIN_RN_CASE(8) GRIFFIN_RN_CASE(9) GRIFFIN_RN_CASE(10)
    GRIFFIN_RN_CASE(11) GRIFFIN_RN_CASE(12) GRIFFIN_RN_CASE(13) GRIFFIN_RN_CASE(14) GRIFFIN_RN_CASE(15)
    GRIFFIN_RN_CASE(16)
#undef GRIFFIN_RN_CASE
    default: return hipErrorInvalidValue;
  }
}

// ------------------------------------------------ rotary + tree K/V write ----
// For a valid tree row r = b*max_tree + i: sum the K-split partials of its
// QKV projection, rotate q and k (rotate-half pairing j <-> j + dh/2) at the
// node's position, write q (bf16) for attention, and k / v into cache slot
// prefix_len[b] + i (k row-major per slot, v transposed: one row per dim),
// and fp32 copies of the tree K/V for the attention merge.
// q is kept as split bf16: q_out holds bf16(q), q_lo the bf16 residual.
// The rotation angle pos * inv_freq[j] and its cosine and sine are evaluated
// in fp64 and rounded to fp32 (inv_freq[j] = base^(-2j/dh), fp64), so no load
// waits on the node's position; the row's metadata and partials are all
// loaded before any is used.
template <int NP>
__global__ __launch_bounds__(256) void qkv_rope_kernel(const float* __restrict__ parts, long long part_stride,
                                                       StepMeta meta, const double* __restrict__ inv_freq,
                                                       int Hq, int Hkv, int dh, int max_tree, int kv_cap,
                                                       uint16_t* __restrict__ q_out, uint16_t* __restrict__ q_lo,
                                                       uint16_t* __restrict__ kc, uint16_t* __restrict__ vc,
                                                       TreeKV32 tree) {
  const int r = blockIdx.x;
  const int b = r / max_tree, i = r % max_tree;
  const int half = dh >> 1;
  const int heads = Hq + 2 * Hkv;
  const int width = heads * dh;
  const int t = blockIdx.y * blockDim.x + threadIdx.x;  // one (head, rotation pair) per thread
  const bool live = t < heads * half;
  const int tt = live ? t : 0;  // clamped: loads stay unconditional
  const int h = tt / half, j = tt % half;
  const int c1 = h * dh + j, c2 = c1 + half;
  const int n_nodes = meta.n_nodes[b];
  const int pos = meta.pos[r];
  const int P = meta.prefix_len[b];
  const double inv = inv_freq[j];
  const float* __restrict__ row = parts + (long long)r * width;
  float a1[NP], a2[NP];  // all K-split partials loaded before any is summed
#pragma unroll
  for (int s = 0; s < NP; ++s) {
    a1[s] = row[s * part_stride + c1];
    a2[s] = row[s * part_stride + c2];
  }
  if (i >= n_nodes || !live) return;
  const int slot = P + i;
  float x1 = 0.f, x2 = 0.f;
#pragma unroll
  for (int s = 0; s < NP; ++s) {
    x1 += a1[s];
    x2 += a2[s];
  }
  if (h < Hq + Hkv) {
    double sd, cd;
    sincos((double)pos * inv, &sd, &cd);
    const float c = (float)cd, sn = (float)sd;
    const float y1 = x1 * c - x2 * sn;
    const float y2 = x2 * c + x1 * sn;
    if (h < Hq) {
      const long long o = ((long long)r * Hq + h) * dh;
      const uint16_t h1 = f32_to_bf16(y1), h2 = f32_to_bf16(y2);
      q_out[o + j] = h1;
      q_out[o + j + half] = h2;
      q_lo[o + j] = f32_to_bf16(y1 - bf16_to_f32(h1));
      q_lo[o + j + half] = f32_to_bf16(y2 - bf16_to_f32(h2));
    } else {
      uint16_t* k = kc + (((long long)b * Hkv + (h - Hq)) * kv_cap + slot) * dh;
      k[j] = f32_to_bf16(y1);
      k[j + half] = f32_to_bf16(y2);
      float* k32 = tree.k + (((long long)b * Hkv + (h - Hq)) * max_tree + i) * dh;
      k32[j] = y1;
      k32[j + half] = y2;
    }
  } else {
    // 32-slot tiles, transposed within the tile: [tile][dim][32]
    uint16_t* v = vc + ((long long)b * Hkv + (h - Hq - Hkv)) * dh * kv_cap + (long long)(slot >> 5) * dh * 32 +
                  (slot & 31);
    v[j * 32] = f32_to_bf16(x1);
    v[(j + half) * 32] = f32_to_bf16(x2);
    float* v32 = tree.v + (((long long)b * Hkv + (h - Hq - Hkv)) * max_tree + i) * dh;
    v32[j] = x1;
    v32[j + half] = x2;
  }
}

hipError_t launch_qkv_rope(const float* qkv_parts, int n_parts, long long part_stride, StepMeta meta,
                           const double* inv_freq, int Hq, int Hkv, int dh, int max_tree, int batch, int kv_cap,
                           uint16_t* q_out, uint16_t* q_lo, uint16_t* k_cache_l, uint16_t* v_cache_l, TreeKV32 tree,
                           hipStream_t s) {
  const int items = (Hq + 2 * Hkv) * (dh / 2);
  const dim3 grid(batch * max_tree, (items + 255) / 256);
  switch (n_parts) {
#define GRIFFIN_ROPE_CASE(n)                                                                                     \
  case n:                                                                                                       \
    hipLaunchKernelGGL(qkv_rope_kernel<n>, grid, dim3(256), 0, s, qkv_parts, part_stride, meta, inv_freq, Hq,     \
                       Hkv, dh, max_tree, kv_cap, q_out, q_lo, k_cache_l, v_cache_l, tree);                     \
    break;
    GRIFFIN_ROPE_CASE(1) GRIFFIN_ROPE_CASE(2) GRIFFIN_ROPE_CASE(3) GRIFFIN_ROPE_CASE(4) GRIFFIN_ROPE_CASE(5)
    GRIFFIN_ROPE_CASE(6) GRIFFIN_ROPE_CASE(7) GRIFFIN_ROPE_CASE(8) GRIFFIN_ROPE_CASE(9) GRIFFIN_ROPE_CASE(10)
    GRIFFIN_ROPE_CASE(11) GRIFFIN_ROPE_CASE(12) GRIFFIN_ROPE_CASE(13) GRIFFIN_ROPE_CASE(14) GRIFFIN_ROPE_CASE(15)
    GRIFFIN_ROPE_CASE(16)
#undef GRIFFIN_ROPE_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ------------------------------------------------------ argmax reduction ----
// pred[r] = argmax over the LM-head column groups' partial maxima; ties keep
// the lowest token id.

// One 256-thread workgroup per row; each thread issues all loads of its
// entries of a 4096-entry chunk before comparing any.  (max, lowest index) is
// a total order and the second largest value of a union does not depend on
// how it is split, so the result does not depend on the reduction order.
// margin[r] = max - second max (0 for a tie at the top; NaN when the row has
// fewer than two non-NaN entries).
constexpr int AR_THREADS = 256, AR_PER = 16;
__global__ __launch_bounds__(AR_THREADS) void argmax_reduce_kernel(const float* __restrict__ pmax,
                                                                   const float* __restrict__ pmax2,
                                                                   const int32_t* __restrict__ pidx,
                                                                   const int32_t* __restrict__ pnan, int n_tiles,
                                                                   int ld_part, int32_t* pred, float* margin,
                                                                   int32_t* nan_row) {
  __shared__ float sb[AR_THREADS / 64], s2[AR_THREADS / 64];
  __shared__ int si[AR_THREADS / 64], sn[AR_THREADS / 64];
  const int r = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const float* pm = pmax + (long long)r * ld_part;
  const float* pm2 = pmax2 + (long long)r * ld_part;
  const int32_t* pi = pidx + (long long)r * ld_part;
  const int32_t* pn = pnan + (long long)r * ld_part;
  float best = -INFINITY, second = -INFINITY;
  int bidx = 0x7fffffff;
  int nan_cnt = 0;
  for (int base = 0; base < n_tiles; base += AR_THREADS * AR_PER) {
    float v[AR_PER], v2[AR_PER];
    int id[AR_PER], nn[AR_PER];
#pragma unroll
    for (int k = 0; k < AR_PER; ++k) {
      const int t = min(base + k * AR_THREADS + tid, n_tiles - 1);  // clamped: loads stay unconditional
      v[k] = pm[t];
      v2[k] = pm2[t];
      id[k] = pi[t];
      nn[k] = pn[t];
    }
#pragma unroll
    for (int k = 0; k < AR_PER; ++k) {
      if (base + k * AR_THREADS + tid < n_tiles) {
        top2_merge(best, bidx, second, v[k], id[k], v2[k]);
        nan_cnt += nn[k];
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o, 64);
    const int oi = __shfl_xor(bidx, o, 64);
    const float os = __shfl_xor(second, o, 64);
    nan_cnt += __shfl_xor(nan_cnt, o, 64);
    top2_merge(best, bidx, second, ob, oi, os);
  }
  if (lane == 0) {
    sb[w] = best;
    s2[w] = second;
    si[w] = bidx;
    sn[w] = nan_cnt;
  }
  __syncthreads();
  if (tid == 0) {
    for (int k = 1; k < AR_THREADS / 64; ++k) {
      top2_merge(best, bidx, second, sb[k], si[k], s2[k]);
      nan_cnt += sn[k];
    }
    pred[r] = bidx;
    margin[r] = second == -INFINITY ? __builtin_nanf("") : best - second;
    nan_row[r] = nan_cnt;
  }
}

hipError_t launch_argmax_reduce(const float* pmax, const float* pmax2, const int32_t* pidx, const int32_t* pnan,
                                int n_tiles, int ld_part, int rows, int32_t* pred, float* margin, int32_t* nan_row,
                                hipStream_t s) {
  if (n_tiles < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(argmax_reduce_kernel, dim3(rows), dim3(AR_THREADS), 0, s, pmax, pmax2, pidx, pnan, n_tiles,
                     ld_part, pred, margin, nan_row);
  return hipGetLastError();
}

// ------------------------------------------------------- acceptance walk ----
// One wavefront per sequence, one lane per tree node.  Node i (i >= 1) matches
// when its token equals the prediction at its parent; it is accepted when every
// node on its root path matches (its ancestor mask, root excluded, lies inside
// the match ballot).  The deepest accepted node wins, smallest id on ties.
__global__ __launch_bounds__(64) void accept_kernel(StepMeta meta, const int32_t* __restrict__ pred,
                                                    const int32_t* __restrict__ nan_row, int max_tree,
                                                    int max_depth, int32_t* __restrict__ result) {
  const int b = blockIdx.x;
  const int i = threadIdx.x;
  const int n = meta.n_nodes[b];
  const int r = b * max_tree + i;
  const bool live = i < n;
  bool match = false;
  int depth = 0;
  uint64_t anc = 0;
  if (live) {
    depth = meta.depth[r];
    anc = meta.anc[r];
    match = (i == 0) || (meta.token[r] == pred[b * max_tree + meta.parent[r]]);
  }
  const uint64_t matched = __ballot(match);
  const bool ok = live && ((anc & ~matched) == 0);
  // key: deeper first, then smaller id
  int key = ok ? (depth << 8) | (255 - i) : -1;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) key = max(key, __shfl_xor(key, o, 64));
  const int best = 255 - (key & 255);
  const int L = key >> 8;
  const uint64_t best_anc = __shfl(anc, best, 64);
  const int nan_any = __any(live && nan_row[r] != 0);
  int32_t* res = result + (long long)b * result_stride(max_depth);
  int32_t* tokens_out = res + 2;
  int32_t* path = res + 3 + max_depth;
  if (live && i != 0 && ((best_anc >> i) & 1ull)) {
    path[depth - 1] = i;
    tokens_out[depth - 1] = meta.token[r];
  }
  if (i >= L && i < max_depth) path[i] = -1;
  if (i > L && i <= max_depth) tokens_out[i] = -1;
  if (i == 0) {
    res[0] = L;
    res[1] = nan_any ? 1 : 0;
    tokens_out[L] = pred[b * max_tree + best];
  }
}

hipError_t launch_accept(StepMeta meta, const int32_t* pred, const int32_t* nan_row, int batch, int max_tree,
                         int max_depth, int32_t* result, hipStream_t s) {
  hipLaunchKernelGGL(accept_kernel, dim3(batch), dim3(64), 0, s, meta, pred, nan_row, max_tree, max_depth, result);
  return hipGetLastError();
}

// ------------------------------------------------------------ KV commit ----
// After the acceptance walk: the accepted path's nodes n_1..n_L (depths
// 1..L) hold K/V already rotated at positions prefix_len + k, in scratch slots
// prefix_len + n_k.  Move them to slots prefix_len + k so that the cache is the
// plain causal cache of prefix + root + accepted tokens.  One workgroup per
// (KV head, sequence, layer); every source is read into LDS before any
// destination is written (a destination slot can be a later source).
constexpr int COMMIT_MAX_DEPTH = 63;
__global__ __launch_bounds__(256) void commit_kernel(const int32_t* __restrict__ result, int max_depth,
                                                     StepMeta meta, int Hkv, int dh, int kv_cap, long long layer_kv,
                                                     uint16_t* __restrict__ kc, uint16_t* __restrict__ vc) {
  __shared__ uint16_t ks[COMMIT_MAX_DEPTH * 128], vs[COMMIT_MAX_DEPTH * 128];
  const int hk = blockIdx.x, b = blockIdx.y, l = blockIdx.z;
  const int32_t* res = result + (long long)b * result_stride(max_depth);
  const int L = res[0];
  const int32_t* path = res + 3 + max_depth;
  const int P = meta.prefix_len[b];
  const long long head = (long long)l * layer_kv + ((long long)b * Hkv + hk) * kv_cap * dh;
  uint16_t* K = kc + head;
  uint16_t* V = vc + head;
  const int n = L * dh;
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    const int k = e / dh, j = e % dh;
    const int src = P + path[k];
    ks[e] = K[(long long)src * dh + j];
    vs[e] = V[(long long)(src >> 5) * dh * 32 + j * 32 + (src & 31)];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    const int k = e / dh, j = e % dh;
    const int dst = P + 1 + k;
    K[(long long)dst * dh + j] = ks[e];
    V[(long long)(dst >> 5) * dh * 32 + j * 32 + (dst & 31)] = vs[e];
  }
}

hipError_t launch_commit(const int32_t* result, int max_depth, StepMeta meta, int batch, int n_layers, int Hkv,
                         int dh, int kv_cap, long long layer_kv, uint16_t* k_cache, uint16_t* v_cache,
                         hipStream_t s) {
  if (max_depth > COMMIT_MAX_DEPTH || dh > 128) return hipErrorInvalidValue;
  hipLaunchKernelGGL(commit_kernel, dim3(Hkv, batch, n_layers), dim3(256), 0, s, result, max_depth, meta, Hkv, dh,
                     kv_cap, layer_kv, k_cache, v_cache);
  return hipGetLastError();
}

// ---------------------------------------------------------- row gather ----
__global__ __launch_bounds__(256) void gather_rows_kernel(const float* __restrict__ x, int d,
                                                          const int32_t* __restrict__ rows, float* __restrict__ out) {
  const int j = blockIdx.x, r = rows[j];
  float* o = out + (long long)j * d;
  for (int k = threadIdx.x; k < d; k += 256) o[k] = r < 0 ? 0.f : x[(long long)r * d + k];
}

hipError_t launch_gather_rows(const float* x, int d, const int32_t* rows, int n, float* out, hipStream_t s) {
  hipLaunchKernelGGL(gather_rows_kernel, dim3(n), dim3(256), 0, s, x, d, rows, out);
  return hipGetLastError();
}

}  // namespace griffin
