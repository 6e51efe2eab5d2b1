// Stochastic tree acceptance at temperature T > 0.
//
// The paper evaluates T in {0, 1} and relies on the method being lossless
// (Sec. 5).  At T > 0 a tree is accepted by recursive rejection sampling over
// each node's children, in node-id order, the children having been drawn from
// the parent's draft distribution q without replacement:
//   p = softmax(logits / T) at the node, q = the node's draft distribution;
//   child with token t: accepted when u_accept[child] < min(1, p(t) / q(t));
//   rejected: p <- max(p - q, 0) renormalised, t leaves q (q renormalised);
//   a child accepted: continue there; none (or no children): emit one token
//   drawn from p with u_final[node] (first token whose cumulative sum exceeds
//   u * sum, in token order).
// Degenerate inputs: q(t) = 0 accepts when p(t) > 0; a residual that sums to
// zero leaves p unchanged; q whose mass is all removed counts as zero.
//
// One workgroup walks one sequence.  Every pass over the vocabulary (the
// normaliser of p, a residual update, the final draw) is block-wide with
// reductions in a fixed order.  The residual is kept unnormalised in one of
// two scratch rows per sequence (double-buffered so that a residual that
// sums to zero can be dropped); before the first rejection at a node it is
// computed from the logits on the fly.

#include "device_common.h"
#include "griffin_internal.h"

namespace griffin {

constexpr int SA_THREADS = 1024;
constexpr int SA_MAX_REMOVED = 64;  // children of one node (max_tree <= 64)

__device__ __forceinline__ float block_max(float v, float* smem /* >= 16 floats */) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) smem[w] = v;
  __syncthreads();
  float t = -INFINITY;
  for (int i = 0; i < nw; ++i) t = fmaxf(t, smem[i]);
  return t;
}

__global__ __launch_bounds__(SA_THREADS) void sampled_accept_kernel(SampledArgs a) {
  __shared__ float red[16];
  __shared__ float scan[SA_THREADS];
  __shared__ int removed[SA_MAX_REMOVED];
  __shared__ int found;
  const int b = blockIdx.x, tid = threadIdx.x, V = a.vocab;
  const int n = a.n_nodes[b];
  const long long row0 = (long long)b * a.max_tree;
  float* buf0 = a.res + (long long)b * 2 * V;
  float* buf1 = buf0 + V;
  int32_t* out = a.result + (long long)b * result_stride(a.max_depth);

  int node = 0, L = 0, nan = 0, emitted = 0;
  while (true) {  // uniform: every branch below depends on block-wide values only
    const float* lg = a.logits + (row0 + node) * V;
    const float* qd = a.q + (row0 + node) * V;
    // target distribution at the node: maximum and normaliser
    float mx = -INFINITY;
    int bad = 0;
    for (int v = tid; v < V; v += SA_THREADS) {
      const float x = lg[v];
      bad |= x != x;
      mx = fmaxf(mx, x);
    }
    mx = block_max(mx, red);
    bad = block_sum((float)bad, red) > 0.f;
    float zl = 0.f, zq = 0.f;
    for (int v = tid; v < V; v += SA_THREADS) {
      zl += expf((lg[v] - mx) * a.inv_t);
      zq += qd[v];
    }
    const float Z = block_sum(zl, red);
    float qZ = block_sum(zq, red);
    if (bad || !(Z > 0.f)) {
      nan = 1;
      break;
    }
    // current residual r (unnormalised, normaliser Zr): -1 = from the logits
    int cur = -1;
    float Zr = Z;
    int n_removed = 0;
    auto r_at = [&](int v) {
      return cur < 0 ? expf((lg[v] - mx) * a.inv_t) : (cur == 0 ? buf0[v] : buf1[v]);
    };
    auto q_at = [&](int v) {
      float x = qd[v];
      for (int k = 0; k < n_removed; ++k) x = removed[k] == v ? 0.f : x;
      return x;
    };
    int next = -1;
    for (int c = 1; c < n; ++c) {
      if (a.parent[row0 + c] != node) continue;
      const int t = a.token[row0 + c];
      const float pt = r_at(t) / Zr;
      const float qt_raw = q_at(t);
      const float qt = qZ > 0.f ? qt_raw / qZ : 0.f;
      const float acc = qt > 0.f ? fminf(1.f, pt / qt) : (pt > 0.f ? 1.f : 0.f);
      if (a.u_accept[row0 + c] < acc) {
        next = c;
        break;
      }
      // residual max(p - q, 0) into the other row
      float* dst = cur == 0 ? buf1 : buf0;
      float s = 0.f;
      for (int v = tid; v < V; v += SA_THREADS) {
        const float qv = qZ > 0.f ? q_at(v) / qZ : 0.f;
        const float d = fmaxf(r_at(v) / Zr - qv, 0.f);
        dst[v] = d;
        s += d;
      }
      s = block_sum(s, red);  // its barriers also publish dst to the block
      if (s > 0.f) {
        cur = dst == buf0 ? 0 : 1;
        Zr = s;
      }
      // the rejected token leaves q
      qZ -= qt_raw;
      if (n_removed < SA_MAX_REMOVED) {
        if (tid == 0) removed[n_removed] = t;
        ++n_removed;
      }
      __syncthreads();
    }
    if (next >= 0) {
      if (tid == 0) out[3 + a.max_depth + L] = next;
      ++L;
      node = next;
      continue;
    }
    // draw from the residual: chunk sums, an inclusive scan over the chunks in
    // a fixed order, then the chunk that holds u * total is walked in order
    const int C = (V + SA_THREADS - 1) / SA_THREADS;
    const int v0 = min(V, tid * C), v1 = min(V, v0 + C);
    float cs = 0.f;
    for (int v = v0; v < v1; ++v) cs += r_at(v);
    scan[tid] = cs;
    if (tid == 0) found = -1;
    __syncthreads();
    for (int off = 1; off < SA_THREADS; off <<= 1) {
      const float add = tid >= off ? scan[tid - off] : 0.f;
      __syncthreads();
      scan[tid] += add;
      __syncthreads();
    }
    const float total = scan[SA_THREADS - 1];
    const float thr = a.u_final[row0 + node] * total;
    const float excl = tid > 0 ? scan[tid - 1] : 0.f;
    if (excl <= thr && thr < scan[tid]) {
      float accum = excl;
      int pick = v1 - 1;
      for (int v = v0; v < v1; ++v) {
        accum += r_at(v);
        if (accum > thr) {
          pick = v;
          break;
        }
      }
      found = pick;  // at most one thread's interval holds thr
    }
    __syncthreads();
    emitted = found >= 0 ? found : V - 1;
    break;
  }
  if (tid == 0) {
    out[0] = L;
    out[1] = nan;
    for (int k = 0; k < L; ++k) out[2 + k] = a.token[row0 + out[3 + a.max_depth + k]];
    out[2 + L] = nan ? -1 : emitted;
    for (int k = L + 1; k <= a.max_depth; ++k) out[2 + k] = -1;
    for (int k = L; k < a.max_depth; ++k) out[3 + a.max_depth + k] = -1;
  }
}

hipError_t launch_sampled_accept(const SampledArgs& a, int batch, hipStream_t s) {
  if (batch < 1 || a.vocab < 1 || a.max_tree < 1 || a.max_tree > SA_MAX_REMOVED + 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(sampled_accept_kernel, dim3(batch), dim3(SA_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace griffin
