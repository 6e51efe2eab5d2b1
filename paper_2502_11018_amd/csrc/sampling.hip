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
// Closed form of the residual (p, q normalised; S_k = mass of q left after k
// rejections, S_0 = 1): after k rejections at a node
//   r_k(v) = max(p(v) - a_k q(v), 0) / D_k    for tokens still in q,
//   r_k(t_j) = f_j / D_k                       for each rejected token t_j,
// with a_0 = 0, D_0 = 1 and, at the next rejection, a_{k+1} = a_k + D_k / S_k
// and D_{k+1} = G = the sum of the unnormalised new residual.  f_j =
// max(p(t_j) - a_{j+1} q(t_j), 0) is frozen when t_j leaves q.  By induction:
// where r_k(v) > 0, r_k(v) - q(v) / S_k = (p(v) - a_{k+1} q(v)) / D_k, and
// where r_k(v) = 0 both sides are <= 0 (a only grows).  So one rejection is
// one read-only reduction G = sum_v max(p(v) - a_{k+1} q(v), 0), corrected
// at the tokens already rejected.
//
// The acceptance probability of a node's k-th child depends only on the k
// rejections before it at the same node, so all nodes advance together, one
// launch per child rank, each spreading a node's vocabulary over `nslice`
// workgroups that write per-slice partial sums:
//   sampled_norm_kernel: softmax normaliser and sum of q (partials);
//   sampled_step_kernel, k = 0, 1, ..: every workgroup first folds the
//     previous launch's partials into the node's state (in slice order; the
//     same arithmetic in every workgroup, workgroup 0 stores it), takes the
//     k-th child's acceptance probability, then reduces G for its rejection;
//   sampled_draw_sums_kernel: walks every tree with the stored probabilities,
//     folds the final node's last partials, sums its residual per slice;
//   sampled_pick_kernel: the inverse CDF: the slice that holds u * total,
//     then an exact in-order scan inside it.
// Kernel boundaries order every hand-over; no counters, fences or atomics.
//
// Deterministic drafts (q == nullptr): a tree ranked from the draft's
// log-probabilities is a function of the draft, so each child is the point
// mass at its own token: accepted with probability p(t) / D, D the mass of p
// left after the node's earlier rejections; a rejection removes t from p (no
// change for a token already removed, or when nothing would be left).  No
// vocabulary pass per rejection: the step launches are skipped and the walk
// itself tests every child of the nodes it visits.  The final node's
// residual is p without its rejected tokens, which the draw kernels take as
// the q-free residual (a = 0) with each rejected token frozen at 0.

#include <algorithm>
#include <mutex>

#include "device_common.h"
#include "griffin_internal.h"
#include "sampling.h"

namespace griffin {

constexpr int SA_THREADS = 256;
constexpr int SA_RM = 64;  // rejected tokens per node (children: max_tree - 1 <= 63)

struct SampState {
  float M, inv_z, inv_q;  // max logit, 1 / softmax normaliser, 1 / sum(q)
  float a, D, S;          // residual parameters and q mass left
  int n_rm, bad;          // rejected tokens so far; NaN in the logits or no mass
};

struct RmEntry {
  int tok;
  float f;     // frozen unnormalised residual
  float p, q;  // normalised p and q at the token
};

struct SampScratch {
  float4* npart;  // [rows][nslice] softmax partials (max, sum, q sum, NaN flag)
  float* gpart;   // [2][rows][nslice] rejection partials, by step parity
  float* dpart;   // [batch][nslice] residual sums of the final node
  SampState* st;  // [2][rows] state before the k-th child's test, by step parity
  RmEntry* rm;    // [rows][SA_RM]
  float* acc;     // [rows] acceptance probability of the node (as a child)
  int* bad;       // [rows] NaN flag of nodes that have children
};

__host__ __device__ inline size_t sa_align(size_t x) { return (x + 255) / 256 * 256; }

__host__ __device__ inline SampScratch sa_carve(void* base, int batch, int max_tree, int nslice) {
  const size_t rows = (size_t)batch * max_tree;
  char* p = static_cast<char*>(base);
  SampScratch s;
  s.npart = reinterpret_cast<float4*>(p);
  p += sa_align(rows * nslice * sizeof(float4));
  s.gpart = reinterpret_cast<float*>(p);
  p += sa_align(2 * rows * nslice * 4);
  s.dpart = reinterpret_cast<float*>(p);
  p += sa_align((size_t)batch * nslice * 4);
  s.st = reinterpret_cast<SampState*>(p);
  p += sa_align(2 * rows * sizeof(SampState));
  s.rm = reinterpret_cast<RmEntry*>(p);
  p += sa_align(rows * SA_RM * sizeof(RmEntry));
  s.acc = reinterpret_cast<float*>(p);
  p += sa_align(rows * 4);
  s.bad = reinterpret_cast<int*>(p);
  return s;
}

int sampled_nslice(int vocab) { return std::min(64, std::max(1, (vocab + 2047) / 2048)); }

size_t sampled_scratch_bytes(int batch, int max_tree, int vocab) {
  const size_t rows = (size_t)batch * max_tree;
  const int ns = sampled_nslice(vocab);
  return sa_align(rows * ns * sizeof(float4)) + sa_align(2 * rows * ns * 4) + sa_align((size_t)batch * ns * 4) +
         sa_align(2 * rows * sizeof(SampState)) + sa_align(rows * SA_RM * sizeof(RmEntry)) + sa_align(rows * 4) +
         sa_align(rows * 4);
}

struct Norm {
  float M, inv_t, inv_z, inv_q;
};

__device__ __forceinline__ float p_of(float x, const Norm& n) { return expf((x - n.M) * n.inv_t) * n.inv_z; }

// unnormalised residual max(p - a q, 0) of a token still in q, from normalised p and q
__device__ __forceinline__ float resid_pq(float p, float q, float a) { return fmaxf(p - a * q, 0.f); }

__device__ __forceinline__ float resid(float x, float y, float a, const Norm& n) {
  return resid_pq(p_of(x, n), y * n.inv_q, a);
}

__device__ __forceinline__ Norm norm_of(const SampState& s, float inv_t) { return {s.M, inv_t, s.inv_z, s.inv_q}; }

__device__ __forceinline__ float block_max(float v, float* smem) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) smem[w] = v;
  __syncthreads();
  float t = -INFINITY;
  for (int i = 0; i < nw; ++i) t = fmaxf(t, smem[i]);
  return t;
}

// Slice s of a row: a multiple of 4 elements long, so that with V % 4 == 0
// every slice starts on a 16-byte boundary of the row.
__device__ __forceinline__ void slice_range(int V, int nslice, int s, int& lo, int& hi) {
  const int chunk = ((V + nslice - 1) / nslice + 3) & ~3;
  lo = min(V, s * chunk);
  hi = min(V, lo + chunk);
}

// f(x, y) for every element of [lo, hi) of a logits row and a q row that this
// thread owns; VEC: 16-byte loads (V % 4 == 0, rows 16-byte aligned).  Q:
// read the q row, else y = 0 (leaves: their q rows are not read).
template <bool VEC, bool Q, typename F>
__device__ __forceinline__ void for_slice(const float* lg, const float* qd, int lo, int hi, F&& f) {
  if constexpr (VEC) {
    const float4* l4 = reinterpret_cast<const float4*>(lg);
    const float4* q4 = reinterpret_cast<const float4*>(qd);
#pragma unroll 2
    for (int i = (lo >> 2) + (int)threadIdx.x; i < (hi >> 2); i += SA_THREADS) {
      const float4 x = l4[i];
      const float4 y = Q ? q4[i] : make_float4(0.f, 0.f, 0.f, 0.f);
      f(x.x, y.x);
      f(x.y, y.y);
      f(x.z, y.z);
      f(x.w, y.w);
    }
  } else {
    for (int v = lo + (int)threadIdx.x; v < hi; v += SA_THREADS) f(lg[v], Q ? qd[v] : 0.f);
  }
}

// ---- wave-wide state transitions (lanes index slices and rejected tokens) -------

// The state before the first test at a node, from its softmax partials
// (pp: this lane's slice, identity for lanes >= nslice).
__device__ __forceinline__ SampState state_from_norm(float4 pp, float inv_t) {
  const float M = wave_max(pp.x);
  const float Z = wave_sum(pp.x > -INFINITY ? pp.y * expf((pp.x - M) * inv_t) : 0.f);
  const float qs = wave_sum(pp.z);
  const float anybad = wave_max(pp.w);
  SampState st;
  st.M = M;
  st.inv_z = 1.f / Z;
  st.inv_q = qs > 0.f ? 1.f / qs : 0.f;
  st.a = 0.f;
  st.D = 1.f;
  st.S = 1.f;
  st.n_rm = 0;
  st.bad = (anybad > 0.f || !(Z > 0.f)) ? 1 : 0;
  return st;
}

// After rejecting a child with token t (p, q normalised at t): gp = this
// lane's slice of G at a + D / S, e = this lane's rejected-token entry.  The
// lane at index st.n_rm receives t's entry in e unless t was rejected before.
__device__ __forceinline__ SampState advance(const SampState& st, float gp, RmEntry& e, int t, float pt, float qt) {
  const int lane = threadIdx.x & 63;
  const bool live = !st.bad && st.S > 0.f;
  const float an = st.a + st.D / st.S;
  const float G = wave_sum(gp);
  // rejected tokens keep their frozen value instead of max(p - a q, 0)
  const float corr = wave_sum(lane < st.n_rm ? e.f - resid_pq(e.p, e.q, an) : 0.f);
  const bool dup = __ballot(lane < st.n_rm && e.tok == t) != 0;
  SampState nx = st;
  if (live && (G + corr) / st.D > 0.f) {
    nx.a = an;
    nx.D = G + corr;
  }
  if (!dup) {
    if (lane == st.n_rm) e = RmEntry{t, resid_pq(pt, qt, nx.a), pt, qt};
    nx.S = st.S - qt;
    nx.n_rm = st.n_rm + 1;
  }
  return nx;
}

// Acceptance probability of a child with token t tested in state st.
__device__ __forceinline__ float accept_prob(const SampState& st, const RmEntry& e, int t, float pt, float qt) {
  const int lane = threadIdx.x & 63;
  const uint64_t dm = __ballot(lane < st.n_rm && e.tok == t);
  const bool dup = dm != 0;
  const float fdup = __shfl(e.f, dup ? __ffsll((unsigned long long)dm) - 1 : 0, 64);
  const float p_res = (dup ? fdup : resid_pq(pt, qt, st.a)) / st.D;
  const float q_res = (dup || !(st.S > 0.f)) ? 0.f : qt / st.S;
  return q_res > 0.f ? fminf(1.f, p_res / q_res) : (p_res > 0.f ? 1.f : 0.f);
}

// ---- softmax normaliser and q's sum of every node --------------------------------
template <bool VEC>
__global__ __launch_bounds__(SA_THREADS) void sampled_norm_kernel(SampledArgs a, int nslice, int n_parents) {
  __shared__ float red[8];
  const SampScratch sc = sa_carve(a.scratch, a.scratch_batch, a.max_tree, nslice);
  const int s = blockIdx.x, row = a.order[blockIdx.y], tid = threadIdx.x, V = a.vocab;
  const float* lg = a.logits + (size_t)row * V;
  const float* qd = a.q ? a.q + (size_t)row * V : nullptr;
  const float inv_t = a.inv_t;
  int lo, hi;
  slice_range(V, nslice, s, lo, hi);
  // running maximum and sum of exp((x - m) / T); -inf logits add nothing, NaN
  // ones are flagged (fmaxf skips them)
  float m = -INFINITY, se = 0.f, sq = 0.f;
  int bad = 0;
  auto f = [&](float x, float y) {
    sq += y;
    bad |= x != x;
    const float mn = fmaxf(m, x);
    se = (mn == m ? se : se * expf((m - mn) * inv_t)) + (x > -INFINITY ? expf((x - mn) * inv_t) : 0.f);
    m = mn;
  };
  if (qd && (int)blockIdx.y < n_parents)  // rows of `order` with children come first
    for_slice<VEC, true>(lg, qd, lo, hi, f);
  else
    for_slice<VEC, false>(lg, qd, lo, hi, f);
  const float mb = block_max(m, red);
  const float seb = block_sum(m > -INFINITY ? se * expf((m - mb) * inv_t) : 0.f, red);
  const float sqb = block_sum(sq, red);
  const float badb = block_max((float)bad, red);
  if (tid == 0) sc.npart[(size_t)row * nslice + s] = make_float4(mb, seb, sqb, badb);
}

// ---- the k-th child of every node with more than k children ----------------------
// Item i: node a.order[i]; its k-th child and token at a.step_child /
// a.step_token[base + i], its (k-1)-th at [prev_base + i].
template <bool VEC>
__global__ __launch_bounds__(SA_THREADS) void sampled_step_kernel(SampledArgs a, int nslice, int k, int base,
                                                                  int prev_base) {
  __shared__ float red[8];
  __shared__ SampState sh_st;
  const SampScratch sc = sa_carve(a.scratch, a.scratch_batch, a.max_tree, nslice);
  const int s = blockIdx.x, item = blockIdx.y, tid = threadIdx.x, V = a.vocab;
  const int row = a.order[item];
  const float* lg = a.logits + (size_t)row * V;
  const float* qd = a.q + (size_t)row * V;
  const size_t rows = (size_t)a.scratch_batch * a.max_tree;
  if (tid < 64) {
    const int lane = tid;
    const int t = a.step_token[base + item], child = a.step_child[base + item];
    SampState st;
    RmEntry e{-1, 0.f, 0.f, 0.f};
    const float x = lg[t], y = qd[t];
    if (k == 0) {
      const float4 pp =
          lane < nslice ? sc.npart[(size_t)row * nslice + lane] : make_float4(-INFINITY, 0.f, 0.f, 0.f);
      st = state_from_norm(pp, a.inv_t);
    } else {
      const int tp = a.step_token[prev_base + item];
      const SampState pv = sc.st[((k - 1) & 1) * rows + row];
      const float gp = lane < nslice ? sc.gpart[(((k - 1) & 1) * rows + row) * nslice + lane] : 0.f;
      e = sc.rm[(size_t)row * SA_RM + lane];
      const Norm np = norm_of(pv, a.inv_t);
      const float xp = lg[tp], yp = qd[tp];
      st = advance(pv, gp, e, tp, p_of(xp, np), yp * np.inv_q);
      if (s == 0 && st.n_rm > pv.n_rm && lane == pv.n_rm) sc.rm[(size_t)row * SA_RM + lane] = e;
    }
    const Norm nm = norm_of(st, a.inv_t);
    const float acc = accept_prob(st, e, t, p_of(x, nm), y * nm.inv_q);
    if (s == 0 && lane == 0) {
      sc.st[(k & 1) * rows + row] = st;
      sc.acc[(size_t)(row / a.max_tree) * a.max_tree + child] = acc;
      if (k == 0) sc.bad[row] = st.bad;
    }
    if (lane == 0) sh_st = st;
  }
  __syncthreads();
  const SampState st = sh_st;
  const Norm nm = norm_of(st, a.inv_t);
  const float an = st.a + st.D / st.S;
  int lo, hi;
  slice_range(V, nslice, s, lo, hi);
  float g = 0.f;
  if (!st.bad && st.S > 0.f)
    for_slice<VEC, true>(lg, qd, lo, hi, [&](float x, float y) { g += resid(x, y, an, nm); });
  g = block_sum(g, red);
  if (tid == 0) sc.gpart[((k & 1) * rows + row) * nslice + s] = g;
}

// ---- the walk and the final node's state (one wave; every workgroup alike) -------
struct WalkEnd {
  int node, L, nan, pathv;  // pathv: this lane's path entry (lane < L)
  SampState st;             // final node: state after all its children's rejections
  RmEntry e;                // this lane's rejected-token entry of the final node
};

// Walk of a deterministic draft's tree: every child a point mass at its token.
__device__ __forceinline__ WalkEnd walk_tree_point_mass(const SampledArgs& a, const SampScratch& sc, int nslice,
                                                        int b) {
  const int lane = threadIdx.x & 63, n = a.n_nodes[b];
  const size_t row0 = (size_t)b * a.max_tree;
  const bool in = lane < n;
  const int ln = min(lane, n - 1);
  const int par = (in && lane >= 1) ? a.parent[row0 + ln] : -1;
  const int tok = in ? a.token[row0 + ln] : 0;
  const float ua = in ? a.u_accept[row0 + ln] : 1.f;
  WalkEnd w;
  w.node = 0;
  w.L = 0;
  w.nan = 0;
  w.pathv = -1;
  for (int it = 0;; ++it) {
    const size_t fr = row0 + w.node;
    const float4 pp = lane < nslice ? sc.npart[fr * nslice + lane] : make_float4(-INFINITY, 0.f, 0.f, 0.f);
    SampState st = state_from_norm(pp, a.inv_t);  // D = 1: all of p left
    w.e = RmEntry{-1, 0.f, 0.f, 0.f};
    w.st = st;
    if (st.bad) {
      w.nan = 1;
      return w;
    }
    const Norm nm = norm_of(st, a.inv_t);
    const bool kid = par == w.node;
    const float pt = kid ? p_of(a.logits[fr * a.vocab + tok], nm) : 0.f;
    int nxt = -1;
    for (uint64_t rest = __ballot(kid); rest && it < a.max_depth; rest &= rest - 1) {
      const int c = __ffsll((unsigned long long)rest) - 1;
      const int t = __shfl(tok, c, 64);
      const float ptc = __shfl(pt, c, 64);
      const bool dup = __ballot(lane < st.n_rm && w.e.tok == t) != 0;
      const float acc = dup ? 0.f : fminf(1.f, ptc / st.D);
      if (__shfl(ua, c, 64) < acc) {
        nxt = c;
        break;
      }
      if (!dup && st.D - ptc > 0.f) {
        if (lane == st.n_rm) w.e = RmEntry{t, 0.f, ptc, 0.f};
        st.D -= ptc;
        ++st.n_rm;
      }
    }
    w.st = st;
    if (nxt < 0) return w;
    if (lane == w.L) w.pathv = nxt;
    ++w.L;
    w.node = nxt;
  }
}

__device__ __forceinline__ WalkEnd walk_tree(const SampledArgs& a, const SampScratch& sc, int nslice, int b) {
  if (!a.q) return walk_tree_point_mass(a, sc, nslice, b);
  const int lane = threadIdx.x & 63, n = a.n_nodes[b];
  const size_t row0 = (size_t)b * a.max_tree, rows = (size_t)a.scratch_batch * a.max_tree;
  const bool in = lane < n;
  const int ln = min(lane, n - 1);
  const int par = (in && lane >= 1) ? a.parent[row0 + ln] : -1;
  const float accv = (in && lane >= 1) ? sc.acc[row0 + ln] : 0.f;
  const float ua = in ? a.u_accept[row0 + ln] : 1.f;
  const int badv = in ? sc.bad[row0 + ln] : 0;
  WalkEnd w;
  w.node = 0;
  w.L = 0;
  w.nan = 0;
  w.pathv = -1;
  for (int it = 0; it <= a.max_depth; ++it) {
    if (!__ballot(par == w.node)) break;  // a leaf: its flag comes from its partials below
    if (__shfl(badv, w.node, 64)) {
      w.nan = 1;
      return w;
    }
    const uint64_t m = __ballot(par == w.node && ua < accv);
    if (!m) break;
    const int nxt = __ffsll((unsigned long long)m) - 1;
    if (lane == w.L) w.pathv = nxt;
    ++w.L;
    w.node = nxt;
  }
  const size_t fr = row0 + w.node;
  const uint64_t kids = __ballot(par == w.node);
  const int nk = __popcll(kids);
  w.e = RmEntry{-1, 0.f, 0.f, 0.f};
  if (nk == 0) {
    const float4 pp = lane < nslice ? sc.npart[fr * nslice + lane] : make_float4(-INFINITY, 0.f, 0.f, 0.f);
    w.st = state_from_norm(pp, a.inv_t);
    w.nan = w.st.bad;
  } else {
    const int last = 63 - __clzll(kids);
    const int t = a.token[row0 + last];
    const SampState pv = sc.st[((nk - 1) & 1) * rows + fr];
    const float gp = lane < nslice ? sc.gpart[(((nk - 1) & 1) * rows + fr) * nslice + lane] : 0.f;
    w.e = sc.rm[fr * SA_RM + lane];
    const Norm np = norm_of(pv, a.inv_t);
    const float x = a.logits[fr * a.vocab + t], y = a.q[fr * a.vocab + t];
    w.st = advance(pv, gp, w.e, t, p_of(x, np), y * np.inv_q);
  }
  return w;
}

// ---- residual sums of every tree's final node, per slice -------------------------
template <bool VEC>
__global__ __launch_bounds__(SA_THREADS) void sampled_draw_sums_kernel(SampledArgs a, int nslice) {
  __shared__ float red[8];
  __shared__ SampState sh_st;
  __shared__ int sh_node, sh_nan;
  __shared__ RmEntry rml[SA_RM];
  const SampScratch sc = sa_carve(a.scratch, a.scratch_batch, a.max_tree, nslice);
  const int s = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, V = a.vocab;
  if (tid < 64) {
    const WalkEnd w = walk_tree(a, sc, nslice, b);
    if (tid == 0) {
      sh_st = w.st;
      sh_node = w.node;
      sh_nan = w.nan;
    }
    rml[tid] = w.e;
  }
  __syncthreads();
  float g = 0.f;
  if (!sh_nan) {
    const SampState st = sh_st;
    const Norm nm = norm_of(st, a.inv_t);
    const size_t fr = (size_t)b * a.max_tree + sh_node;
    int lo, hi;
    slice_range(V, nslice, s, lo, hi);
    const float af = st.a;
    const float* qd = a.q ? a.q + fr * V : nullptr;
    auto f = [&](float x, float y) { g += resid(x, y, af, nm); };
    if (st.n_rm > 0 && qd)  // a node without children (or rejections) draws from p alone
      for_slice<VEC, true>(a.logits + fr * V, qd, lo, hi, f);
    else
      for_slice<VEC, false>(a.logits + fr * V, qd, lo, hi, f);
    if (tid < st.n_rm) {  // rejected tokens in this slice: frozen value instead
      const RmEntry e = rml[tid];
      if (e.tok >= lo && e.tok < hi) g += e.f - resid_pq(e.p, e.q, af);
    }
  }
  g = block_sum(g, red);
  if (tid == 0) sc.dpart[(size_t)b * nslice + s] = g;
}

// ---- the emitted token: inverse CDF over the final node's residual ---------------
template <bool VEC>
__global__ __launch_bounds__(SA_THREADS) void sampled_pick_kernel(SampledArgs a, int nslice) {
  __shared__ float scan[SA_THREADS];
  __shared__ RmEntry rml[SA_RM];
  __shared__ SampState sh_st;
  __shared__ int sh_node, sh_nan, pick_s, found;
  __shared__ float pick_thr;
  const SampScratch sc = sa_carve(a.scratch, a.scratch_batch, a.max_tree, nslice);
  const int b = blockIdx.x, tid = threadIdx.x, V = a.vocab;
  const size_t row0 = (size_t)b * a.max_tree;
  WalkEnd w;
  if (tid < 64) {
    w = walk_tree(a, sc, nslice, b);
    rml[tid] = w.e;
    // inclusive scan of the slice sums, in slice order
    const float ps = tid < nslice ? sc.dpart[(size_t)b * nslice + tid] : 0.f;
    float inc = ps;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float up = __shfl_up(inc, o, 64);
      if (tid >= o) inc += up;
    }
    const float total = __shfl(inc, 63, 64);
    const float thr = a.u_final[row0 + w.node] * total;
    const uint64_t hit = __ballot(tid < nslice && inc > thr);
    const int si = hit ? __ffsll((unsigned long long)hit) - 1 : -1;
    if (tid == 0) {
      sh_st = w.st;
      sh_node = w.node;
      sh_nan = w.nan;
      pick_s = si;
      found = -1;
    }
    if (si >= 0 && tid == si) pick_thr = thr - (inc - ps);
  }
  __syncthreads();
  int emitted = -1;
  if (!sh_nan) {
    const int si = pick_s;
    if (si < 0) {
      emitted = V - 1;
    } else {
      const SampState st = sh_st;
      const Norm nm = norm_of(st, a.inv_t);
      const size_t fr = row0 + sh_node;
      const float* lg = a.logits + fr * V;
      const float* qd = a.q ? a.q + fr * V : nullptr;
      // exact residual inside slice si, thread ranges in order
      int clo, chi;
      slice_range(V, nslice, si, clo, chi);
      const int per = (chi - clo + SA_THREADS - 1) / SA_THREADS;
      const int v0 = min(chi, clo + tid * per), v1 = min(chi, v0 + per);
      const int nrm = st.n_rm;
      const float af = st.a;
      auto r_at = [&](int v) {
        float r = resid(lg[v], (nrm > 0 && qd) ? qd[v] : 0.f, af, nm);
        for (int j = 0; j < nrm; ++j) r = rml[j].tok == v ? rml[j].f : r;
        return r;
      };
      float cs = 0.f;
      for (int v = v0; v < v1; ++v) cs += r_at(v);
      scan[tid] = cs;
      __syncthreads();
      for (int off = 1; off < SA_THREADS; off <<= 1) {
        const float add = tid >= off ? scan[tid - off] : 0.f;
        __syncthreads();
        scan[tid] += add;
        __syncthreads();
      }
      const float thr = pick_thr;
      const float excl = tid > 0 ? scan[tid - 1] : 0.f;
      if (v0 < v1 && excl <= thr && thr < scan[tid]) {
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
      emitted = found >= 0 ? found : chi - 1;
    }
  }
  if (tid < 64) {
    int32_t* out = a.result + (size_t)b * result_stride(a.max_depth);
    const int D = a.max_depth;
    if (tid == 0) {
      out[0] = w.L;
      out[1] = w.nan;
    }
    if (tid <= D) out[2 + tid] = tid < w.L ? a.token[row0 + w.pathv] : (tid == w.L ? emitted : -1);
    if (tid < D) out[3 + D + tid] = tid < w.L ? w.pathv : -1;
  }
}

template <bool VEC>
static void launch_all(const SampledArgs& a, const int* rows_with, int max_children, int ns, hipStream_t s) {
  // a deterministic draft's walk tests the children itself: no step launches
  const int steps = a.q ? max_children : 0;
  hipLaunchKernelGGL(sampled_norm_kernel<VEC>, dim3(ns, rows_with[0]), dim3(SA_THREADS), 0, s, a, ns,
                     steps > 0 ? rows_with[1] : 0);
  for (int k = 0, base = 0, prev = 0; k < steps; prev = base, base += rows_with[++k])
    hipLaunchKernelGGL(sampled_step_kernel<VEC>, dim3(ns, rows_with[k + 1]), dim3(SA_THREADS), 0, s, a, ns, k, base,
                       prev);
  hipLaunchKernelGGL(sampled_draw_sums_kernel<VEC>, dim3(ns, a.batch), dim3(SA_THREADS), 0, s, a, ns);
  hipLaunchKernelGGL(sampled_pick_kernel<VEC>, dim3(a.batch), dim3(SA_THREADS), 0, s, a, ns);
}

hipError_t launch_sampled_accept(const SampledArgs& a, const int* rows_with, int max_children, hipStream_t s) {
  if (a.batch < 1 || a.batch > a.scratch_batch || !a.order || !a.step_child || !a.step_token || a.vocab < 1 ||
      a.max_tree < 1 || a.max_tree > SA_RM || a.max_depth >= a.max_tree || max_children < 0 ||
      max_children >= a.max_tree || !a.scratch || !rows_with || rows_with[0] < 1)
    return hipErrorInvalidValue;
  const int ns = sampled_nslice(a.vocab);
  const bool vec = a.vocab % 4 == 0 && (reinterpret_cast<uintptr_t>(a.logits) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(a.q) & 15) == 0;
  if (vec)
    launch_all<true>(a, rows_with, max_children, ns, s);
  else
    launch_all<false>(a, rows_with, max_children, ns, s);
  return hipGetLastError();
}

// Fixed scratch of the allocation-free walk.  Host code never uses the
// array's name as an address (on the host it names a stand-in, not device
// memory): the device address comes from hipGetSymbolAddress, once per device
// with that device current, and is kept per device.
static __device__ __align__(256) char scratch[kStaticScratchBytes];

hipError_t static_scratch(void** ptr, size_t* bytes) {
  constexpr int kMaxDevices = 64;
  static void* addr[kMaxDevices] = {};
  static std::mutex mu;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  *bytes = kStaticScratchBytes;
  return hipSuccess;
}

}  // namespace griffin
