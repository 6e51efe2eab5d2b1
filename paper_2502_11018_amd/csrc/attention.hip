// Tree-masked attention of the verify pass.
//
// A tree node r of sequence b sees the cached prefix slots [0, P_b) and the
// tree slots P_b + j for every node j on its root path (bit j of anc[r]).  One
// wavefront handles one query head and a block of 32 tree rows over one split
// of the key range; splits are merged by attn_combine with the usual
// (max, sum, weighted output) rescaling in a fixed order.
//
// Per 32-key block the wave computes S^T = K Q^T and O^T += V^T P^T with
// v_mfma_f32_32x32x16_bf16, so that each lane owns one query row (column of
// the MFMA output) and the softmax bookkeeping is lane-local:
//  * Keys are fed to the MFMA in a permuted row order so that accumulator
//    register q of lane half h holds key 16 h + q of the block; the P operand
//    of the second product is then the lane's own registers 8 t .. 8 t + 7.
//  * V is cached transposed ([dim][slot]), so the V^T operand is one 16-byte
//    load of 8 consecutive slots per lane.
//  * Q and K use the same head-dim permutation as the projection GEMMs: a lane
//    reads 32 consecutive head dims and feeds 8 of them to each of 4 MFMAs.
// Scores are kept in the log2 domain (scaled by log2(e)/sqrt(dh)) and exp2 is
// used throughout; masked keys contribute exactly zero.

#include "device_common.h"
#include "griffin_internal.h"

namespace griffin {

template <int DH>
__global__ __launch_bounds__(64) void tree_attention_kernel(AttnArgs a) {
  constexpr int CH = DH / 64;   // 64-dim chunks of Q/K per lane pair
  constexpr int DB = DH / 32;   // 32-dim blocks of the output
  const int lane = threadIdx.x;
  const int col = lane & 31, hh = lane >> 5;
  const int split = blockIdx.x;
  const int hq = blockIdx.y;
  const int b = blockIdx.z / a.qblocks, qb = blockIdx.z % a.qblocks;
  const int hk = hq / (a.Hq / a.Hkv);
  const int n_nodes = a.meta.n_nodes[b];
  const int P = a.meta.prefix_len[b];
  const int Lb = P + n_nodes;
  const int qrows = a.qblocks * 32;

  float* po = a.part_o + ((((long long)b * a.Hq + hq) * a.splits + split) * qrows + qb * 32) * DH;
  float* pml = a.part_ml + ((((long long)b * a.Hq + hq) * a.splits + split) * qrows + qb * 32) * 2;

  if (qb * 32 >= n_nodes) return;  // no live query rows in this block

  // key range of this split, in whole 32-key blocks
  const int nblk = (Lb + 31) >> 5;
  const int kb0 = (int)((long long)nblk * split / a.splits);
  const int kb1 = (int)((long long)nblk * (split + 1) / a.splits);

  // query row of this lane
  const int qi = qb * 32 + col;
  const bool qlive = qi < n_nodes;
  const int qr = b * a.max_tree + (qlive ? qi : 0);
  const uint64_t anc = qlive ? a.meta.anc[qr] : 0ull;

  // Q^T operand (B): lane (col = query row, hh = k-group), 32 dims per chunk
  u32x4 qf[CH][4];
  {
    const uint16_t* qp = a.q + ((long long)qr * a.Hq + hq) * DH + 32 * hh;
#pragma unroll
    for (int c = 0; c < CH; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) qf[c][j] = ld_u4(qp + 64 * c + 8 * j);
  }

  const long long head = ((long long)b * a.Hkv + hk) * a.kv_cap * DH;
  const uint16_t* kbase = a.k_cache + head;
  const uint16_t* vbase = a.v_cache + head;
  // MFMA row -> key offset inside a 32-key block: row 8q + 4h + e holds key 16h + 4q + e
  const int krow = 16 * ((col >> 2) & 1) + 4 * (col >> 3) + (col & 3);

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 oacc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[d][r] = 0.f;

  for (int kb = kb0; kb < kb1; ++kb) {
    const int key0 = kb * 32;
    // ---- S^T = K Q^T (rows: keys, cols: queries)
    u32x4 kf[CH][4];
    {
      const uint16_t* kp = kbase + (long long)(key0 + krow) * DH + 32 * hh;
#pragma unroll
      for (int c = 0; c < CH; ++c)
#pragma unroll
        for (int j = 0; j < 4; ++j) kf[c][j] = ld_u4(kp + 64 * c + 8 * j);
    }
    // V^T operand (A): lane (dim row col of block d, k-group hh); step t covers
    // keys 16 hh + 8 t + [0, 8)
    u32x4 vf[DB][2];
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int t = 0; t < 2; ++t)
        vf[d][t] = ld_u4(vbase + (long long)(32 * d + col) * a.kv_cap + key0 + 16 * hh + 8 * t);

    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
    for (int c = 0; c < CH; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[c][j]), as_bf16x8(qf[c][j]), s, 0, 0, 0);

    // ---- mask + online softmax (this lane: query qi, keys key0 + 16 hh + r)
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = key0 + 16 * hh + r;
      bool vis;
      if (key < P) vis = true;
      else {
        const int j = key - P;
        vis = (j < n_nodes) && ((anc >> j) & 1ull);
      }
      s[r] = vis ? s[r] * a.scale_log2 : -INFINITY;
      mx = fmaxf(mx, s[r]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    float psum = 0.f;
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      p[r] = exp2f(s[r] - m_use);
      psum += p[r];
    }
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[d][r] *= alpha;

    // keys at or beyond the end of the sequence may hold stale or never
    // written cache bytes; zero their V so that 0 * garbage cannot appear
    if (key0 + 32 > Lb) {
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int kfirst = key0 + 16 * hh + 8 * t;
#pragma unroll
          for (int w = 0; w < 4; ++w) {  // bf16 element 2w is the low half of dword w
            uint32_t v = vf[d][t][w];
            if (kfirst + 2 * w >= Lb) v &= 0xffff0000u;
            if (kfirst + 2 * w + 1 >= Lb) v &= 0x0000ffffu;
            vf[d][t][w] = v;
          }
        }
    }

    // ---- O^T += V^T P^T
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      u32x4 pf;
      pf[0] = pack_bf16x2(p[8 * t + 0], p[8 * t + 1]);
      pf[1] = pack_bf16x2(p[8 * t + 2], p[8 * t + 3]);
      pf[2] = pack_bf16x2(p[8 * t + 4], p[8 * t + 5]);
      pf[3] = pack_bf16x2(p[8 * t + 6], p[8 * t + 7]);
#pragma unroll
      for (int d = 0; d < DB; ++d)
        oacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vf[d][t]), as_bf16x8(pf), oacc[d], 0, 0, 0);
    }
  }

  // ---- partials: O^T layout, lane owns query col, dims 32 d + 8 (r/4) + 4 hh + r%4
  float* orow = po + (long long)col * DH;
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg)
      *reinterpret_cast<float4*>(orow + 32 * d + 8 * rg + 4 * hh) =
          make_float4(oacc[d][4 * rg], oacc[d][4 * rg + 1], oacc[d][4 * rg + 2], oacc[d][4 * rg + 3]);
  if (hh == 0) {
    pml[2 * col] = m_run;
    pml[2 * col + 1] = l_run;
  }
}

hipError_t launch_attention(const AttnArgs& a, int batch, hipStream_t s) {
  dim3 grid(a.splits, a.Hq, batch * a.qblocks);
  if (a.dh == 128) hipLaunchKernelGGL(tree_attention_kernel<128>, grid, dim3(64), 0, s, a);
  else if (a.dh == 64) hipLaunchKernelGGL(tree_attention_kernel<64>, grid, dim3(64), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// Merge the splits of every (row, head): o = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s.
// Absent rows get zeros.  One workgroup per row, one thread per (head, dim).
__global__ __launch_bounds__(256) void attn_combine_kernel(const float* __restrict__ part_o,
                                                           const float* __restrict__ part_ml, StepMeta meta,
                                                           int Hq, int dh, int splits, int qrows, int max_tree,
                                                           uint16_t* __restrict__ o_out) {
  const int r = blockIdx.x;
  const int b = r / max_tree, i = r % max_tree;
  const bool live = i < meta.n_nodes[b];
  for (int t = threadIdx.x; t < Hq * dh; t += blockDim.x) {
    const int h = t / dh, d = t % dh;
    float out = 0.f;
    if (live) {
      const long long base = ((long long)b * Hq + h) * splits;
      float M = -INFINITY;
      for (int s = 0; s < splits; ++s) M = fmaxf(M, part_ml[((base + s) * qrows + i) * 2]);
      float num = 0.f, den = 0.f;
      if (M != -INFINITY) {
        for (int s = 0; s < splits; ++s) {
          const float ms = part_ml[((base + s) * qrows + i) * 2];
          if (ms == -INFINITY) continue;
          const float w = exp2f(ms - M);
          num += w * part_o[((base + s) * qrows + i) * dh + d];
          den += w * part_ml[((base + s) * qrows + i) * 2 + 1];
        }
        out = num / den;
      }
    }
    o_out[(long long)r * Hq * dh + t] = f32_to_bf16(out);
  }
}

hipError_t launch_attn_combine(const float* part_o, const float* part_ml, StepMeta meta, int Hq, int dh, int splits,
                               int qrows, int max_tree, int batch, uint16_t* o_out, hipStream_t s) {
  hipLaunchKernelGGL(attn_combine_kernel, dim3(batch * max_tree), dim3(256), 0, s, part_o, part_ml, meta, Hq, dh,
                     splits, qrows, max_tree, o_out);
  return hipGetLastError();
}

}  // namespace griffin
