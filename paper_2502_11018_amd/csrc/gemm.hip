// Skinny bf16 GEMM of the verify pass: out = X W^T, X the activations of the
// tree rows ([rows][K], 64 rows per tile) and W a weight matrix [N][K] that is
// streamed once from HBM.  With ~64 rows the weights carry almost all the
// traffic (64 flop per weight byte, far below the MFMA ridge), so the kernel is
// shaped around keeping HBM busy:
//
// * Weights are repacked once (at context creation) into fragment order: a
//   block of 32 rows x 64 K (4 KB) holds, for piece j = 0..3 and lane
//   l = r + 32 g, the 8 values W[32 nb + r][64 s + 32 g + 8 j + 0..7] at
//   element j * 512 + 8 l, so one wave instruction reads one contiguous KB that
//   is directly an MFMA operand.  Blocks are laid out step-major over the
//   launch's wave streams (block (t, q, b) at ((t * Q + q) * NB + b) * 2048),
//   so at any moment all waves read one compact window of the matrix, the way
//   a plain streaming copy does.
// * Activations are produced in the same fragment order by the kernels that
//   write them (RMSNorm, attention merge, SwiGLU epilogue).  A workgroup's WN
//   waves own different weight rows over the same K range, so each 8 KB
//   activation stage is loaded once per workgroup into an LDS ring of PF slots
//   and read by all waves.
// * Each wave keeps PF - 1 stages of weight loads in flight in registers; the
//   main loop has no data-dependent branches.
//
// MFMA: v_mfma_f32_32x32x16_bf16 with A = weight rows, B = activation rows.
// Piece j of lane (r, g) feeds MFMA j, so MFMA j sums k in
// {64 s + 8 j + [0,8)} U {64 s + 32 + 8 j + [0,8)}: both operands use the same
// permutation of K and every dot product is unchanged.  Output layout (lane l,
// register i): m = l % 32, n = 8 (i / 4) + 4 (l / 32) + (i % 4).
//
// K is split across `splits` workgroups; each split writes fp32 partial sums
// that the consumer kernel adds in split order (no atomics, reproducible).

#include "device_common.h"
#include "griffin_internal.h"

namespace griffin {

// Merge the KS K slices of a workgroup in slice order through LDS (red: at
// least WN * NB * 8 KB, free: every wave's reads of it have returned).  Every
// wave of the workgroup calls it (its barriers are uniform); waves whose kh
// is not a slice index only take part in the barriers.  Slice 0 ends with the
// sum.
template <int NB, int WN, int KS>
__device__ __forceinline__ void ks_merge(f32x16 (&acc)[NB][2], float* red, int kh, int wc, int lane) {
  wait_vmcnt_lds<0>();
  __builtin_amdgcn_s_barrier();
  for (int k = 1; k < KS; ++k) {
    if (kh == k) {
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int i = 0; i < 16; ++i) red[(((wc * NB + b) * 2 + mb) * 16 + i) * 64 + lane] = acc[b][mb][i];
    }
    wait_vmcnt_lds<0>();
    __builtin_amdgcn_s_barrier();
    if (kh == 0) {
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[b][mb][i] += red[(((wc * NB + b) * 2 + mb) * 16 + i) * 64 + lane];
    }
    wait_vmcnt_lds<0>();
    __builtin_amdgcn_s_barrier();
  }
}

// The epilogues, every wave for its own NB column blocks of one 64-row tile.
template <int EPI, int NB, int WN>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& a, f32x16 (&acc)[NB][2], int e, int m_tile, int wg,
                                              int wc, int zsplit, int rows_e, int lane) {
  const int lr = lane & 31, g = lane >> 5;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    const int ml = m_tile * 64 + mb * 32 + lr;  // tile row
    const bool row_ok = ml < rows_e;
    const long long orow = (long long)e * a.o_erows + ml;
    if constexpr (EPI == EPI_STORE) {
      if (!row_ok) continue;
      float* out = a.out + (long long)zsplit * a.out_split_stride + orow * a.ldo;
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int n = ((wg * WN + wc) * NB + b) * 32 + 8 * rg + 4 * g;
          if (n < a.N)
            *reinterpret_cast<float4*>(out + n) = make_float4(acc[b][mb][4 * rg], acc[b][mb][4 * rg + 1],
                                                              acc[b][mb][4 * rg + 2], acc[b][mb][4 * rg + 3]);
        }
    } else if constexpr (EPI == EPI_SWIGLU) {
      // blocks [0, NB/2) hold gate rows, block b + NB/2 the up rows of block b
      static_assert(EPI != EPI_SWIGLU || NB % 2 == 0, "SwiGLU pairs gate and up blocks");
      constexpr int HB = NB / 2;
      if (!row_ok) continue;
#pragma unroll
      for (int hb = 0; hb < HB; ++hb)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int n = ((wg * WN + wc) * HB + hb) * 32 + 8 * rg + 4 * g;
          if (n < a.N) {
            float h[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) h[i] = silu_f32(acc[hb][mb][4 * rg + i]) * acc[hb + HB][mb][4 * rg + i];
            uint16_t* dst = a.act + xpack_off(orow, n, a.act_ks);
            const Hilo2 p0 = pack_hilo2(h[0], h[1]), p1 = pack_hilo2(h[2], h[3]);
            *reinterpret_cast<uint2*>(dst) = make_uint2(p0.hi, p1.hi);
            *reinterpret_cast<uint2*>(dst + XPACK_LO) = make_uint2(p0.lo, p1.lo);
          }
        }
    } else {  // EPI_ARGMAX: partial (max, argmax, second max, NaN count) over this wave's columns
      float best = -INFINITY, second = -INFINITY;
      int bidx = 0x7fffffff;
      int nan_cnt = 0;
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int n = ((wg * WN + wc) * NB + b) * 32 + 8 * rg + 4 * g + i;
            const float v = acc[b][mb][4 * rg + i];
            if (n < a.N) {
              if (v != v) ++nan_cnt;
              else top2_push(best, bidx, second, v, n);
            }
          }
      const float ob = __shfl_xor(best, 32, 64);
      const int oi = __shfl_xor(bidx, 32, 64);
      const float os = __shfl_xor(second, 32, 64);
      nan_cnt += __shfl_xor(nan_cnt, 32, 64);
      top2_merge(best, bidx, second, ob, oi, os);
      const int part = wg * WN + wc;
      if (g == 0) {
        a.pmax[orow * a.ld_part + part] = best;
        a.pmax2[orow * a.ld_part + part] = second;
        a.pidx[orow * a.ld_part + part] = bidx;
        a.pnan[orow * a.ld_part + part] = nan_cnt;
      }
      if (a.logits && orow < a.logit_rows) {
        float* out = a.logits + orow * a.ld_logits;
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int rg = 0; rg < 4; ++rg) {
            const int n = ((wg * WN + wc) * NB + b) * 32 + 8 * rg + 4 * g;
            if (n < a.N)
              *reinterpret_cast<float4*>(out + n) = make_float4(acc[b][mb][4 * rg], acc[b][mb][4 * rg + 1],
                                                                acc[b][mb][4 * rg + 2], acc[b][mb][4 * rg + 3]);
          }
      }
    }
  }
}

template <int EPI, int NB, int WN, int PF, int KS, bool XLO, int TG, bool NT_W>
__global__ __launch_bounds__(64 * WN * KS) void gemm_kernel(GemmArgs a) {
  // per step: {hi, lo} (XLO) or {hi} x {rows 0-31, 32-63} x 4 pieces of 1 KB,
  // for each of the TG 64-row tiles of the workgroup
  constexpr int XH = XLO ? 2 : 1;
  constexpr int XPIECES = 8 * XH;
  constexpr int XP = XPIECES / WN;          // activation pieces each wave stages per step and tile
  constexpr int LOADS = NB * 4 + TG * XP;   // vector-memory instructions per stage per wave
  static_assert(LOADS * (PF - 2) < 64, "wait count out of range");
  static_assert(PF >= 2 && XPIECES % WN == 0, "pipeline shape");
  static_assert(WN * NB * 8 <= PF * KS * XPIECES || KS == 1, "K-split merge buffer");
  static_assert(TG == 1 || KS == 1, "several tiles per workgroup merge no K slices");
  __shared__ u32x4 xs[PF][KS][TG][XPIECES][64];

  stamp_begin(a.stamp);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wc = wave % WN;            // column group of this wave
  const int kh = wave / WN;            // K slice of this wave inside the workgroup
  const int e = blockIdx.y;
  // XCD-aware decode: workgroups are dispatched round-robin over the 8 XCDs
  // (linear id % 8, and the grid's x extent is a multiple of 8), so the
  // workgroups of the groups of TG row tiles that stream the same weights
  // get the same id % 8 and the re-reads of those weights hit that XCD's L2.
  const int groups = (a.m_tiles + TG - 1) / TG;
  int tgrp = 0, wg = blockIdx.x;
  if (groups > 1) {
    const int grp = blockIdx.x / (8 * groups), r = blockIdx.x % (8 * groups);
    tgrp = r >> 3;
    wg = grp * 8 + (r & 7);
    if (wg >= a.n_wgs) return;  // padding of the grid to a multiple of 8 (uniform)
  }
  const int zsplit = blockIdx.z;       // output split (its KS slices are merged in the workgroup)
  const int split = zsplit * KS + kh;  // K slice of this wave's weight stream
  const int rows_e = a.count ? a.count[e] : a.m_tiles * 64;
  const int tile0 = tgrp * TG;         // first row tile of the workgroup
  if (tile0 * 64 >= rows_e) return;    // uniform over the workgroup

  const long long Q = (long long)a.n_wgs * a.splits * WN;
  const long long q = ((long long)split * a.n_wgs + wg) * WN + wc;
  const uint16_t* W = a.W + (long long)e * a.w_estride + q * NB * 2048 + lane * 8;
  const long long wstep = Q * NB * 2048;  // elements between consecutive steps of a stream
  // activation tiles of the group, the last one repeated where the group
  // runs past the tiles (their results are not stored)
  const uint16_t* X[TG];
#pragma unroll
  for (int g = 0; g < TG; ++g)
    X[g] = a.X + ((long long)(e * a.x_etiles + min(tile0 + g, a.m_tiles - 1)) * a.x_ks +
                  (long long)zsplit * KS * a.len) * XPACK_STEP + lane * 8;

  f32x16 acc[TG][NB][2];
#pragma unroll
  for (int g = 0; g < TG; ++g)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[g][b][mb][i] = 0.f;

  // Stage t: this wave's weight blocks into registers, its share of the
  // activation stage of every tile straight into LDS slot t % PF (lane l's 16
  // bytes land at the piece base + 16 l, which is the fragment order).
  // NT_W: non-temporal weight loads (see launch_gemm for where they are used)
  u32x4 wb[PF][NB][4];
  auto issue = [&](u32x4 (&wv)[NB][4], int slot, int t) {
    const uint16_t* wp = W + t * wstep;
    if constexpr (NT_W) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int b = 0; b < NB; ++b) wv[b][j] = ld_u4_nt(wp + b * 2048 + j * 512);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int b = 0; b < NB; ++b) wv[b][j] = ld_u4(wp + b * 2048 + j * 512);
    }
#pragma unroll
    for (int g = 0; g < TG; ++g)
#pragma unroll
      for (int p = 0; p < XP; ++p) {
        const int pp = wave * XP + p, sk = pp / XPIECES, pc = pp % XPIECES;  // slice, piece
        __builtin_amdgcn_global_load_lds(
            (const void*)(X[g] + ((long long)sk * a.len + t) * XPACK_STEP + pc * 512),
            (lds_void*)&xs[slot][sk][g][pc][0], 16, 0, 0);
      }
  };
  // Consume stage t from slot u: the weights times the activation's bf16 high
  // part plus, with XLO, its bf16 low part (two MFMAs into one accumulator),
  // for every tile with the same weight registers.
  auto compute = [&](int u) {
#pragma unroll
    for (int g = 0; g < TG; ++g) {
      u32x4 xv[XH][2][4];
#pragma unroll
      for (int h = 0; h < XH; ++h)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int j = 0; j < 4; ++j) xv[h][mb][j] = xs[u][kh][g][h * 8 + mb * 4 + j][lane];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int h = 0; h < XH; ++h)
#pragma unroll
          for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
              acc[g][b][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                  as_bf16x8(wb[u][b][j]), as_bf16x8(xv[h][mb][j]), acc[g][b][mb], 0, 0, 0);
    }
  };

  // Pipeline: stages t+1 .. t+PF-2 stay in flight while stage t is consumed.
  // At the top of iteration t the wave waits for its own stage-t loads
  // (vector-memory counters retire in issue order) and for its LDS reads of
  // slot (t-1) % PF; the barrier then makes every wave's share of stage t
  // visible and guarantees that no wave still reads slot (t-1) % PF, which
  // stage t+PF-1 overwrites.  A plain s_barrier: the explicit waits are the
  // only ones needed (a fence would drain all loads in flight).
  const int len = a.len;
#pragma unroll
  for (int p = 0; p < PF - 1; ++p) issue(wb[p], p, min(p, len - 1));
  int base = 0;
  for (; base + PF <= len; base += PF) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      wait_vmcnt_lds<(PF - 2) * LOADS>();
      __builtin_amdgcn_s_barrier();
      issue(wb[(u + PF - 1) % PF], (u + PF - 1) % PF, min(base + u + PF - 1, len - 1));
      compute(u);
    }
  }
  const int rem = len - base;  // < PF steps, already issued into slots 0 .. rem-1 (uniform)
  wait_vmcnt_lds<0>();
  __builtin_amdgcn_s_barrier();
#pragma unroll
  for (int u = 0; u < PF - 1; ++u)
    if (u < rem) compute(u);

  if constexpr (KS > 1) {
    ks_merge<NB, WN, KS>(acc[0], reinterpret_cast<float*>(&xs[0][0][0][0][0]), kh, wc, lane);
    if (kh != 0) return;
  }
#pragma unroll
  for (int g = 0; g < TG; ++g)
    if (tile0 + g < a.m_tiles && (tile0 + g) * 64 < rows_e)
      gemm_epilogue<EPI, NB, WN>(a, acc[g], e, tile0 + g, wg, wc, zsplit, rows_e, lane);
  stamp_end(a.stamp);
}

template <int EPI, int NB, int WN, int PF, int KS, bool XLO, int TG, bool NT_W>
static hipError_t launch_one(const GemmArgs& a, int experts, hipStream_t s) {
  const int groups = (a.m_tiles + TG - 1) / TG;
  const int gx = groups > 1 ? (a.n_wgs + 7) / 8 * 8 * groups : a.n_wgs;
  dim3 grid(gx, experts, a.splits / KS);
  hipLaunchKernelGGL((gemm_kernel<EPI, NB, WN, PF, KS, XLO, TG, NT_W>), grid, dim3(64 * WN * KS), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs& a, int experts, hipStream_t s) {
  const int epi = a.epi, nb = a.nb, wn = a.wn, pf = a.pf, ks = a.kslices;
  if (ks < 1 || a.splits % ks != 0) return hipErrorInvalidValue;
  const int tg = a.tg < 1 ? 1 : a.tg;
  // Non-temporal weight loads where they measured faster: the two-slice store
  // form (down) and the LM head over one row tile (a.nt; 189 -> 182 us, while
  // over eight tiles, whose re-reads L2 serves, they took it 891 -> 1217 us).
  // The one-slice store and the SwiGLU forms measured slower with them.
#define GRIFFIN_GEMM_CASE(E, B, N_, P, K_, T_)                                                         \
  if (epi == (E) && nb == (B) && wn == (N_) && pf == (P) && ks == (K_) && tg == (T_)) {               \
    constexpr bool nts = (E) == EPI_STORE && (K_) == 2;                                               \
    if constexpr ((E) == EPI_ARGMAX) {                                                                \
      if (a.nt)                                                                                       \
        return a.xlo ? launch_one<E, B, N_, P, K_, true, T_, true>(a, experts, s)                     \
                     : launch_one<E, B, N_, P, K_, false, T_, true>(a, experts, s);                   \
    }                                                                                                 \
    return a.xlo ? launch_one<E, B, N_, P, K_, true, T_, nts>(a, experts, s)                          \
                 : launch_one<E, B, N_, P, K_, false, T_, nts>(a, experts, s);                        \
  }
  // one 64-row tile per workgroup
  GRIFFIN_GEMM_CASE(EPI_STORE, 1, 4, 4, 1, 1)
  GRIFFIN_GEMM_CASE(EPI_STORE, 1, 4, 2, 1, 1)
  GRIFFIN_GEMM_CASE(EPI_STORE, 1, 4, 3, 2, 1)
  GRIFFIN_GEMM_CASE(EPI_SWIGLU, 2, 2, 3, 2, 1)
  GRIFFIN_GEMM_CASE(EPI_SWIGLU, 2, 2, 2, 2, 1)
  GRIFFIN_GEMM_CASE(EPI_SWIGLU, 2, 2, 2, 1, 1)
  GRIFFIN_GEMM_CASE(EPI_ARGMAX, 2, 4, 4, 1, 1)
  GRIFFIN_GEMM_CASE(EPI_ARGMAX, 2, 4, 2, 1, 1)
  // two row tiles per workgroup sharing each weight fragment (batched rows)
  GRIFFIN_GEMM_CASE(EPI_SWIGLU, 4, 4, 3, 1, 2)
  GRIFFIN_GEMM_CASE(EPI_STORE, 2, 4, 3, 1, 2)
#undef GRIFFIN_GEMM_CASE
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------- weight packing ----
// One thread per 16-byte piece of the packed matrix: decode its (step, stream,
// block, piece, lane), read the 8 source values (zero outside [rows, K)).
__global__ __launch_bounds__(256) void pack_weight_kernel(const uint16_t* __restrict__ src, int rows, int K,
                                                          PackShape p, uint16_t* __restrict__ dst,
                                                          long long pieces) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= pieces) return;
  const int lane = (int)(i & 63);
  const int j = (int)((i >> 6) & 3);
  long long blk = i >> 8;  // ((t * Q + q) * nb + b)
  const int b = (int)(blk % p.nb);
  blk /= p.nb;
  const long long Q = (long long)p.n_wgs * p.splits * p.wn;
  const int q = (int)(blk % Q);
  const int t = (int)(blk / Q);
  const int wave = q % p.wn;
  const int rest = q / p.wn;
  const int wg = rest % p.n_wgs;
  const int split = rest / p.n_wgs;
  const int s = split * p.len + t;
  const int r = lane & 31, gg = lane >> 5;
  long long row;
  bool ok;
  if (p.swiglu) {  // blocks [0, nb/2): gate rows of the wave's column blocks; b + nb/2: their up rows
    const int hb = p.nb / 2;
    const int c = ((wg * p.wn + wave) * hb + b % hb) * 32 + r;
    ok = c < p.n_out;
    row = c + (b >= hb ? p.n_out : 0);
  } else {
    row = ((long long)(wg * p.wn + wave) * p.nb + b) * 32 + r;
    ok = row < rows;
  }
  const int k = s * 64 + 32 * gg + 8 * j;
  ok = ok && k < K;
  u32x4 v = zero_u4();
  if (ok) v = *reinterpret_cast<const u32x4*>(src + row * K + k);
  *reinterpret_cast<u32x4*>(dst + i * 8) = v;
}

hipError_t launch_pack_weight(const uint16_t* src, int rows, int K, const PackShape& p, uint16_t* dst,
                              hipStream_t s) {
  const long long pieces = packed_elems(p) / 8;
  const long long grid = (pieces + 255) / 256;
  hipLaunchKernelGGL(pack_weight_kernel, dim3((unsigned)grid), dim3(256), 0, s, src, rows, K, p, dst, pieces);
  return hipGetLastError();
}

}  // namespace griffin
