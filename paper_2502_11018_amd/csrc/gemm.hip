// Skinny bf16 GEMM for the verify pass: out = X W^T with X the activations of
// the tree nodes ([rows][K], rows = 64 per tile) and W a weight matrix [N][K]
// streamed once from HBM.  At tree sizes of ~64 rows the weights dominate the
// traffic (64 flop per weight byte, far below the MFMA ridge), so the kernel is
// built to keep HBM busy: every weight byte is loaded exactly once with 16-byte
// loads, whole 128-byte lines per row, and the activations are re-read from
// L1/L2.
//
// Tiling.  A workgroup owns NB blocks of 32 weight rows and one 64-row tile of
// X.  Its KW waves split the K range (and `splits` workgroups split it
// further); each wave accumulates the full (32*NB) x 64 tile with
// v_mfma_f32_32x32x16_bf16 (A = weight rows, B = activation rows, so D[n][m]),
// then the waves are summed through LDS in a fixed tree order.
//
// Operand mapping.  Lane l serves row l % 32 of a block and k-group g = l / 32.
// For each 64-wide K step it loads 32 consecutive bf16 (64 B) of its row
// starting at k0 + 32 g and feeds piece j (8 values) to MFMA j.  MFMA j thus
// sums k in {k0 + 8j + [0,8)} U {k0 + 32 + 8j + [0,8)}; the weight and the
// activation operands use the same permutation of K, so every dot product is
// unchanged while the two lanes of a row read one full 128-byte line.
//
// Output layout of the 32x32 MFMA (lane l, accumulator register r):
// m = l % 32, n = 8 (r / 4) + 4 (l / 32) + (r % 4).

#include "device_common.h"
#include "griffin_internal.h"

namespace griffin {

template <int EPI, int NB, int KW, int PF, bool NTL = false>
__global__ __launch_bounds__(64 * KW) void gemm_kernel(GemmArgs a) {
  constexpr int NT = NB * 32;
  constexpr int NREG = NB * 2 * 16;
  __shared__ float red[(KW > 1 ? KW / 2 : 1) * NREG * 64];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 31, g = lane >> 5;
  const int e = blockIdx.y;
  const int m_tile = blockIdx.x % a.m_tiles;
  const int n_tile = blockIdx.x / a.m_tiles;
  const int split = blockIdx.z;
  const int rows_e = a.count ? a.count[e] : a.m_tiles * 64;
  if (m_tile * 64 >= rows_e) return;  // uniform over the workgroup

  // ---- operand row pointers (row offset 32 g already applied)
  const uint16_t* W = a.W + (long long)e * a.w_estride;
  const uint16_t* wrow[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    int n;
    bool ok;
    if constexpr (EPI == EPI_SWIGLU) {
      const int c = n_tile * 32 + lr;
      ok = c < a.N;
      n = c + (b ? a.N : 0);
    } else {
      n = n_tile * NT + b * 32 + lr;
      ok = n < a.N;
    }
    wrow[b] = W + (long long)(ok ? n : 0) * a.K + 32 * g;
  }
  const uint16_t* xrow[2];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    const int ml = m_tile * 64 + mb * 32 + lr;
    int src;
    if (a.gather) src = ml < rows_e ? a.gather[e * a.cap + ml] : -1;
    else src = e * a.x_erows + ml;
    xrow[mb] = a.X + (long long)(src >= 0 ? src : 0) * a.ldx + 32 * g;
  }

  // ---- K range of this wave
  const int steps = (a.K + 63) >> 6;
  const int ws = split * KW + wave, nws = a.splits * KW;
  const int s0 = (int)((long long)steps * ws / nws);
  const int s1 = (int)((long long)steps * (ws + 1) / nws);

  f32x16 acc[NB][2];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[b][mb][r] = 0.f;

  if (s0 < s1) {
    u32x4 wb[PF][NB][4];
    u32x4 xb[PF][2][4];
    auto load_stage = [&](u32x4 (&wv)[NB][4], u32x4 (&xv)[2][4], int s) {
      const int kb = s * 64;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool kok = kb + 32 * g + 8 * j < a.K;
        const int off = kok ? kb + 8 * j : -32 * g;
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          u32x4 v = NTL ? ld_u4_nt(wrow[b] + off) : ld_u4(wrow[b] + off);
          wv[b][j] = kok ? v : zero_u4();
        }
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
          u32x4 v = ld_u4(xrow[mb] + off);
          xv[mb][j] = kok ? v : zero_u4();
        }
      }
    };
    auto compute = [&](const u32x4 (&wv)[NB][4], const u32x4 (&xv)[2][4]) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int mb = 0; mb < 2; ++mb)
            acc[b][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(wv[b][j]), as_bf16x8(xv[mb][j]),
                                                                 acc[b][mb], 0, 0, 0);
    };
    // Register ring of PF stages: stage s lives in slot (s - s0) % PF.  The
    // main loop has no data-dependent branches, so the compiler's wait counts
    // leave PF - 1 stages in flight; loads past the end re-read the last step.
#pragma unroll
    for (int p = 0; p < PF - 1; ++p) load_stage(wb[p], xb[p], min(s0 + p, s1 - 1));
    int base = s0;
    for (; base + PF <= s1; base += PF) {
#pragma unroll
      for (int u = 0; u < PF; ++u) {
        load_stage(wb[(u + PF - 1) % PF], xb[(u + PF - 1) % PF], min(base + u + PF - 1, s1 - 1));
        compute(wb[u], xb[u]);
      }
    }
    const int rem = s1 - base;  // < PF steps, already loaded in slots 0 .. rem-1
#pragma unroll
    for (int u = 0; u < PF - 1; ++u)
      if (u < rem) compute(wb[u], xb[u]);
  }

  // ---- fixed-order tree reduction over the KW waves; wave 0 ends with the sum
#pragma unroll
  for (int half = KW / 2; half >= 1; half >>= 1) {
    __syncthreads();
    if (wave >= half && wave < 2 * half) {
      float* dst = red + (wave - half) * (NREG * 64);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) dst[((b * 2 + mb) * 16 + r) * 64 + lane] = acc[b][mb][r];
    }
    __syncthreads();
    if (wave < half) {
      const float* src = red + wave * (NREG * 64);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[b][mb][r] += src[((b * 2 + mb) * 16 + r) * 64 + lane];
    }
  }
  if (wave != 0) return;

  // ---- epilogues (wave 0, MFMA output layout)
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    const int ml = m_tile * 64 + mb * 32 + lr;   // tile row
    const bool row_ok = ml < rows_e;
    const long long orow = (long long)e * a.o_erows + ml;
    if constexpr (EPI == EPI_STORE) {
      if (!row_ok) continue;
      float* out = a.out + (long long)split * a.out_split_stride + orow * a.ldo;
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int n = n_tile * NT + b * 32 + 8 * rg + 4 * g;
          if (n < a.N) {
            float4 v = make_float4(acc[b][mb][4 * rg], acc[b][mb][4 * rg + 1], acc[b][mb][4 * rg + 2],
                                   acc[b][mb][4 * rg + 3]);
            *reinterpret_cast<float4*>(out + n) = v;
          }
        }
    } else if constexpr (EPI == EPI_SWIGLU) {
      if (!row_ok) continue;
      uint16_t* out = a.act + orow * a.lda;
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int n = n_tile * 32 + 8 * rg + 4 * g;
        if (n < a.N) {
          float h[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) h[i] = silu_f32(acc[0][mb][4 * rg + i]) * acc[1][mb][4 * rg + i];
          uint2 v = make_uint2(pack_bf16x2(h[0], h[1]), pack_bf16x2(h[2], h[3]));
          *reinterpret_cast<uint2*>(out + n) = v;
        }
      }
    } else {  // EPI_ARGMAX
      float best = -INFINITY;
      int bidx = 0x7fffffff;
      int nan_cnt = 0;
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int n = n_tile * NT + b * 32 + 8 * rg + 4 * g + i;
            const float v = acc[b][mb][4 * rg + i];
            if (n < a.N) {
              if (v != v) ++nan_cnt;
              else if (v > best || (v == best && n < bidx)) { best = v; bidx = n; }
            }
          }
      const float ob = __shfl_xor(best, 32, 64);
      const int oi = __shfl_xor(bidx, 32, 64);
      nan_cnt += __shfl_xor(nan_cnt, 32, 64);
      if (ob > best || (ob == best && oi < bidx)) { best = ob; bidx = oi; }
      if (g == 0) {
        a.pmax[orow * a.ld_part + n_tile] = best;
        a.pidx[orow * a.ld_part + n_tile] = bidx;
        a.pnan[orow * a.ld_part + n_tile] = nan_cnt;
      }
      if (a.logits && orow < a.logit_rows) {
        float* out = a.logits + orow * a.ld_logits;
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int rg = 0; rg < 4; ++rg) {
            const int n = n_tile * NT + b * 32 + 8 * rg + 4 * g;
            if (n < a.N)
              *reinterpret_cast<float4*>(out + n) =
                  make_float4(acc[b][mb][4 * rg], acc[b][mb][4 * rg + 1], acc[b][mb][4 * rg + 2],
                              acc[b][mb][4 * rg + 3]);
          }
      }
    }
  }
}

template <int EPI, int NB, int KW, int PF = 2>
static hipError_t launch_one(const GemmArgs& a, int experts, hipStream_t s) {
  const int nt = EPI == EPI_SWIGLU ? (a.N + 31) / 32 : (a.N + NB * 32 - 1) / (NB * 32);
  dim3 grid(nt * a.m_tiles, experts, EPI == EPI_STORE ? a.splits : 1);
  hipLaunchKernelGGL((gemm_kernel<EPI, NB, KW, PF>), grid, dim3(64 * KW), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemm(int epi, int nb, int kw, const GemmArgs& a, int experts, hipStream_t s) {
  if (epi == EPI_STORE && nb == 1 && kw == 4) return launch_one<EPI_STORE, 1, 4>(a, experts, s);
  if (epi == EPI_STORE && nb == 1 && kw == 8) return launch_one<EPI_STORE, 1, 8>(a, experts, s);
  if (epi == EPI_STORE && nb == 2 && kw == 4) return launch_one<EPI_STORE, 2, 4>(a, experts, s);
  if (epi == EPI_SWIGLU && nb == 2 && kw == 4) return launch_one<EPI_SWIGLU, 2, 4>(a, experts, s);
  if (epi == EPI_SWIGLU && nb == 2 && kw == 2) return launch_one<EPI_SWIGLU, 2, 2>(a, experts, s);
  if (epi == EPI_ARGMAX && nb == 1 && kw == 4) return launch_one<EPI_ARGMAX, 1, 4>(a, experts, s);
  if (epi == EPI_ARGMAX && nb == 1 && kw == 2) return launch_one<EPI_ARGMAX, 1, 2>(a, experts, s);
  return hipErrorInvalidValue;
}

}  // namespace griffin
