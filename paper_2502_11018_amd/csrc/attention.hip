// Tree-masked attention of the verify pass.
//
// A tree node r of sequence b sees the cached prefix slots [0, P_b) and the
// tree slots P_b + j for every node j on its root path (bit j of anc[r]).
// The prefix part is the bulk of the work and is computed here; the few tree
// keys of each node (its ancestors) are added by attn_combine in fp32, from
// fp32 copies of the tree K/V, while it merges the prefix splits.
//
// tree_attention_kernel: a workgroup handles one (sequence, KV head, block of
// 32 tree rows, prefix split, chunk of NW query heads of that KV head's
// group).  Its NW waves share every 32-key block of K and V, which the
// workgroup stages once into an LDS ring with global_load_lds_dwordx4 (each
// wave issues an equal share of the block's 1 KB pieces), so the cache is read
// once per head group rather than once per head.
//
// Per 32-key block each wave computes S^T = K Q^T and O^T += V^T P^T with
// v_mfma_f32_32x32x16_bf16, so that each lane owns one query row (column of
// the MFMA output) and the softmax bookkeeping is lane-local:
//  * Keys are fed to the MFMA in a permuted row order so that accumulator
//    register q of lane half h holds key 16 h + q of the block; the P operand
//    of the second product is then the lane's own registers 8 t .. 8 t + 7.
//  * V is cached in 32-slot tiles stored transposed ([tile][dim][32]), so a
//    block's V^T is one contiguous 8 KB tile.
//  * The ring holds each block in MFMA fragment order (piece, lane, 8 values):
//    the DMA gathers every lane's 16 bytes from the cache, and the compute
//    side reads each operand with one conflict-free ds_read_b128.
//  * Q and K use the same head-dim permutation as the projection GEMMs: a lane
//    reads 32 consecutive head dims and feeds 8 of them to each of 4 MFMAs.
//  * Q and P enter the matrix cores as split bf16 (hi + lo, two MFMAs each),
//    so only the cached K/V carry bf16 rounding.
// Scores are kept in the log2 domain (scaled by log2(e)/sqrt(dh)) and exp2 is
// used throughout; masked keys contribute exactly zero.

#include <type_traits>

#include "device_common.h"
#include "griffin_internal.h"

namespace griffin {

// LEAN: two workgroups per CU (at most 256 registers per lane): no
// cross-block software pipeline in a wave, K and V fragments read from LDS
// half a block at a time; the second wave of each SIMD hides what the first
// one waits on.  Chosen when a step has enough key-split units to fill two
// workgroups per CU (long prefixes, several sequences).
template <int DH, int NW, bool RAGGED, bool LEAN>
__global__ __launch_bounds__(64 * NW, LEAN ? 2 : 1) void tree_attention_kernel(AttnArgs a) {
  constexpr int CH = DH / 64;          // 64-dim chunks of Q/K per lane pair
  constexpr int DB = DH / 32;          // 32-dim blocks of the output
  constexpr int KP = CH * 4;           // 1 KB pieces of a K block
  constexpr int PIECES = KP + DB * 2;  // K and V pieces of one 32-key block
  constexpr int PPW = PIECES / NW;     // pieces each wave stages per block
  constexpr int D = ATTN_RING;         // ring slots
  static_assert(PIECES % NW == 0 && PPW * (D - 2) < 64, "ring shape");
  __shared__ u32x4 ring[D][PIECES][64];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = lane & 31, hh = lane >> 5;
  // Work units: the step's key-split table holds, per unit j, a sequence b,
  // one of its key splits and that sequence's split count (sequences get
  // splits in proportion to their prefix lengths).  XCD-aware decode:
  // workgroups are dispatched round-robin over the 8 XCDs (id % 8), so every
  // workgroup of one (unit, KV head) gets the same id % 8 and the K/V blocks
  // it re-reads are shared through that XCD's L2.
  const int G = a.Hq / a.Hkv;
  const int chunks = (G + NW - 1) / NW;
  const int per_unit = chunks * a.qblocks;
  const int id = blockIdx.x;
  const int rest = id >> 3;
  const int u_raw = (rest / per_unit) * 8 + (id & 7);
  // a workgroup past the last unit (the grid is rounded up) runs the
  // prologue's loads for unit 0 and leaves with the workgroups without live
  // rows: no branch before the loads, so the kernel arguments are fetched at
  // once
  const bool unit_live = u_raw < a.units * a.Hkv;  // uniform over the workgroup
  const int u = unit_live ? u_raw : 0;
  const int within = rest % per_unit;
  const int qb = within % a.qblocks;
  const int chunk = within / a.qblocks;
  const int hk = u % a.Hkv;
  // RAGGED: the unit comes from the step's split table; else every sequence
  // has a.sp splits and unit j is split j % sp of sequence j / sp
  int4 ent;
  if constexpr (RAGGED) {
    ent = a.meta.split_tab[u / a.Hkv];
    if (ent.x < 0) return;  // a unit without work this step
  } else {
    ent = make_int4((u / a.Hkv / a.sp) | ((u / a.Hkv % a.sp) << 16), a.sp, 0, 0);
  }
  const int b = ent.x & 0xffff, split = ent.x >> 16, nsplit = ent.y;
  const int gh = chunk * NW + w;           // head within the group
  const bool head_live = gh < G;           // wave-uniform
  const int hq = hk * G + (head_live ? gh : 0);
  const int qrows = a.qblocks * 32;

  // Q^T operand (B): lane (col = query row, hh = k-group), 32 dims per chunk;
  // split bf16, so S = K (q_hi + q_lo).  Loaded before the per-sequence
  // metadata is known (rows past the tree hold stale values and are never
  // written out; the row index stays inside the sequence's max_tree rows).
  const int qi = qb * 32 + col;
  const int qr = b * a.max_tree + min(qi, a.max_tree - 1);
  u32x4 qf[2][CH][4];
  {
    const long long qo = ((long long)qr * a.Hq + hq) * DH + 32 * hh;
#pragma unroll
    for (int c = 0; c < CH; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        qf[0][c][j] = ld_u4(a.q + qo + 64 * c + 8 * j);
        qf[1][c][j] = ld_u4(a.q_lo + qo + 64 * c + 8 * j);
      }
  }

  const int P = RAGGED ? ent.z : a.meta.prefix_len[b];
  const int n_nodes = RAGGED ? ent.w : a.meta.n_nodes[b];

  // prefix key range of this split, in whole 32-key blocks
  const int nblk = (P + 31) >> 5;
  const int kb0 = (int)((long long)nblk * split / nsplit);
  const int kb1 = (int)((long long)nblk * (split + 1) / nsplit);
  const int nb = kb1 - kb0;

  const long long head = ((long long)b * a.Hkv + hk) * a.kv_cap * DH;
  const uint16_t* kbase = a.k_cache + head;
  const uint16_t* vbase = a.v_cache + head;
  // MFMA row -> key offset inside a 32-key block: row 8q + 4h + e holds key 16h + 4q + e
  const int krow = 16 * ((col >> 2) & 1) + 4 * (col >> 3) + (col & 3);
  // this lane's byte offset inside a block, for each piece this wave stages
  // (each DMA takes a wave-uniform block base plus this offset)
  const int wu = __builtin_amdgcn_readfirstlane(w);
  uint32_t goff[PPW];
#pragma unroll
  for (int p = 0; p < PPW; ++p) {
    const int pc = wu * PPW + p;
    if (pc < KP) {
      const int c = pc >> 2, j = pc & 3;
      goff[p] = 2u * (krow * DH + 64 * c + 32 * hh + 8 * j);
    } else {
      const int v = pc - KP, d = v >> 1, t = v & 1;
      goff[p] = 2u * ((32 * d + col) * 32 + 16 * hh + 8 * t);
    }
  }
  auto issue = [&](int slot, int kb) {
#pragma unroll
    for (int p = 0; p < PPW; ++p) {
      const int pc = wu * PPW + p;
      const char* blk = reinterpret_cast<const char*>((pc < KP ? kbase : vbase) + (long long)kb * 32 * DH);
      __builtin_amdgcn_global_load_lds((const void*)(blk + goff[p]), (lds_void*)&ring[slot][pc][0], 16, 0, 0);
    }
  };
  // The first D - 1 blocks go out as soon as the prefix length is known (the
  // longest latency of the prologue), before the check for live rows: a
  // workgroup without live rows lets them land and leaves.
  if (nb > 0) {
#pragma unroll
    for (int i = 0; i < D - 1; ++i) issue(i, kb0 + min(i, nb - 1));
  }
  if (!unit_live || qb * 32 >= n_nodes) {  // no unit, or no live query rows in this block (uniform)
    wait_vmcnt_lds<0>();
    return;
  }

  // Softmax reference: each lane's row uses a fixed reference m_ref (log2
  // domain), the maximum of its scores in the split's first block, so the
  // output accumulators are never rescaled inside the block loop (a rescale
  // there would make the compiler shuttle them between register files every
  // block), and later blocks compute no maximum at all.  Later scores may
  // exceed m_ref: a row whose sum of p = 2^(s - m_ref) passes 2^64 (which
  // every row with a key more than 64 above its reference does) is flagged,
  // and the merge recomputes that split exactly.  So p needs no clamp: only
  // flagged rows can overflow, and a NaN score stays NaN (a clamp cost 0.8 us
  // per launch, the running maximum 10 us at 16384 keys per sequence).
  float m_ref = -INFINITY, l_run = 0.f;
  f32x16 oacc[DB];

  // QK: S^T = K Q^T for the block in `slot` (rows: keys, cols: queries),
  // q = q_hi + q_lo.
  auto qk = [&](int slot) {
    // all K fragments are read before the first MFMA, so the LDS latency is
    // paid once per block (LEAN: once per 64-dim chunk)
    constexpr int KR = LEAN ? 4 : CH * 4;  // K fragments held at once
    f32x16 sacc;
#pragma unroll
    for (int r = 0; r < 16; ++r) sacc[r] = 0.f;
#pragma unroll
    for (int c0 = 0; c0 < CH * 4; c0 += KR) {
      u32x4 kf[KR];
#pragma unroll
      for (int x = 0; x < KR; ++x) kf[x] = ring[slot][c0 + x][lane];
#pragma unroll
      for (int x = 0; x < KR; ++x)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[x]), as_bf16x8(qf[h][(c0 + x) / 4][(c0 + x) % 4]),
                                                         sacc, 0, 0, 0);
    }
    return sacc;
  };

  // SV: softmax of one block's scores and O^T += V^T P^T.  TAIL is true only
  // for the last prefix block when P is not a multiple of 32: its keys at or
  // beyond P get probability 0 and their V is zeroed (those slots hold tree
  // or stale values), with branch-free selects.  `first` marks the block
  // that sets m_ref.
  auto sv = [&](auto tail, const f32x16& sacc, int slot, int kb, bool first) {
    constexpr bool TAIL = decltype(tail)::value;
    const int key0 = kb * 32;
    // mask (this lane: keys key0 + 16 hh + r); the log2-domain scale is
    // applied inside the exponent (scale > 0 commutes with max)
    float s[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s[r] = sacc[r];
      if constexpr (TAIL) s[r] = (key0 + 16 * hh + r < P) ? s[r] : -INFINITY;
    }
    if (first) {  // wave-uniform
      float mx = fmaxf(fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])), fmaxf(fmaxf(s[4], s[5]), fmaxf(s[6], s[7])));
      mx = fmaxf(mx, fmaxf(fmaxf(fmaxf(s[8], s[9]), fmaxf(s[10], s[11])),
                           fmaxf(fmaxf(s[12], s[13]), fmaxf(s[14], s[15]))));
      m_ref = fmaxf(mx, __shfl_xor(mx, 32, 64)) * a.scale_log2;
    }
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) p[r] = __builtin_amdgcn_exp2f(fmaf(s[r], a.scale_log2, -m_ref));
    const float psum = ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7])) +
                       (((p[8] + p[9]) + (p[10] + p[11])) + ((p[12] + p[13]) + (p[14] + p[15])));
    l_run += psum + __shfl_xor(psum, 32, 64);

    // O^T += V^T P^T, P as split bf16 (p_hi + p_lo); all V fragments are
    // read before the first MFMA (LEAN: those of each 16-key half)
    constexpr int VT = LEAN ? 1 : 2;  // 16-key halves of V held at once
    u32x4 vfr[2][DB];
#pragma unroll
    for (int t = 0; t < VT; ++t)
#pragma unroll
      for (int d = 0; d < DB; ++d) vfr[t][d] = ring[slot][KP + d * 2 + t][lane];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (LEAN && t == 1) {
#pragma unroll
        for (int d = 0; d < DB; ++d) vfr[0][d] = ring[slot][KP + d * 2 + 1][lane];
      }
      const int tv = LEAN ? 0 : t;  // where this half's V fragments are held
      u32x4 pf[2];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const Hilo2 hl = pack_hilo2(p[8 * t + 2 * q], p[8 * t + 2 * q + 1]);
        pf[0][q] = hl.hi;
        pf[1][q] = hl.lo;
      }
      uint32_t keep[4];
      if constexpr (TAIL) {
        const int kfirst = key0 + 16 * hh + 8 * t;
#pragma unroll
        for (int q = 0; q < 4; ++q)  // bf16 element 2q is the low half of dword q
          keep[q] = (kfirst + 2 * q < P ? 0x0000ffffu : 0u) | (kfirst + 2 * q + 1 < P ? 0xffff0000u : 0u);
      }
#pragma unroll
      for (int d = 0; d < DB; ++d) {
        u32x4 vf = vfr[tv][d];
        if constexpr (TAIL) {
#pragma unroll
          for (int q = 0; q < 4; ++q) vf[q] &= keep[q];
        }
#pragma unroll
        for (int h = 0; h < 2; ++h)
          oacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vf), as_bf16x8(pf[h]), oacc[d], 0, 0, 0);
      }
    }
  };

  // Ring pipeline over the split's blocks (same structure as the GEMM's),
  // software-pipelined by one block: step i computes the scores of block
  // i + 1 (matrix cores) before the softmax and P V of block i (vector ALU,
  // then matrix cores), so the two overlap.  At the top of step i every wave
  // waits for its own DMA pieces of block i + 1 (vector-memory counters
  // retire in issue order) and for its LDS reads of earlier slots; the
  // barrier then publishes block i + 1 and frees the slot of block i - 1,
  // which block i + D - 1 overwrites.  Issues past the last block re-read it
  // into slots that are never consumed; every DMA has landed before the waves
  // leave.  The loop is unrolled by the ring depth (slot indices are
  // compile-time constants) and the split's last block, the only one that
  // can be partial (the TAIL form), is handled after it: with one path
  // through the loop body the accumulators stay in place and the only
  // vector-memory waits are the ones written here.
  static_assert(D >= 3, "one block of scores runs ahead of the ring");
  const int nfull = (kb0 + nb) * 32 <= P ? nb : nb - 1;
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[d][r] = 0.f;
  if (nb > 0 && LEAN) {
    // one block per step: wait for block i (blocks i+1 .. i+D-2 stay in
    // flight), publish it, refill the slot of block i - 1, then scores,
    // softmax and P V of block i
    auto step = [&](auto tail, int u, int i) {
      wait_vmcnt_lds<(D - 2) * PPW>();
      __builtin_amdgcn_s_barrier();
      issue((u + D - 1) % D, kb0 + min(i + D - 1, nb - 1));
      const f32x16 sc = qk(u);
      sv(tail, sc, u, kb0 + i, i == 0);
    };
    int base = 0;
    for (; base + D <= nfull; base += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) step(std::false_type{}, u, base + u);
    }
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int i = base + u;
      if (i < nfull) step(std::false_type{}, u, i);  // uniform
      else if (i < nb) step(std::true_type{}, u, i);
    }
    wait_vmcnt_lds<0>();
  } else if (nb > 0) {
    // Q (loaded before the first DMAs) and block 0
    wait_vmcnt_lds<(D - 2) * PPW>();
    __builtin_amdgcn_s_barrier();
    f32x16 sc = qk(0);
    // block i (slot u = i % D) when block i + 1 exists
    auto step = [&](auto tail, int u, int i) {
      wait_vmcnt_lds<(D - 3) * PPW>();
      __builtin_amdgcn_s_barrier();
      issue((u + D - 1) % D, kb0 + min(i + D - 1, nb - 1));
      const f32x16 sn = qk((u + 1) % D);
      // waves past the end of the head group compute a duplicate of the
      // group's first head and write nothing
      sv(tail, sc, u, kb0 + i, i == 0);
      sc = sn;
    };
    int base = 0;
    for (; base + D < nb && base + D <= nfull; base += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) step(std::false_type{}, u, base + u);
    }
    // the remaining blocks (at most D): full ones with a successor, then the
    // last block (full or partial)
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int i = base + u;
      if (i + 1 < nb) step(std::false_type{}, u, i);  // uniform; i + 1 < nb implies a full block
      else if (i + 1 == nb) {
        if (i < nfull) sv(std::false_type{}, sc, u, kb0 + i, i == 0);
        else sv(std::true_type{}, sc, u, kb0 + i, i == 0);
      }
    }
    wait_vmcnt_lds<0>();
  }
  // a row whose probabilities went past the cap marks its partial invalid
  // (l < 0); the merge recomputes that split exactly
  if (l_run > 0x1p64f) l_run = -1.f;

  // ---- partials, row-major [32 rows][DH].  The accumulators hold O^T (lane:
  // query col, dims 32 d + 8 (r/4) + 4 hh + r%4), so each wave transposes its
  // tile through its own part of the ring, which every wave has left after
  // this barrier: 16-byte chunk c of row `col` sits at chunk c ^ (col & 7)
  // (conflict-free writes and reads), and the global stores are contiguous.
  constexpr int CHUNKS = DH / 4;  // 16-byte chunks per row
  constexpr int RPI = 64 / CHUNKS;  // rows per wave-wide store
  static_assert(NW * 32 * DH * 4 <= (int)sizeof(ring), "transpose tiles fit in the ring");
  __builtin_amdgcn_s_barrier();
  if (!head_live) return;
  float* po = a.part_o + ((((long long)b * a.Hq + hq) * a.sp + split) * qrows + qb * 32) * DH;
  float* pml = a.part_ml + ((((long long)b * a.Hq + hq) * a.sp + split) * qrows + qb * 32) * 2;
  float* tile = reinterpret_cast<float*>(&ring[0][0][0]) + w * 32 * DH;
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int c = 8 * d + 2 * rg + hh;
      *reinterpret_cast<float4*>(tile + col * DH + 4 * (c ^ (col & 7))) =
          make_float4(oacc[d][4 * rg], oacc[d][4 * rg + 1], oacc[d][4 * rg + 2], oacc[d][4 * rg + 3]);
    }
  // rows of absent nodes are not stored (the merge reads live rows only)
  const int live_rows = min(32, n_nodes - qb * 32);
#pragma unroll
  for (int n = 0; n < 32 / RPI; ++n) {
    if (n * RPI >= live_rows) break;  // uniform
    const int r = n * RPI + lane / CHUNKS, c = lane % CHUNKS;
    *reinterpret_cast<float4*>(po + r * DH + 4 * c) =
        *reinterpret_cast<const float4*>(tile + r * DH + 4 * (c ^ (r & 7)));
  }
  if (hh == 0 && col < live_rows) {
    pml[2 * col] = m_ref;
    pml[2 * col + 1] = l_run;
    // the sequence's last split marks its unused slots empty, so that the
    // merge reads all sp slots without knowing the split count
    if (RAGGED && split == nsplit - 1)
      for (int s2 = nsplit; s2 < a.sp; ++s2) {
        float* pe = a.part_ml + ((((long long)b * a.Hq + hq) * a.sp + s2) * qrows + qb * 32 + col) * 2;
        pe[0] = -INFINITY;
        pe[1] = 0.f;
      }
  }
}

int attn_waves(int group) { return group >= 4 ? 4 : group >= 2 ? 2 : 1; }

template <int DH, int NW>
static void launch_attn_nw(const AttnArgs& a, dim3 grid, hipStream_t s) {
  // two workgroups per CU pay off once the grid fills them (measured at 8
  // sequences x 16384 keys); smaller grids keep the one-wave-per-SIMD form
  const bool lean = grid.x >= 512;
  if (a.meta.split_tab) {
    if (lean) hipLaunchKernelGGL((tree_attention_kernel<DH, NW, true, true>), grid, dim3(64 * NW), 0, s, a);
    else hipLaunchKernelGGL((tree_attention_kernel<DH, NW, true, false>), grid, dim3(64 * NW), 0, s, a);
  } else {
    if (lean) hipLaunchKernelGGL((tree_attention_kernel<DH, NW, false, true>), grid, dim3(64 * NW), 0, s, a);
    else hipLaunchKernelGGL((tree_attention_kernel<DH, NW, false, false>), grid, dim3(64 * NW), 0, s, a);
  }
}

template <int DH>
static void launch_attn_dh(const AttnArgs& a, int nw, dim3 grid, hipStream_t s) {
  if (nw == 4) launch_attn_nw<DH, 4>(a, grid, s);
  else if (nw == 2) launch_attn_nw<DH, 2>(a, grid, s);
  else launch_attn_nw<DH, 1>(a, grid, s);
}

hipError_t launch_attention(const AttnArgs& a, int batch, hipStream_t s) {
  if (a.batch != batch) return hipErrorInvalidValue;
  const int G = a.Hq / a.Hkv;
  const int nw = attn_waves(G);
  if (a.units < 1 || a.sp < 1 || a.sp > 16) return hipErrorInvalidValue;
  const int streams = a.units * a.Hkv;
  const int per_unit = ((G + nw - 1) / nw) * a.qblocks;
  dim3 grid(((streams + 7) / 8) * 8 * per_unit);
  if (a.dh == 128) launch_attn_dh<128>(a, nw, grid, s);
  else if (a.dh == 64) launch_attn_dh<64>(a, nw, grid, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// Finish attention for every (row, head): merge the prefix splits and add the
// node's tree keys.  Prefix split s contributes (m_s, l_s, o_s) in the log2
// domain; the tree keys are the node's ancestors and itself (bits of anc),
// scored in fp32 from q = q_hi + q_lo and the fp32 tree K/V, with a running
// (m_t, l_t, o_t).  Then o = (sum_s 2^(m_s - M) o_s + 2^(m_t - M) o_t) /
// (sum_s 2^(m_s - M) l_s + 2^(m_t - M) l_t).  Absent rows get zeros.  One
// workgroup per row, one thread per (head, 4 dims); the dot products of a
// tree key reduce over the head's dh/4 threads with xor shuffles (a fixed
// order).  It reads the first MAXS of the sp partial slots of each (sequence,
// head): the step's largest split count rounded up, so that a batch whose
// sequences all hold the even share does not read the slots kept for
// uneven ones.  The merged rows are written fragment-packed split bf16 (o_ks K
// steps per tile) as the activation operand of the output projection.
template <int MAXS, bool RAGGED>
__global__ __launch_bounds__(256) void attn_combine_kernel(const float* __restrict__ part_o,
                                                           const float* __restrict__ part_ml, StepMeta meta,
                                                           int Hq, int Hkv, int dh, int sp, int qrows, int max_tree,
                                                           const uint16_t* __restrict__ q,
                                                           const uint16_t* __restrict__ q_lo, TreeKV32 tree,
                                                           PrefixKV prefix, float scale_log2,
                                                           uint16_t* __restrict__ o_out, int o_ks) {
  const int r = blockIdx.x;
  const int b = r / max_tree, i = r % max_tree;
  const int quads = dh / 4;
  const int t = blockIdx.y * blockDim.x + threadIdx.x;
  if (t >= Hq * quads) return;  // whole heads at a time (quads divides the block size)
  const int h = t / quads, d = (t % quads) * 4;
  // Every load that does not wait on another is issued first: the row's
  // metadata, its q and all split partials (row slots of absent nodes are
  // allocated, so these loads stay unconditional).
  const int n_nodes = meta.n_nodes[b];
  const int P = meta.prefix_len[b];
  const int ns = RAGGED ? meta.n_split[b] : MAXS;
  uint64_t anc = meta.anc[r];
  // the sequence's key splits fill the first of its sp slots and the
  // attention kernel marks the rest empty (m = -inf, l = 0), so the first
  // MAXS (at least the step's largest split count) hold every split
  const long long base = ((long long)b * Hq + h) * sp;
  float ms[MAXS], ls[MAXS];
  float4 os[MAXS];
#pragma unroll
  for (int s = 0; s < MAXS; ++s) {
    const long long row = (base + s) * qrows + i;
    ms[s] = part_ml[row * 2];
    ls[s] = part_ml[row * 2 + 1];
    os[s] = *reinterpret_cast<const float4*>(part_o + row * dh + d);
  }
  const long long qo = ((long long)r * Hq + h) * dh + d;
  const uint2 qh = *reinterpret_cast<const uint2*>(q + qo), ql = *reinterpret_cast<const uint2*>(q_lo + qo);
  float4 out = make_float4(0.f, 0.f, 0.f, 0.f);
  if (i < n_nodes) {  // uniform over the workgroup
    const int hk = h / (Hq / Hkv);
    const float q0 = bf16_to_f32(qh.x & 0xffff) + bf16_to_f32(ql.x & 0xffff);
    const float q1 = bf16_to_f32(qh.x >> 16) + bf16_to_f32(ql.x >> 16);
    const float q2 = bf16_to_f32(qh.y & 0xffff) + bf16_to_f32(ql.y & 0xffff);
    const float q3 = bf16_to_f32(qh.y >> 16) + bf16_to_f32(ql.y >> 16);
    // splits flagged by the attention kernel (their p = 2^(s - m_ref) summed
    // past 2^64, where p may have overflowed): recompute
    // (m, l, o) over the split's prefix keys in fp32 from the bf16 cache, with
    // an exact running maximum
    {
      const int nblk = (P + 31) >> 5;
      const uint16_t* kh = prefix.k + ((long long)b * Hkv + hk) * prefix.kv_cap * dh + d;
      const uint16_t* vh = prefix.v + ((long long)b * Hkv + hk) * prefix.kv_cap * dh;
#pragma unroll
      for (int s = 0; s < MAXS; ++s) {
        if (!(ls[s] < 0.f)) continue;  // uniform over the head's lanes
        const int k0 = 32 * (int)((long long)nblk * s / ns);
        const int k1 = min(P, 32 * (int)((long long)nblk * (s + 1) / ns));
        float m = -INFINITY, l = 0.f;
        float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int key = k0; key < k1; ++key) {
          const uint2 kk = *reinterpret_cast<const uint2*>(kh + (long long)key * dh);
          float dot = q0 * bf16_to_f32(kk.x & 0xffff) + q1 * bf16_to_f32(kk.x >> 16) +
                      q2 * bf16_to_f32(kk.y & 0xffff) + q3 * bf16_to_f32(kk.y >> 16);
          for (int o2 = quads >> 1; o2 > 0; o2 >>= 1) dot += __shfl_xor(dot, o2, 64);
          const float sj = dot * scale_log2;
          const float mn = fmaxf(m, sj);
          const float al = exp2f(m - mn), e = exp2f(sj - mn);
          // V tiles: element (key, dim) at ((key / 32) * dh + dim) * 32 + key % 32
          const uint16_t* vk = vh + ((long long)(key >> 5) * dh + d) * 32 + (key & 31);
          l = l * al + e;
          o = make_float4(o.x * al + e * bf16_to_f32(vk[0]), o.y * al + e * bf16_to_f32(vk[32]),
                          o.z * al + e * bf16_to_f32(vk[64]), o.w * al + e * bf16_to_f32(vk[96]));
          m = mn;
        }
        ms[s] = m;
        ls[s] = l;
        os[s] = o;
      }
    }
    // tree keys
    const float* tk = tree.k + ((long long)b * Hkv + hk) * max_tree * dh + d;
    const float* tv = tree.v + ((long long)b * Hkv + hk) * max_tree * dh + d;
    float mt = -INFINITY, lt = 0.f;
    float4 ot = make_float4(0.f, 0.f, 0.f, 0.f);
    constexpr int TB = 8;  // ancestors per batch: all their loads are issued before any is used
    while (anc) {          // uniform over the workgroup (one row)
      int js[TB];
      bool ok[TB];
#pragma unroll
      for (int u = 0; u < TB; ++u) {
        ok[u] = anc != 0;
        js[u] = ok[u] ? __builtin_ctzll(anc) : 0;
        anc &= anc - 1;
      }
      float4 k4[TB], v4[TB];
#pragma unroll
      for (int u = 0; u < TB; ++u) {
        k4[u] = *reinterpret_cast<const float4*>(tk + (long long)js[u] * dh);
        v4[u] = *reinterpret_cast<const float4*>(tv + (long long)js[u] * dh);
      }
      // the batch's scores side by side: TB independent dot products and
      // shuffle reductions, one maximum, then the exponentials (a chain of
      // dependent per-key updates measured 1.3 us slower per launch)
      float sc[TB];
#pragma unroll
      for (int u = 0; u < TB; ++u) sc[u] = q0 * k4[u].x + q1 * k4[u].y + q2 * k4[u].z + q3 * k4[u].w;
      for (int o = quads >> 1; o > 0; o >>= 1)
#pragma unroll
        for (int u = 0; u < TB; ++u) sc[u] += __shfl_xor(sc[u], o, 64);
      float mn = mt;
#pragma unroll
      for (int u = 0; u < TB; ++u) {
        sc[u] = ok[u] ? sc[u] * scale_log2 : -INFINITY;
        mn = fmaxf(mn, sc[u]);
      }
      const float al = exp2f(mt - mn);
      lt *= al;
      ot = make_float4(ot.x * al, ot.y * al, ot.z * al, ot.w * al);
#pragma unroll
      for (int u = 0; u < TB; ++u) {
        if (!ok[u]) break;  // uniform over the workgroup
        const float e = exp2f(sc[u] - mn);
        lt += e;
        ot = make_float4(ot.x + e * v4[u].x, ot.y + e * v4[u].y, ot.z + e * v4[u].z, ot.w + e * v4[u].w);
      }
      mt = mn;
    }
    float M = mt;
#pragma unroll
    for (int s = 0; s < MAXS; ++s) M = fmaxf(M, ms[s]);
    const float wt = exp2f(mt - M);
    float4 num = make_float4(wt * ot.x, wt * ot.y, wt * ot.z, wt * ot.w);
    float den = wt * lt;
#pragma unroll
    for (int s = 0; s < MAXS; ++s)
      if (ms[s] != -INFINITY) {
        const float w = exp2f(ms[s] - M);
        num.x += w * os[s].x; num.y += w * os[s].y; num.z += w * os[s].z; num.w += w * os[s].w;
        den += w * ls[s];
      }
    const float inv = 1.f / den;
    out = make_float4(num.x * inv, num.y * inv, num.z * inv, num.w * inv);
  }
  uint16_t* dst = o_out + xpack_off(r, h * dh + d, o_ks);
  const Hilo2 p0 = pack_hilo2(out.x, out.y), p1 = pack_hilo2(out.z, out.w);
  *reinterpret_cast<uint2*>(dst) = make_uint2(p0.hi, p1.hi);
  *reinterpret_cast<uint2*>(dst + XPACK_LO) = make_uint2(p0.lo, p1.lo);
}

hipError_t launch_attn_combine(const float* part_o, const float* part_ml, StepMeta meta, int Hq, int Hkv, int dh,
                               int slots, int sp, int qrows, int max_tree, int batch, const uint16_t* q,
                               const uint16_t* q_lo, TreeKV32 tree, PrefixKV prefix, float scale_log2,
                               uint16_t* o_out, int o_ks, hipStream_t s) {
  const int quads = dh / 4;
  if (256 % quads != 0 || slots < 1 || slots > sp) return hipErrorInvalidValue;
  const int items = Hq * quads;
  const dim3 grid(batch * max_tree, (items + 255) / 256);
  switch (slots) {
#define GRIFFIN_COMB_CASE(n)                                                                                   \
  case n:                                                                                                     \
    if (meta.split_tab)                                                                                       \
      hipLaunchKernelGGL((attn_combine_kernel<n, true>), grid, dim3(256), 0, s, part_o, part_ml, meta, Hq, Hkv,   \
                         dh, sp, qrows, max_tree, q, q_lo, tree, prefix, scale_log2, o_out, o_ks);                \
    else                                                                                                      \
      hipLaunchKernelGGL((attn_combine_kernel<n, false>), grid, dim3(256), 0, s, part_o, part_ml, meta, Hq, Hkv,  \
                         dh, sp, qrows, max_tree, q, q_lo, tree, prefix, scale_log2, o_out, o_ks);                \
    break;
    GRIFFIN_COMB_CASE(1) GRIFFIN_COMB_CASE(2) GRIFFIN_COMB_CASE(3) GRIFFIN_COMB_CASE(4) GRIFFIN_COMB_CASE(5)
    GRIFFIN_COMB_CASE(6) GRIFFIN_COMB_CASE(7) GRIFFIN_COMB_CASE(8) GRIFFIN_COMB_CASE(9) GRIFFIN_COMB_CASE(10)
    GRIFFIN_COMB_CASE(11) GRIFFIN_COMB_CASE(12) GRIFFIN_COMB_CASE(13) GRIFFIN_COMB_CASE(14) GRIFFIN_COMB_CASE(15)
    GRIFFIN_COMB_CASE(16)
#undef GRIFFIN_COMB_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace griffin
