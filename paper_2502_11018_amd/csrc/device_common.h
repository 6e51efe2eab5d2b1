// Device helpers shared by the kernels: bf16 bit conversions, vector types,
// wave-level reductions.  gfx950 only (64-wide wavefronts).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace griffin {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// fp32 -> bf16 with the hardware conversion (v_cvt_pk_bf16_f32: round to
// nearest even, NaN stays NaN).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return uint16_t(pack_bf16x2(f, 0.f)); }

// Split-bf16 operand: x ~ hi + lo with hi = bf16(x) and lo = bf16(x - hi),
// which carries about 16 significant bits through the bf16 matrix cores.
struct Hilo2 {
  uint32_t hi, lo;
};
__device__ __forceinline__ Hilo2 pack_hilo2(float a, float b) {
  const uint32_t hi = pack_bf16x2(a, b);
  return {hi, pack_bf16x2(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xffff0000u))};
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ u32x4 zero_u4() { return u32x4{0u, 0u, 0u, 0u}; }

// 16-byte loads of 8 bf16 values
__device__ __forceinline__ u32x4 ld_u4(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }

// non-temporal: data read once (streamed weights)
__device__ __forceinline__ u32x4 ld_u4_nt(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

typedef __attribute__((address_space(3))) void lds_void;

// Wait until at most N vector-memory instructions of this wave are
// outstanding and all of its LDS reads have returned (gfx9 s_waitcnt encoding:
// vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N>
__device__ __forceinline__ void wait_vmcnt_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0x0 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide sum for blockDim.x a multiple of 64 (<= 1024); every thread gets
// the total.  The combination order is fixed, so results are reproducible.
__device__ __forceinline__ float block_sum(float v, float* smem /* >= 16 floats */) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) smem[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += smem[i];
  return t;
}

__device__ __forceinline__ float silu_f32(float z) { return z / (1.0f + __expf(-z)); }

// Top-2 of (value, index) candidates, NaN-free: best with the lowest index
// among equal maxima, and the second largest value of the union counted with
// multiplicity (equal maxima at two indices give second == best).  Merging
// two such summaries gives the summary of the union, in any order.
__device__ __forceinline__ void top2_push(float& best, int& bidx, float& second, float v, int id) {
  if (v > best || (v == best && id < bidx)) {
    second = best;
    best = v;
    bidx = id;
  } else if (v > second) {
    second = v;
  }
}
__device__ __forceinline__ void top2_merge(float& best, int& bidx, float& second, float ob, int oi, float os) {
  if (ob > best || (ob == best && oi < bidx)) {
    second = fmaxf(best, os);
    best = ob;
    bidx = oi;
  } else {
    second = fmaxf(second, ob);
  }
}

// Launch timing by the kernel itself: the earliest workgroup start (stored
// complemented, so that one zero fill initialises both words and a max
// atomic takes the minimum) and the latest wave end, on the device wall
// clock.  A null pointer (the untimed case) skips both.
__device__ __forceinline__ void stamp_begin(unsigned long long* st) {
  if (st && threadIdx.x == 0) atomicMax(st, ~(unsigned long long)__builtin_amdgcn_s_memrealtime());
}
__device__ __forceinline__ void stamp_end(unsigned long long* st) {
  if (st) {
    __builtin_amdgcn_s_waitcnt(0);  // this wave's stores have completed
    if ((threadIdx.x & 63) == 0) atomicMax(st + 1, (unsigned long long)__builtin_amdgcn_s_memrealtime());
  }
}

}  // namespace griffin
