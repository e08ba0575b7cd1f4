// Wavefront (64-lane) primitives for gfx950: DPP reductions and scans,
// ballot helpers and LDS ordering within one wave.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fs {

constexpr int WAVE = 64;

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

// Predicates of ballots are built with & rather than && when no operand reads
// memory: the short-circuit form is compiled to lane-masked branches.
__device__ __forceinline__ uint64_t ballot(bool p) { return (uint64_t)__ballot(p); }

// Number of set bits of `mask` below the calling lane.
__device__ __forceinline__ int mbcnt(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ int readlane(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint32_t uniu(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}
__device__ __forceinline__ int64_t uni64(int64_t v) {
  uint32_t lo = uniu((uint32_t)v), hi = uniu((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ int first_lane(uint64_t m) { return m ? __builtin_ctzll(m) : -1; }

// DPP move with a compile-time control word.
template <int CTRL, int ROW_MASK = 0xf, int BANK_MASK = 0xf, bool BOUND = false>
__device__ __forceinline__ int dpp(int old, int src) {
  return __builtin_amdgcn_update_dpp(old, src, CTRL, ROW_MASK, BANK_MASK, BOUND);
}

// DPP permutation of v in which every lane's source lane is valid (quad
// permutes, mirrors, row rotates): no "old" value is needed, so the move can
// fuse into the instructions that consume it.
template <int CTRL>
__device__ __forceinline__ int dpp_perm(int v) {
  return __builtin_amdgcn_mov_dpp(v, CTRL, 0xf, 0xf, true);
}

// quad_perm [1,0,3,2], [2,3,0,1]; row_half_mirror; row_mirror; row_bcast15; row_bcast31
enum : int {
  DPP_QP_XOR1 = 0xB1,
  DPP_QP_XOR2 = 0x4E,
  DPP_HALF_MIRROR = 0x141,
  DPP_MIRROR = 0x140,
  DPP_BCAST15 = 0x142,
  DPP_BCAST31 = 0x143,
  DPP_ROW_SHR1 = 0x111,
  DPP_ROW_SHR2 = 0x112,
  DPP_ROW_SHR3 = 0x113,
  DPP_ROW_SHR4 = 0x114,
  DPP_ROW_SHR8 = 0x118,
  DPP_WAVE_SHL1 = 0x130,  // lane i reads lane i + 1 (lane 63 keeps the old value)
};

// Reductions: after the butterfly inside each row of 16 every lane holds its
// row's value; the two broadcasts fold rows 0..3 into lanes 48..63.  The DPP
// moves take the operation's identity as their "old" value (every lane read
// here has a valid source, and rows outside a broadcast's row mask are not
// written), which lets the compiler fuse each move into the min / max itself.
__device__ __forceinline__ int wave_min(int v) {
  constexpr int ID = 0x7FFFFFFF;
  v = min(v, dpp<DPP_QP_XOR1>(ID, v));
  v = min(v, dpp<DPP_QP_XOR2>(ID, v));
  v = min(v, dpp<DPP_HALF_MIRROR>(ID, v));
  v = min(v, dpp<DPP_MIRROR>(ID, v));
  v = min(v, dpp<DPP_BCAST15, 0xa>(ID, v));
  v = min(v, dpp<DPP_BCAST31, 0xc>(ID, v));
  return readlane(v, 63);
}

__device__ __forceinline__ int wave_max(int v) {
  constexpr int ID = (int)0x80000000;
  v = max(v, dpp<DPP_QP_XOR1>(ID, v));
  v = max(v, dpp<DPP_QP_XOR2>(ID, v));
  v = max(v, dpp<DPP_HALF_MIRROR>(ID, v));
  v = max(v, dpp<DPP_MIRROR>(ID, v));
  v = max(v, dpp<DPP_BCAST15, 0xa>(ID, v));
  v = max(v, dpp<DPP_BCAST31, 0xc>(ID, v));
  return readlane(v, 63);
}

__device__ __forceinline__ uint32_t wave_umin(uint32_t v) {
  constexpr int ID = (int)0xFFFFFFFFu;
  int x = (int)v;
  x = (int)min((uint32_t)x, (uint32_t)dpp<DPP_QP_XOR1>(ID, x));
  x = (int)min((uint32_t)x, (uint32_t)dpp<DPP_QP_XOR2>(ID, x));
  x = (int)min((uint32_t)x, (uint32_t)dpp<DPP_HALF_MIRROR>(ID, x));
  x = (int)min((uint32_t)x, (uint32_t)dpp<DPP_MIRROR>(ID, x));
  x = (int)min((uint32_t)x, (uint32_t)dpp<DPP_BCAST15, 0xa>(ID, x));
  x = (int)min((uint32_t)x, (uint32_t)dpp<DPP_BCAST31, 0xc>(ID, x));
  return (uint32_t)readlane(x, 63);
}

// Sum of int32 values (the caller guarantees the total fits).
__device__ __forceinline__ int wave_sum(int v) {
  v += dpp<DPP_QP_XOR1>(0, v);
  v += dpp<DPP_QP_XOR2>(0, v);
  v += dpp<DPP_HALF_MIRROR>(0, v);
  v += dpp<DPP_MIRROR>(0, v);
  v += dpp<DPP_BCAST15, 0xa>(0, v);
  v += dpp<DPP_BCAST31, 0xc>(0, v);
  return readlane(v, 63);
}

// Inclusive prefix sum over lanes 0..63.
__device__ __forceinline__ int wave_scan_incl(int x) {
  int v = x;
  v += dpp<DPP_ROW_SHR1, 0xf, 0xf, true>(0, x);
  v += dpp<DPP_ROW_SHR2, 0xf, 0xf, true>(0, x);
  v += dpp<DPP_ROW_SHR3, 0xf, 0xf, true>(0, x);
  v += dpp<DPP_ROW_SHR4, 0xf, 0xe, false>(0, v);
  v += dpp<DPP_ROW_SHR8, 0xf, 0xc, false>(0, v);
  v += dpp<DPP_BCAST15, 0xa, 0xf, false>(0, v);
  v += dpp<DPP_BCAST31, 0xc, 0xf, false>(0, v);
  return v;
}

// Inclusive prefix max over lanes 0..63 (identity INT_MIN).
__device__ __forceinline__ int wave_scan_incl_max(int x) {
  constexpr int ID = (int)0x80000000;
  int v = x;
  v = max(v, dpp<DPP_ROW_SHR1, 0xf, 0xf, false>(ID, x));
  v = max(v, dpp<DPP_ROW_SHR2, 0xf, 0xf, false>(ID, x));
  v = max(v, dpp<DPP_ROW_SHR3, 0xf, 0xf, false>(ID, x));
  v = max(v, dpp<DPP_ROW_SHR4, 0xf, 0xe, false>(ID, v));
  v = max(v, dpp<DPP_ROW_SHR8, 0xf, 0xc, false>(ID, v));
  v = max(v, dpp<DPP_BCAST15, 0xa, 0xf, false>(ID, v));
  v = max(v, dpp<DPP_BCAST31, 0xc, 0xf, false>(ID, v));
  return v;
}

// Inclusive prefix min over lanes 0..63 (identity INT_MAX).
__device__ __forceinline__ int wave_scan_incl_min(int x) {
  constexpr int ID = 0x7FFFFFFF;
  int v = x;
  v = min(v, dpp<DPP_ROW_SHR1, 0xf, 0xf, false>(ID, x));
  v = min(v, dpp<DPP_ROW_SHR2, 0xf, 0xf, false>(ID, x));
  v = min(v, dpp<DPP_ROW_SHR3, 0xf, 0xf, false>(ID, x));
  v = min(v, dpp<DPP_ROW_SHR4, 0xf, 0xe, false>(ID, v));
  v = min(v, dpp<DPP_ROW_SHR8, 0xf, 0xc, false>(ID, v));
  v = min(v, dpp<DPP_BCAST15, 0xa, 0xf, false>(ID, v));
  v = min(v, dpp<DPP_BCAST31, 0xc, 0xf, false>(ID, v));
  return v;
}

// Value of lane (lane ^ D), D a power of two below 64: DPP for 1, 2 (quad
// permutes) and 8 (rotate a row of 16 by 8), swizzle in bit mode for 4 and 16
// (xor mask within 32 lanes), a permute through the LDS crossbar for 32.
template <int D>
__device__ __forceinline__ int shfl_xor_c(int v) {
  static_assert(D > 0 && D < WAVE && (D & (D - 1)) == 0, "xor distance");
  if constexpr (D == 1) return dpp_perm<DPP_QP_XOR1>(v);
  else if constexpr (D == 2) return dpp_perm<DPP_QP_XOR2>(v);
  else if constexpr (D == 8) return dpp_perm<0x128>(v);  // row_ror:8
  else if constexpr (D == 4 || D == 16) return __builtin_amdgcn_ds_swizzle(v, (D << 10) | 0x1F);
  else return __shfl_xor(v, D);
}

// DPP move of a 64-bit value (both halves with the same control word).
template <int CTRL, int ROW_MASK = 0xf, int BANK_MASK = 0xf, bool BOUND = false>
__device__ __forceinline__ uint64_t dpp64(uint64_t old, uint64_t src) {
  const uint32_t lo =
      (uint32_t)dpp<CTRL, ROW_MASK, BANK_MASK, BOUND>((int)(uint32_t)old, (int)(uint32_t)src);
  const uint32_t hi = (uint32_t)dpp<CTRL, ROW_MASK, BANK_MASK, BOUND>(
      (int)(uint32_t)(old >> 32), (int)(uint32_t)(src >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Inclusive prefix sum of 64-bit values over lanes 0..63 (same DPP pattern as
// the 32-bit scan).
__device__ __forceinline__ int64_t wave_scan_incl64(int64_t x) {
  const uint64_t s = (uint64_t)x;
  uint64_t v = s;
  v += dpp64<DPP_ROW_SHR1, 0xf, 0xf, true>(0, s);
  v += dpp64<DPP_ROW_SHR2, 0xf, 0xf, true>(0, s);
  v += dpp64<DPP_ROW_SHR3, 0xf, 0xf, true>(0, s);
  v += dpp64<DPP_ROW_SHR4, 0xf, 0xe>(0, v);
  v += dpp64<DPP_ROW_SHR8, 0xf, 0xc>(0, v);
  v += dpp64<DPP_BCAST15, 0xa, 0xf>(0, v);
  v += dpp64<DPP_BCAST31, 0xc, 0xf>(0, v);
  return (int64_t)v;
}

__device__ __forceinline__ int64_t readlane64(int64_t v, int l) {
  const uint32_t lo = (uint32_t)readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)readlane((int)(uint32_t)((uint64_t)v >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// 64-bit max and sum, same DPP pattern as the 32-bit reductions.
__device__ __forceinline__ int64_t wave_max64(int64_t v) {
  uint64_t x = (uint64_t)v;
  auto mx = [](uint64_t a, uint64_t b) { return (int64_t)a > (int64_t)b ? a : b; };
  x = mx(x, dpp64<DPP_QP_XOR1>(x, x));
  x = mx(x, dpp64<DPP_QP_XOR2>(x, x));
  x = mx(x, dpp64<DPP_HALF_MIRROR>(x, x));
  x = mx(x, dpp64<DPP_MIRROR>(x, x));
  x = mx(x, dpp64<DPP_BCAST15, 0xa>(x, x));
  x = mx(x, dpp64<DPP_BCAST31, 0xc>(x, x));
  return readlane64((int64_t)x, 63);
}

__device__ __forceinline__ int64_t wave_sum64(int64_t v) {
  uint64_t x = (uint64_t)v;
  x += dpp64<DPP_QP_XOR1>(0, x);
  x += dpp64<DPP_QP_XOR2>(0, x);
  x += dpp64<DPP_HALF_MIRROR>(0, x);
  x += dpp64<DPP_MIRROR>(0, x);
  x += dpp64<DPP_BCAST15, 0xa>(0, x);
  x += dpp64<DPP_BCAST31, 0xc>(0, x);
  return readlane64((int64_t)x, 63);
}

// Order LDS accesses of this wave: all lanes of a wave issue LDS operations in
// program order; this keeps the compiler from moving memory operations across
// a cross-lane hand-off and waits for outstanding LDS traffic.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

}  // namespace fs
