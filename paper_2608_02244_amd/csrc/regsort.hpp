// Register bitonic sorts of one wavefront's keys (64 * KS of them, KS per
// lane), used for the priority order, the drain sweep and the event order of
// the re-scoring kernel.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wave.hpp"

namespace fs {

// Lane-major register sort of 64 * KS keys: position p = lane * KS + k, so
// the exchanges of distance below KS stay inside a lane and only the longer
// ones cross lanes.  Ascending, keys only, in the form of the bitonic network
// whose comparators all point the same way: each merge of two sorted blocks of
// size/2 first compares p with its mirror p ^ (size - 1), then half-cleans
// with p ^ d for d = size/4 .. 1; the lower position keeps the minimum.
template <int M>
__device__ __forceinline__ int shfl_mirror_c(int v) {
  // value of lane (lane ^ M), M = 2^j - 1 (every lane's source is valid, so
  // the DPP forms leave "old" undefined and fuse into their consumers)
  if constexpr (M == 1) return dpp_perm<DPP_QP_XOR1>(v);
  else if constexpr (M == 3) return dpp_perm<0x1B>(v);  // quad_perm [3,2,1,0]
  else if constexpr (M == 7) return dpp_perm<DPP_HALF_MIRROR>(v);
  else if constexpr (M == 15) return dpp_perm<DPP_MIRROR>(v);
  else if constexpr (M == 31) return __builtin_amdgcn_ds_swizzle(v, (31 << 10) | 0x1F);
  else return __shfl_xor(v, 63);
}

template <int SZ, int KS>  // mirror inside a lane's registers (block of SZ <= KS)
__device__ __forceinline__ void lm_mirror_regs(uint32_t (&key)[KS]) {
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    if ((k & (SZ >> 1)) == 0) {
      const int h = k ^ (SZ - 1);
      const uint32_t x = key[k], y = key[h];
      key[k] = min(x, y);
      key[h] = max(x, y);
    }
  }
}

template <int M, int KS>  // mirror across lanes: lane ^ M, register KS - 1 - k
__device__ __forceinline__ void lm_mirror_lanes(uint32_t (&key)[KS], int lane) {
  const bool lower = (lane & ((M + 1) >> 1)) == 0;
#pragma unroll
  for (int k = 0; k < KS / 2 + (KS & 1); ++k) {
    const int h = KS - 1 - k;
    const uint32_t a = key[k], b = key[h];
    const uint32_t pa = (uint32_t)shfl_mirror_c<M>((int)b);
    if (h != k) {
      const uint32_t pb = (uint32_t)shfl_mirror_c<M>((int)a);
      key[h] = lower ? min(b, pb) : max(b, pb);
    }
    key[k] = lower ? min(a, pa) : max(a, pa);
  }
}

template <int DK, int KS>  // half-cleaner inside a lane: registers k and k | DK
__device__ __forceinline__ void lm_half_regs(uint32_t (&key)[KS]) {
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    if ((k & DK) == 0) {
      const uint32_t x = key[k], y = key[k | DK];
      key[k] = min(x, y);
      key[k | DK] = max(x, y);
    }
  }
}

template <int D, int KS>  // half-cleaner across lanes: lane ^ D, same register
__device__ __forceinline__ void lm_half_lanes(uint32_t (&key)[KS], int lane) {
  const bool lower = (lane & D) == 0;
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    const uint32_t pk = (uint32_t)shfl_xor_c<D>((int)key[k]);
    key[k] = lower ? min(key[k], pk) : max(key[k], pk);
  }
}

// The same two lane stages, each key taking its half of the exchange with a
// median of three: with c = 0 it is min(a, b) and with c = ~0u max(a, b), c
// chosen per lane.  One instruction fewer per key, but a DPP partner then
// needs a register of its own instead of fusing into the min and the max:
// taken by the re-scoring kernel and by the simulation kernels' priority and
// drain-sweep sorts (measured faster there; the payload sorts keep the
// min / max form).
__device__ __forceinline__ uint32_t umed3(uint32_t a, uint32_t b, uint32_t c) {
  return max(min(a, b), min(max(a, b), c));
}

template <int M, int KS>
__device__ __forceinline__ void lm3_mirror_lanes(uint32_t (&key)[KS], int lane) {
  const uint32_t side = (lane & ((M + 1) >> 1)) == 0 ? 0u : ~0u;  // lower lanes keep the min
#pragma unroll
  for (int k = 0; k < KS / 2 + (KS & 1); ++k) {
    const int h = KS - 1 - k;
    const uint32_t a = key[k], b = key[h];
    const uint32_t pa = (uint32_t)shfl_mirror_c<M>((int)b);
    if (h != k) key[h] = umed3(b, (uint32_t)shfl_mirror_c<M>((int)a), side);
    key[k] = umed3(a, pa, side);
  }
}

template <int D, int KS>
__device__ __forceinline__ void lm3_half_lanes(uint32_t (&key)[KS], int lane) {
  const uint32_t side = (lane & D) == 0 ? 0u : ~0u;  // lower lanes keep the min
#pragma unroll
  for (int k = 0; k < KS; ++k) key[k] = umed3(key[k], (uint32_t)shfl_xor_c<D>((int)key[k]), side);
}

template <int M, int KS, bool MED3>
__device__ __forceinline__ void mirror_lanes(uint32_t (&key)[KS], int lane) {
  if constexpr (MED3) lm3_mirror_lanes<M>(key, lane);
  else lm_mirror_lanes<M>(key, lane);
}

template <int D, int KS, bool MED3>
__device__ __forceinline__ void half_lanes(uint32_t (&key)[KS], int lane) {
  if constexpr (MED3) lm3_half_lanes<D>(key, lane);
  else lm_half_lanes<D>(key, lane);
}

// Sort the 64 * KS keys held in registers, ascending in lane-major order.
// The stages are expanded at compile time (merge sizes 2, 4, .. 64 * KS, each
// a mirror step and half-cleaners of distance size/4 .. 1), so every stage is
// straight-line code with its exchange pattern fixed.
template <int KS, bool MED3, int D>
__device__ __forceinline__ void reg_sort_halves(uint32_t (&key)[KS], int lane) {
  if constexpr (D > 0) {
    if constexpr (D < KS) lm_half_regs<D>(key);
    else half_lanes<D / KS, KS, MED3>(key, lane);
    reg_sort_halves<KS, MED3, D / 2>(key, lane);
  }
}

template <int KS, bool MED3 = false, int SIZE = 2>
__device__ __forceinline__ void reg_sort_keys(uint32_t (&key)[KS], int lane) {
  if constexpr (SIZE <= KS * WAVE) {
    if constexpr (SIZE <= KS) lm_mirror_regs<SIZE>(key);
    else mirror_lanes<SIZE / KS - 1, KS, MED3>(key, lane);
    reg_sort_halves<KS, MED3, SIZE / 4>(key, lane);
    reg_sort_keys<KS, MED3, SIZE * 2>(key, lane);
  }
}

// The same network with one payload word per key (equal keys keep their own
// payloads, a valid outcome of an exchange).
template <int DK, int KS>
__device__ __forceinline__ void lmp_cx_regs(uint32_t (&key)[KS], int (&val)[KS], int size,
                                            int lane) {
  const bool lane_asc = ((lane * KS) & size) == 0;
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    if ((k & DK) == 0) {
      const int h = k | DK;
      const bool asc = lane_asc && (k & size) == 0;
      const uint32_t x = key[k], y = key[h];
      const int vx = val[k], vy = val[h];
      const bool sw = asc ? (x > y) : (x < y);
      key[k] = sw ? y : x;
      key[h] = sw ? x : y;
      val[k] = sw ? vy : vx;
      val[h] = sw ? vx : vy;
    }
  }
}

template <int D, int KS>
__device__ __forceinline__ void lmp_cx_lanes(uint32_t (&key)[KS], int (&val)[KS], int size,
                                             int lane) {
  const bool take_min = ((lane & D) == 0) == (((lane * KS) & size) == 0);
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    const uint32_t pk = (uint32_t)shfl_xor_c<D>((int)key[k]);
    const int pv = shfl_xor_c<D>(val[k]);
    const uint32_t nk = take_min ? min(key[k], pk) : max(key[k], pk);
    val[k] = nk == key[k] ? val[k] : pv;
    key[k] = nk;
  }
}

template <int KS, int SIZE, int D>
__device__ __forceinline__ void reg_sort_payload_stage(uint32_t (&key)[KS], int (&val)[KS],
                                                       int lane) {
  if constexpr (D > 0) {
    if constexpr (D < KS) lmp_cx_regs<D>(key, val, SIZE, lane);
    else lmp_cx_lanes<D / KS>(key, val, SIZE, lane);
    reg_sort_payload_stage<KS, SIZE, D / 2>(key, val, lane);
  }
}

// Merge sizes 2, 4, .. 64 * KS, each with exchanges of distance size/2 .. 1,
// expanded at compile time like the keys-only sort.
template <int KS, int SIZE = 2>
__device__ __forceinline__ void reg_sort_payload(uint32_t (&key)[KS], int (&val)[KS], int lane) {
  if constexpr (SIZE <= KS * WAVE) {
    reg_sort_payload_stage<KS, SIZE, SIZE / 2>(key, val, lane);
    reg_sort_payload<KS, SIZE * 2>(key, val, lane);
  }
}

// Sort W[0 .. 64*KS) ascending through registers (W is read in any order and
// written back sorted).
template <int KS, bool MED3 = false>
__device__ inline void wave_reg_sort(uint32_t* W, int lane) {
  uint32_t key[KS];
#pragma unroll
  for (int k = 0; k < KS; ++k) key[k] = W[k * WAVE + lane];
  reg_sort_keys<KS, MED3>(key, lane);
  wave_lds_sync();
#pragma unroll
  for (int k = 0; k < KS; ++k) W[lane * KS + k] = key[k];
}

}  // namespace fs
