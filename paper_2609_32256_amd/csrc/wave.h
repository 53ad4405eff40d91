// Wave-wide reductions by data-parallel primitive moves (DPP): lane moves that
// stay in the register file, where a butterfly of __shfl_xor steps goes
// through LDS and waits for each step.  The moves, on a 64-lane wave: swaps
// within quads (neighbours, then pairs), across the quads of each half row of
// 8 (row_half_mirror), across the halves of each row of 16 (row_mirror), then
// lane 15 of rows 0 and 2 into rows 1 and 3 (row_bcast:15), and lane 31 into
// rows 2 and 3 (row_bcast:31).  Each step combines disjoint partial results,
// so after it lane 63 holds the whole wave's; a lane that a move does not
// write gets the operation's identity.  Every lane of the wave must be active.
// Sums in binary64 are taken in this fixed order (different from a butterfly's,
// equally exact to within the usual bound for n terms).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace lam {

#define LAM_WAVE_DPP_STEPS(STEP) \
  STEP(0xb1, 0xf)                \
  STEP(0x4e, 0xf)                \
  STEP(0x141, 0xf)               \
  STEP(0x140, 0xf)               \
  STEP(0x142, 0xa)               \
  STEP(0x143, 0xc)

// move of a 32-bit lane value; `old` for lanes the move does not write
#define LAM_DPP_MOVE(old, v, ctrl, rmask) __builtin_amdgcn_update_dpp((int)(old), (int)(v), ctrl, rmask, 0xf, false)

__device__ __forceinline__ float wave_max_f32(float v) {
#define LAM_STEP(ctrl, rmask) v = fmaxf(v, __int_as_float(LAM_DPP_MOVE(__float_as_int(v), __float_as_int(v), ctrl, rmask)));
  LAM_WAVE_DPP_STEPS(LAM_STEP)
#undef LAM_STEP
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#define LAM_STEP(ctrl, rmask) v = max(v, (uint32_t)LAM_DPP_MOVE(v, v, ctrl, rmask));
  LAM_WAVE_DPP_STEPS(LAM_STEP)
#undef LAM_STEP
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

__device__ __forceinline__ unsigned long long wave_max_u64(unsigned long long key) {
  uint32_t lo = (uint32_t)key, hi = (uint32_t)(key >> 32);
#define LAM_STEP(ctrl, rmask)                                                          \
  {                                                                                    \
    const uint32_t olo = (uint32_t)LAM_DPP_MOVE(lo, lo, ctrl, rmask);                  \
    const uint32_t ohi = (uint32_t)LAM_DPP_MOVE(hi, hi, ctrl, rmask);                  \
    const bool gt = ohi > hi || (ohi == hi && olo > lo);                               \
    lo = gt ? olo : lo;                                                                \
    hi = gt ? ohi : hi;                                                                \
  }
  LAM_WAVE_DPP_STEPS(LAM_STEP)
#undef LAM_STEP
  const uint32_t rlo = (uint32_t)__builtin_amdgcn_readlane((int)lo, 63);
  const uint32_t rhi = (uint32_t)__builtin_amdgcn_readlane((int)hi, 63);
  return ((unsigned long long)rhi << 32) | rlo;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#define LAM_STEP(ctrl, rmask)                                                                     \
  {                                                                                               \
    const unsigned long long b = (unsigned long long)__double_as_longlong(v);                    \
    const uint32_t olo = (uint32_t)LAM_DPP_MOVE(0, (uint32_t)b, ctrl, rmask);                     \
    const uint32_t ohi = (uint32_t)LAM_DPP_MOVE(0, (uint32_t)(b >> 32), ctrl, rmask);             \
    v += __longlong_as_double((long long)(((unsigned long long)ohi << 32) | olo));                \
  }
  LAM_WAVE_DPP_STEPS(LAM_STEP)
#undef LAM_STEP
  const unsigned long long b = (unsigned long long)__double_as_longlong(v);
  const uint32_t rlo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, 63);
  const uint32_t rhi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), 63);
  return __longlong_as_double((long long)(((unsigned long long)rhi << 32) | rlo));
}

#undef LAM_DPP_MOVE
#undef LAM_WAVE_DPP_STEPS

}  // namespace lam
