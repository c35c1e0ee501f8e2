// Device helpers shared by the kernels of libagn.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "agn_internal.h"

namespace agn {

constexpr int kNumXcd = 8;  // MI355X: 8 XCDs, workgroups dispatched round-robin

// Workgroups are handed to the XCDs round-robin (workgroup i to XCD i % 8).
// Map the hardware id to a logical tile id so that each XCD receives one
// contiguous range of logical tiles: tiles that share operands (one worker's
// weights, one row block) then share that XCD's L2.  A bijection on [0, nblk).
__device__ __forceinline__ int xcd_remap(int pid, int nblk) {
  const int xcd = pid % kNumXcd, local = pid / kNumXcd;
  const int q = nblk / kNumXcd, rem = nblk % kNumXcd;
  return xcd < rem ? xcd * (q + 1) + local : rem * (q + 1) + (xcd - rem) * q + local;
}

// A data-parallel (DPP) move within each row of 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float lane_value(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

// Reduction over the wave with a commutative op (every lane active): within
// each row of 16 lanes by DPP moves (quad pairs 1<->0, 3<->2, then 2<->0,
// 3<->1; then the two quads of each half row, i <-> 7-i; then the two
// halves, i <-> 15-i), then the four row results in row order.  The same
// value in every lane and on every call.
template <typename Op>
__device__ __forceinline__ float wave_reduce(float v, Op op) {
  v = op(v, dpp_move<0xB1>(v));   // quad_perm(1, 0, 3, 2)
  v = op(v, dpp_move<0x4E>(v));   // quad_perm(2, 3, 0, 1)
  v = op(v, dpp_move<0x141>(v));  // row_half_mirror
  v = op(v, dpp_move<0x140>(v));  // row_mirror
  return op(op(op(lane_value(v, 0), lane_value(v, 16)), lane_value(v, 32)), lane_value(v, 48));
}
__device__ __forceinline__ float wave_sum(float v) {
  return wave_reduce(v, [](float a, float b) { return a + b; });
}
__device__ __forceinline__ float wave_max(float v) {
  return wave_reduce(v, [](float a, float b) { return fmaxf(a, b); });
}

// Data-set row of row j of worker k's mini-batch at local step t.
__device__ __forceinline__ int64_t batch_row(int64_t k, int64_t t, int64_t mb, int64_t S, int64_t j) {
  return k * S + (t * mb + j) % S;
}

__device__ __forceinline__ int64_t gather_step(const Gather& g) {
  return (*g.round) * (int64_t)g.lam + g.step;
}

// Adam (Kingma & Ba 2015) bias corrections 1/(1 - beta^t) at the worker's
// local step t = round*lambda + step + 1 (the round counter lives on the
// device, so a recorded round stays valid in every replay).
struct AdamCoef {
  float c1, c2;
};
__device__ __forceinline__ AdamCoef adam_coef(const Gather& g, const AdamArgs& a) {
  const double t = (double)(*g.round) * g.lam + g.step + 1;
  return {(float)(1.0 / (1.0 - pow((double)a.beta1, t))), (float)(1.0 / (1.0 - pow((double)a.beta2, t)))};
}
// One Adam moment update of gradient g (m and v in place); returns the step
// direction mhat / (sqrt(vhat) + eps), to be scaled by -eta.
__device__ __forceinline__ float adam_moments(float g, float& m, float& v, const AdamArgs& a, const AdamCoef& c) {
  m = a.beta1 * m + (1.f - a.beta1) * g;
  v = a.beta2 * v + (1.f - a.beta2) * g * g;
  return (m * c.c1) / (sqrtf(v * c.c2) + a.eps);
}
// the same for element e of the moment arrays m and v
__device__ __forceinline__ float adam_dir(float g, float* m, float* v, int64_t e, const AdamArgs& a,
                                          const AdamCoef& c) {
  float m1 = m[e], v1 = v[e];
  const float d = adam_moments(g, m1, v1, a, c);
  m[e] = m1;
  v[e] = v1;
  return d;
}

// float32 -> bfloat16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

}  // namespace agn
