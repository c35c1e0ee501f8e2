// Output-layer weight gradient + update, as units of work that a kernel of
// its own or another kernel's workgroups run.  Unit = (worker, 64 input
// units), 4 waves (256 threads); lane owns input unit i, wave w takes rows
// j = w mod 4 (16 rows in flight per wave) and the 4 partial sums are
// added in wave order.  The bias sum over the m rows is split over up to 16
// row groups per class and added in group order.
#pragma once

#include "device_common.h"

namespace agn {
namespace {

constexpr int HDW_CHUNK = 128;  // rows of dZ staged in LDS at a time
constexpr int HDW_WAVES = 4;
template <int CMAX>
constexpr int hdw_bg() { return 64 * HDW_WAVES / CMAX < 16 ? 64 * HDW_WAVES / CMAX : 16; }  // bias row groups
// LDS of one unit (floats): staged dZ rows, the waves' partial sums, the bias partial sums
template <int CMAX>
constexpr int hdw_smem_floats() { return HDW_CHUNK * CMAX + HDW_WAVES * CMAX * 64 + hdw_bg<CMAX>() * CMAX; }
__host__ __device__ inline int hdw_units(const HeadDwArgs& a) { return a.n * ((a.d + 63) / 64); }

template <int CMAX>
__device__ __forceinline__ void head_dw_unit(const HeadDwArgs& a, int unit, float* smem) {
  constexpr int HDW_BG = hdw_bg<CMAX>();
  float* dzs = smem;
  float (*part)[CMAX][64] = reinterpret_cast<float (*)[CMAX][64]>(smem + HDW_CHUNK * CMAX);
  float (*bpart)[CMAX] = reinterpret_cast<float (*)[CMAX]>(smem + HDW_CHUNK * CMAX + HDW_WAVES * CMAX * 64);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int blocks_per_worker = (a.d + 63) / 64;
  const int k = unit / blocks_per_worker;
  const int ib = unit % blocks_per_worker;
  const int i = ib * 64 + lane;
  const int ic = i < a.d ? i : a.d - 1;
  const int C = a.C;
  const int64_t t = a.gather ? gather_step(a.g) : 0;
  const float* hb = a.h + (int64_t)k * a.hstride;
  const float* dzb = a.dz + (int64_t)k * a.dzstride;
  const int64_t wo = (int64_t)k * a.pstride;
  // operands of the epilogue first, all in flight together (indices clamped
  // into the tensors, so the loads are unconditional): this thread's weights
  // (class wave + 8s, input unit ic) and snapshot, and the bias
  constexpr int CPW = (CMAX + HDW_WAVES - 1) / HDW_WAVES;
  float wsrc[CPW], wsnap[CPW];
#pragma unroll
  for (int s = 0; s < CPW; ++s) {
    const int64_t e = wo + (int64_t)min(wave + HDW_WAVES * s, C - 1) * a.ldw + ic;
    wsrc[s] = a.w_src[e];
    wsnap[s] = a.w_snap[e];
  }
  const float bsrc = a.b_src[wo + min(tid, C - 1)], bsnap = a.b_snap[wo + min(tid, C - 1)];
  float acc[CMAX];
#pragma unroll
  for (int c = 0; c < CMAX; ++c) acc[c] = 0.f;
  // bias: thread (group, class) for tid < HDW_BG*CMAX
  const int bg = tid / CMAX, bc = tid % CMAX;
  float bsum = 0.f;
  constexpr int FIT = (HDW_CHUNK * CMAX + 64 * HDW_WAVES - 1) / (64 * HDW_WAVES);
  for (int j0 = 0; j0 < a.m; j0 += HDW_CHUNK) {
    const int rows = min(HDW_CHUNK, a.m - j0);
    // this chunk of dZ: loads first (clamped), then the LDS writes
    float dv[FIT];
#pragma unroll
    for (int s = 0; s < FIT; ++s) {
      const int e = min(tid + 64 * HDW_WAVES * s, rows * CMAX - 1);
      const int r = e / CMAX, c = min(e - r * CMAX, C - 1);
      dv[s] = dzb[(int64_t)(j0 + r) * a.lddz + c];
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < FIT; ++s) {
      const int e = tid + 64 * HDW_WAVES * s;
      if (e < rows * CMAX) dzs[e] = e % CMAX < C ? dv[s] : 0.f;
    }
    __syncthreads();
    if (ib == 0 && bg < HDW_BG)
      for (int r = bg; r < rows; r += HDW_BG) bsum += dzs[r * CMAX + bc];
    int r = wave;
    for (; r + 15 * HDW_WAVES < rows; r += 16 * HDW_WAVES) {   // 16 rows per wave in flight
      float hv[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int j = j0 + r + HDW_WAVES * u;
        const int64_t row = a.gather ? batch_row(k, t, a.g.mb, a.g.S, j) : j;
        hv[u] = hb[row * a.ldh + ic];
      }
#pragma unroll
      for (int u = 0; u < 16; ++u)
#pragma unroll
        for (int c = 0; c < CMAX; ++c) acc[c] += dzs[(r + HDW_WAVES * u) * CMAX + c] * hv[u];
    }
    for (; r < rows; r += HDW_WAVES) {
      const int j = j0 + r;
      const int64_t row = a.gather ? batch_row(k, t, a.g.mb, a.g.S, j) : j;
      const float hv = hb[row * a.ldh + ic];
#pragma unroll
      for (int c = 0; c < CMAX; ++c) acc[c] += dzs[r * CMAX + c] * hv;
    }
  }
#pragma unroll
  for (int c = 0; c < CMAX; ++c) part[wave][c][lane] = acc[c];
  if (ib == 0 && bg < HDW_BG) bpart[bg][bc] = bsum;
  __syncthreads();
  // the prefetched operands are in registers by now: use them here, in
  // straight-line code, so that no wait for them lands between the stores
#pragma unroll
  for (int s = 0; s < CPW; ++s) asm volatile("" ::"v"(wsrc[s]), "v"(wsnap[s]));
  asm volatile("" ::"v"(bsrc), "v"(bsnap));
  const AdamCoef ac = a.adam.on ? adam_coef(a.g, a.adam) : AdamCoef{1.f, 1.f};
#pragma unroll
  for (int s = 0; s < CPW; ++s) {
    const int c = wave + HDW_WAVES * s;
    if (c >= C) break;
    float g = part[0][c][lane];
#pragma unroll
    for (int w = 1; w < HDW_WAVES; ++w) g += part[w][c][lane];
    if (i < a.d) {
      const int64_t e = wo + (int64_t)c * a.ldw + i;
      const float step = a.adam.on ? adam_dir(g, a.adam.mw, a.adam.vw, e, a.adam, ac) : g;
      const float nw = wsrc[s] - a.eta * step;
      a.w_dst[e] = a.last ? (nw - wsnap[s]) / a.lam : nw;
    }
  }
  if (ib == 0 && tid < C) {
    float gb = bpart[0][tid];
#pragma unroll
    for (int q = 1; q < HDW_BG; ++q) gb += bpart[q][tid];
    const int64_t e = wo + tid;
    const float step = a.adam.on ? adam_dir(gb, a.adam.mb, a.adam.vb, e, a.adam, ac) : gb;
    const float nb = bsrc - a.eta * step;
    a.b_dst[e] = a.last ? (nb - bsnap) / a.lam : nb;
  }
}


}  // namespace
}  // namespace agn
