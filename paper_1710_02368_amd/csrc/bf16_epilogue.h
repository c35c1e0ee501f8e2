// Epilogues of the bf16 products (128 x 128 output tiles of 256 threads,
// four waves of 64 x 64, each as 2 x 2 blocks of v_mfma_f32_32x32x16_bf16),
// shared by the register-staged and the direct-load kernels.  Block (bi, bj)
// of wave (wm, wn) holds in accumulator register r of lane (li, lh) the
// output at tile row wm*64 + 32*bi + 8*(r/4) + 4*lh + r%4 and tile column
// wn*64 + 32*bj + li.
#pragma once

#include "device_common.h"

namespace agn {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float epi_f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t epi_u32x2 __attribute__((ext_vector_type(2)));

constexpr int TB = 128;          // tile edge (M and N)
constexpr int NT = 256;          // threads per workgroup
constexpr int EPI_LD = TB + 4;   // LDS row stride (floats) of the epilogue accumulator tile
constexpr int EPI_BYTES = TB * EPI_LD * 4;

// Weight-gradient epilogue through LDS: the float32 accumulator tile is
// written to LDS, then every thread streams 16-byte chunks of rows (W_src
// read, W_dst and its bf16 shadow written), so the master-weight traffic is
// coalesced.  Needs 16-byte rows.  The master weights (and snapshot) come
// in and the updated weights and their bf16 shadow go out as streaming
// (non-temporal) accesses: each is touched once per local step, at the
// wide workload 14 B per parameter of 200M-parameter layers, far beyond the
// caches, where cached accesses only evicted the operands the products
// share.
__host__ __device__ inline bool dw_vec_ok(const GemmArgs& g) {
  const uintptr_t p = (uintptr_t)g.w_src | (uintptr_t)g.w_dst | (g.last ? (uintptr_t)g.w_snap : 0);
  return (p & 15) == 0 && ((uintptr_t)g.w_dst16 & 7) == 0 && g.ldw % 4 == 0 && g.pstride % 4 == 0 && g.N % 4 == 0;
}

template <bool LAST>
__device__ __forceinline__ void dw_epilogue_lds(const GemmArgs& g, int worker, int m0, int n0, const f32x16 (&acc)[2][2],
                                                float* et, const AdamCoef& ac) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, li = lane & 31, lh = lane >> 5;
  const int64_t wo = (int64_t)worker * g.pstride;
  constexpr int CH = TB * TB / 4 / NT;  // 16-byte chunks per thread: chunk c = tid + NT*u
  // the weight (and, on the last step, snapshot) loads of a pass first,
  // all in flight together: unconditional, from indices clamped into the
  // matrix (N a multiple of 4); values outside it are never stored.  One
  // pass over the tile's 16 chunks per thread, two on the last step (the
  // snapshot doubles the registers).  (Loads issued after a store wait for
  // that store too: one counter for both.)
  constexpr int NP = LAST ? 2 : 1, PER = CH / NP;
  float4 w[PER], sn[LAST ? PER : 1];
#pragma unroll
  for (int pass = 0; pass < NP; ++pass) {
#pragma unroll
    for (int v = 0; v < PER; ++v) {
      const int c = tid + NT * (pass * PER + v), row = c / (TB / 4), col = 4 * (c % (TB / 4));
      const int64_t el = wo + (int64_t)min(m0 + row, g.M - 1) * g.ldw + min(n0 + col, g.N - 4);
      const epi_f32x4 t = __builtin_nontemporal_load(reinterpret_cast<const epi_f32x4*>(g.w_src + el));
      w[v] = make_float4(t.x, t.y, t.z, t.w);
      if (LAST) {
        const epi_f32x4 u = __builtin_nontemporal_load(reinterpret_cast<const epi_f32x4*>(g.w_snap + el));
        sn[v] = make_float4(u.x, u.y, u.z, u.w);
      }
    }
    if (pass == 0) {
      // the accumulator tile to LDS while they are in flight
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            et[(wm * 64 + 32 * bi + 8 * (r >> 2) + 4 * lh + (r & 3)) * EPI_LD + wn * 64 + 32 * bj + li] = acc[bi][bj][r];
      __syncthreads();
    }
#pragma unroll
    for (int v = 0; v < PER; ++v) {
      asm volatile("" ::"v"(w[v].x), "v"(w[v].w));
      if (LAST) asm volatile("" ::"v"(sn[v].x), "v"(sn[v].w));
    }
#pragma unroll
    for (int v = 0; v < PER; ++v) {
      const int c = tid + NT * (pass * PER + v), row = c / (TB / 4), col = 4 * (c % (TB / 4));
      float4 a = *reinterpret_cast<const float4*>(et + row * EPI_LD + col);
      if (m0 + row >= g.M || n0 + col >= g.N) continue;
      const int64_t e = wo + (int64_t)(m0 + row) * g.ldw + n0 + col;
      if (g.adam.on) {
        a.x = adam_dir(a.x, g.adam.mw, g.adam.vw, e, g.adam, ac);
        a.y = adam_dir(a.y, g.adam.mw, g.adam.vw, e + 1, g.adam, ac);
        a.z = adam_dir(a.z, g.adam.mw, g.adam.vw, e + 2, g.adam, ac);
        a.w = adam_dir(a.w, g.adam.mw, g.adam.vw, e + 3, g.adam, ac);
      }
      float4 nw = make_float4(w[v].x - g.eta * a.x, w[v].y - g.eta * a.y, w[v].z - g.eta * a.z,
                              w[v].w - g.eta * a.w);
      if (LAST) {
        nw = make_float4((nw.x - sn[v].x) / g.lam, (nw.y - sn[v].y) / g.lam, (nw.z - sn[v].z) / g.lam,
                         (nw.w - sn[v].w) / g.lam);
        const epi_f32x4 dv = {nw.x, nw.y, nw.z, nw.w};
        __builtin_nontemporal_store(dv, reinterpret_cast<epi_f32x4*>(g.w_dst + e));
      } else {
        const epi_f32x4 nv = {nw.x, nw.y, nw.z, nw.w};
        __builtin_nontemporal_store(nv, reinterpret_cast<epi_f32x4*>(g.w_dst + e));
        const epi_u32x2 h = {f32_to_bf16_rne(nw.x) | ((uint32_t)f32_to_bf16_rne(nw.y) << 16),
                             f32_to_bf16_rne(nw.z) | ((uint32_t)f32_to_bf16_rne(nw.w) << 16)};
        __builtin_nontemporal_store(h, reinterpret_cast<epi_u32x2*>(g.w_dst16 + e));
      }
    }
  }
}

// Epilogue of the forward and input-gradient products through LDS: the
// float32 accumulator tile goes to LDS, then each thread takes row chunks of
// the output (8 bf16 or 4 float32 columns) with their operands (bias, ReLU
// mask) loaded up front from indices clamped into the matrix, and stores
// each chunk with one 16-byte store (element by element only where a chunk
// crosses the matrix edge, so padding columns are never written).
template <int EPI>
__device__ __forceinline__ void out_epilogue_lds(const GemmArgs& g, int worker, int m0, int n0,
                                                 const f32x16 (&acc)[2][2], float* et) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, li = lane & 31, lh = lane >> 5;
  constexpr bool F32 = EPI == EPI_FWD_LINEAR;
  constexpr int CW = F32 ? 4 : 8;            // columns per chunk
  constexpr int CPR = TB / CW;               // chunks per row
  constexpr int NC = TB * CPR / NT;          // chunks per thread
  const int colc = (tid % CPR) * CW;         // this thread's chunk column (the same for all its chunks)
  const int cbase = n0 + colc;
  // bias of the chunk's columns (forward)
  float bv[CW];
  if (EPI == EPI_FWD_RELU || EPI == EPI_FWD_LINEAR) {
#pragma unroll
    for (int j = 0; j < CW; ++j) bv[j] = g.bias[(int64_t)worker * g.bstride + min(cbase + j, g.N - 1)];
  }
  // mask rows of the chunks (input gradient): 8 bf16 at a clamped chunk start
  uint4 mv[NC];
  if (EPI == EPI_DX_MASK) {
    const int cm = min(cbase, (g.N - 1) / 8 * 8);  // (rows of the mask are padded to 8)
#pragma unroll
    for (int u = 0; u < NC; ++u) {
      const int row = min(m0 + (tid + NT * u) / CPR, g.M - 1);
      mv[u] = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(g.mask) +
                                              (int64_t)worker * g.mstride + (int64_t)row * g.ldm + cm);
    }
  }
  // the accumulator tile to LDS while those loads are in flight
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        et[(wm * 64 + 32 * bi + 8 * (r >> 2) + 4 * lh + (r & 3)) * EPI_LD + wn * 64 + 32 * bj + li] = acc[bi][bj][r];
  __syncthreads();
  if (EPI == EPI_FWD_RELU || EPI == EPI_FWD_LINEAR) {
#pragma unroll
    for (int j = 0; j < CW; j += 2) asm volatile("" ::"v"(bv[j]), "v"(bv[j + 1]));
  }
  if (EPI == EPI_DX_MASK) {
#pragma unroll
    for (int u = 0; u < NC; ++u) asm volatile("" ::"v"(mv[u].x), "v"(mv[u].w));
  }
  if (cbase >= g.N) return;
  const bool whole = cbase + CW <= g.N;
#pragma unroll
  for (int u = 0; u < NC; ++u) {
    const int rl = (tid + NT * u) / CPR, row = m0 + rl;
    if (row >= g.M) continue;
    float v[CW];
#pragma unroll
    for (int j = 0; j < CW; j += 4) {
      const float4 a = *reinterpret_cast<const float4*>(et + rl * EPI_LD + colc + j);
      v[j] = a.x;
      v[j + 1] = a.y;
      v[j + 2] = a.z;
      v[j + 3] = a.w;
    }
    const int64_t o = (int64_t)worker * g.ostride + (int64_t)row * g.ldo + cbase;
    if (F32) {
      float* out = reinterpret_cast<float*>(g.out) + o;
#pragma unroll
      for (int j = 0; j < CW; ++j) v[j] += bv[j];
      if (whole) {
        *reinterpret_cast<float4*>(out) = make_float4(v[0], v[1], v[2], v[3]);
      } else {
        for (int j = 0; j < CW && cbase + j < g.N; ++j) out[j] = v[j];
      }
    } else {
      uint16_t hv[CW];
      if (EPI == EPI_FWD_RELU) {
#pragma unroll
        for (int j = 0; j < CW; ++j) {
          const float h = v[j] + bv[j];
          hv[j] = f32_to_bf16_rne(h > 0.f ? h : 0.f);
        }
      } else {  // EPI_DX_MASK
        const uint32_t mw[4] = {mv[u].x, mv[u].y, mv[u].z, mv[u].w};
#pragma unroll
        for (int j = 0; j < CW; ++j) {
          const uint16_t m = (uint16_t)(mw[j / 2] >> (16 * (j % 2)));
          hv[j] = f32_to_bf16_rne(bf16_to_f32(m) > 0.f ? v[j] : 0.f);
        }
      }
      uint16_t* out = reinterpret_cast<uint16_t*>(g.out) + o;
      if (whole) {
        uint4 pk;
        pk.x = (uint32_t)hv[0] | ((uint32_t)hv[1] << 16);
        pk.y = (uint32_t)hv[2] | ((uint32_t)hv[3] << 16);
        pk.z = (uint32_t)hv[4] | ((uint32_t)hv[5] << 16);
        pk.w = (uint32_t)hv[6] | ((uint32_t)hv[7] << 16);
        *reinterpret_cast<uint4*>(out) = pk;
      } else {
        for (int j = 0; j < CW && cbase + j < g.N; ++j) out[j] = hv[j];
      }
    }
  }
}

// the output can take 16-byte chunk stores (and the mask 16-byte loads)
__host__ __device__ inline bool out_vec_ok(const GemmArgs& g) {
  const bool f32 = g.epi == EPI_FWD_LINEAR;
  const int cw = f32 ? 4 : 8;
  bool ok = ((uintptr_t)g.out & 15) == 0 && g.ldo % cw == 0 && g.ostride % cw == 0;
  if (g.epi == EPI_DX_MASK)
    ok = ok && ((uintptr_t)g.mask & 15) == 0 && g.ldm % 8 == 0 && g.mstride % 8 == 0 && g.ldm >= (g.N + 7) / 8 * 8;
  return ok;
}

}  // namespace
}  // namespace agn
