// Backward launch of a hidden layer l >= 1 (float32) as column strips of the
// layer's weights: the input-gradient product dZ_l = (dZ_{l+1} W_l) * [H_l > 0]
// and the weight-gradient product dW_l = dZ_{l+1}^T H_l fused with the SGD
// update of W_l and b_l (Algorithm 1, gradient line and local step).
//
// Both products read the same weights: the input gradient contracts W_l over
// its rows (the layer's outputs i), the update rewrites it.  A workgroup owns
// one worker and one strip of 64 columns j of W_l (64 inputs of the layer):
// it holds H_l[:, strip] in LDS for the whole launch and walks the blocks of
// 64 rows i.  Per block, dZ_{l+1}[:, block] and W_l[block, strip] travel into
// LDS once (direct global->LDS loads, double-buffered) and feed both the
// input gradient's 128 x 64 accumulator of the strip (K = the block's 64
// rows i; masked by H_l from LDS at the end) and the block's 64 x 64 weight
// gradient (K = the mini-batch) with its epilogue W_dst = W_src - eta * dW,
// W_src from the same LDS tile (a round's last step stores (W_dst - W_snap)
// / lambda instead).  So the weights are read from memory once and written
// once per local step.  Eight waves, two per SIMD, each with a share of both
// products (see below).
//
// MFMA v_mfma_f32_16x16x4f32: lane l supplies A[l%16][k] and B[k][l%16] for
// k = its lane group's k, and holds D[4*(l/16) + r][l%16] in register r.
//
// LDS tiles hold 64 floats of each row followed by padding; the padded row
// lengths make every LDS read of the inner loops a per-lane base address
// plus a constant offset, free of bank conflicts:
//   * dZ block, 128 x 64, rows of 68 floats: a column read over 16
//     consecutive rows touches 16 distinct 16-byte bank groups, and a row
//     read by four lane groups at rows 4 apart touches 64 distinct banks;
//   * H strip, 128 x 64, rows of 72 floats: two lane groups at rows 4 apart
//     reading 32 floats each touch opposite halves of the banks;
//   * W block, 64 x 64, unpadded: it is read only along its rows.
// A load instruction fills 1 KB of the tile; each lane loads the global chunk
// that belongs at its 16 bytes, or a zeroed page for padding and past an edge.
#include <type_traits>

#include "direct_load.h"

namespace agn {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int STRIP = 64;        // columns j of W_l per workgroup
constexpr int BLK = 64;          // rows i of W_l per block
constexpr int ROWS = 128;        // mini-batch rows held (m <= ROWS)
constexpr int NT_S = 512;        // 8 waves
constexpr int ZS = 68;           // floats per LDS row: dZ block
constexpr int HS = 72;           //                     H strip
constexpr int WS = 64;           //                     W block
constexpr int Z_F = ROWS * ZS;   // tile sizes in floats
constexpr int H_F = ROWS * HS;
constexpr int W_F = BLK * WS;
constexpr int Z_Q = Z_F / 256;   // load instructions (1 KB each) per tile
constexpr int H_Q = H_F / 256;
constexpr int W_Q = W_F / 256;
static_assert(Z_F % 256 == 0 && H_F % 256 == 0 && W_F % 256 == 0, "tiles fill whole load instructions");
static_assert((H_F + 2 * (Z_F + W_F)) * 4 <= 160 * 1024, "LDS: H strip and two stages of dZ and W");
// fewest workgroups (workers x strips) for which the strip schedule is used:
// one workgroup per compute unit at a time (136 KB of LDS), so fewer would
// leave compute units idle or the last wave of workgroups mostly empty
constexpr int64_t kStripMinGroups = 1024;
// waves that issue a block's loads inside the loop (the others go straight
// to their MFMAs while these wait for room in the memory pipeline)
constexpr int FIRE_WAVES = 4;

// Source of this lane's 16 bytes in load instruction q of a tile with S
// floats per LDS row whose row r is row row0 + r of a row-major matrix (ld
// floats per row), columns col0 .. col0 + 63; padding, rows >= nrow and
// columns >= ncol (a multiple of 4) read zeros.
template <int S>
__device__ __forceinline__ const float* tile_src(const float* base, int64_t ld, int row0, int nrow, int col0,
                                                 int ncol, int q, int lane, const float* zero) {
  const int f = 256 * q + 4 * lane;
  const int r = f / S, c = f - r * S;
  const int gr = row0 + r, gc = col0 + c;
  return (c < 64 && gr < nrow && gc < ncol) ? base + (int64_t)gr * ld + gc : zero;
}

struct StripCtx {
  const float* dz;   // dZ_{l+1} of this worker [m][ld_z]
  const float* w;    // W_l (source) of this worker [d_{l+1}][ldw]
  int64_t ld_z, ldw;
  int m, mo, j0, ncol;  // rows, layer outputs d_{l+1}, strip start, layer inputs d_l
  const float* zero;
};

// The loads of block t (rows i0 = 64t): dZ[:, i0..] and W[i0.., strip] into
// stage buffers zs, ws; instruction q of a tile is issued by wave q % NW
// (waves NW.. issue none).
template <int NW>
__device__ __forceinline__ void fire_block(const StripCtx& s, int t, float* zs, float* ws, int wave, int lane) {
  if (wave >= NW) return;
  const int i0 = BLK * t;
#pragma unroll
  for (int u = 0; u < (Z_Q + NW - 1) / NW; ++u) {
    const int q = wave + NW * u;
    if (q < Z_Q) fire(tile_src<ZS>(s.dz, s.ld_z, 0, s.m, i0, s.mo, q, lane, s.zero), lds_off(zs) + 1024 * q);
  }
#pragma unroll
  for (int u = 0; u < (W_Q + NW - 1) / NW; ++u) {
    const int q = wave + NW * u;
    if (q < W_Q) fire(tile_src<WS>(s.w, s.ldw, i0, s.mo, s.j0, s.ncol, q, lane, s.zero), lds_off(ws) + 1024 * q);
  }
}

// Every wave computes a part of both products for each block:
//   * input gradient: rows 16w + 0..15 of the 128-row mini-batch (w = wave)
//     x the strip's 64 columns, as 4 blocks of 16 x 16; block cb covers
//     columns 4*(0..15) + cb, so one 16-byte LDS read of W gives a lane its
//     operand of all four blocks.  K = the block's 64 rows i: lane group g
//     supplies i = 16c + 4g + e in slice (c, e); four groups c of four
//     slices, each reading A once (i = 16c + 4g .. +3 of row 16w + li) and
//     B per slice.  Group c covers rows 16c .. 16c + 15 of the block, so the
//     groups past the layer's last row (zeros in both tiles) are skipped.
//   * weight gradient: rows i 16wi + 0..15 (wi = w / 2) x columns j
//     32wj + 2*(0..15) + (0, 1) (wj = w % 2) of the block's 64 x 64, as 2
//     blocks of 16 x 16 read with one 8-byte LDS read of H per slice.
//     K = the mini-batch rows: lane group g supplies m = 16c + 4g + e in
//     slice (c, e); eight groups c of four slices.
//     A wave whose 16 rows i all lie past the layer's last row skips its
//     MFMAs (only the last block of a ragged layer has such rows).
// Every wave runs its weight-gradient part first, then its input-gradient
// part: the older wave of a SIMD wins the MFMA arbitration, so in the other
// order one wave's update epilogue ran while its partner had no MFMAs left.
// In each part the reads of group c + 1 are issued before the MFMAs of group
// c; scheduling fences keep the scheduler from sinking them next to their
// use.
struct DxFrag {
  f32x4 a, b[4];
};

// pa: row 16w + li, column 4g of the dZ block; pb: row 4g, column 4li of
// the W block
__device__ __forceinline__ void dx_read(const float* pa, const float* pb, int c, DxFrag& f) {
  f.a = *reinterpret_cast<const f32x4*>(pa + 16 * c);
#pragma unroll
  for (int e = 0; e < 4; ++e) f.b[e] = *reinterpret_cast<const f32x4*>(pb + WS * (16 * c + e));
}

__device__ __forceinline__ void dx_mma(const DxFrag& f, f32x4 (&acc)[4]) {
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.a[e], f.b[e][cb], acc[cb], 0, 0, 0);
}

__device__ __forceinline__ void dx_part(const float* pa, const float* pb, f32x4 (&acc)[4]) {
  DxFrag f[2];
  dx_read(pa, pb, 0, f[0]);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    if (c + 1 < 4) {
      dx_read(pa, pb, c + 1, f[(c + 1) & 1]);
      __builtin_amdgcn_sched_group_barrier(0x100, 5, 0);  // the next group's LDS reads first
    }
    dx_mma(f[c & 1], acc);
    __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);  // then this group's MFMAs
    __builtin_amdgcn_sched_barrier(0);
  }
}

struct DwFrag {
  float a[4];
  f32x2 b[4];
};

// qa: row 4g, column 16wi + li of the dZ block; qb: row 4g, column
// 32wj + 2li of the H strip
__device__ __forceinline__ void dw_read(const float* qa, const float* qb, int c, DwFrag& f) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f.a[e] = qa[ZS * (16 * c + e)];
    f.b[e] = *reinterpret_cast<const f32x2*>(qb + HS * (16 * c + e));
  }
}

// Slices of even and odd e accumulate into separate sets, added at the end:
// four independent MFMA chains, as in the input-gradient part, instead of
// two.  BIAS: also the lane's partial column sum of dZ (only the waves that
// store the bias gradient pay for it)
template <bool BIAS>
__device__ __forceinline__ void dw_part(const float* qa, const float* qb, f32x4 (&out)[2], float& bsum) {
  f32x4 acc[2][2];
#pragma unroll
  for (int h = 0; h < 2; ++h) acc[h][0] = acc[h][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  DwFrag f[2];
  dw_read(qa, qb, 0, f[0]);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    if (c + 1 < 8) {
      dw_read(qa, qb, c + 1, f[(c + 1) & 1]);
      __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[e & 1][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(f[c & 1].a[e], f[c & 1].b[e].x, acc[e & 1][0], 0, 0, 0);
      acc[e & 1][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(f[c & 1].a[e], f[c & 1].b[e].y, acc[e & 1][1], 0, 0, 0);
      if (BIAS) bsum += f[c & 1].a[e];
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  out[0] = acc[0][0] + acc[1][0];
  out[1] = acc[0][1] + acc[1][1];
}

// The weight update of a 64 x 64 block: W_dst = W_src - eta * dW, or with
// Adam W_src - eta * mhat / (sqrt(vhat) + eps) (a round's last step: (W_dst -
// W_snap) / lambda); lane: rows i = i0 + 16wi + 4lg + r, columns
// j = j0 + 32wj + 2li + (0, 1) (wi = wave / 2, wj = wave % 2); in the strip
// that holds column 0 the waves with wj == 0 also update b at rows
// i = i0 + 16wi + li.
struct Update {
  f32x4 aw[2];         // dW
  f32x2 wsrc[4];       // W_src
  f32x2 snap[4];       // W_snap (last step)
  f32x2 mw[4], vw[4];  // Adam moments of the weights
  float bsum;          // partial column sum of dZ (bias waves)
  float bsrc, bsnap, mb, vb;
};

// ADAM: Adam as the local rule, its moments read with the update's other
// memory operands and written with the weights
template <bool LAST, bool ADAM>
struct StripUpdate {
  const GemmArgs& dw;
  AdamCoef ac;
  int wi, wj, li, lg, lane;
  int owa, owb, owe;  // per-lane read offsets in the dZ, H and W tiles

  __device__ __forceinline__ StripUpdate(const GemmArgs& g, int wave, int li_, int lg_, int lane_)
      : dw(g), ac(ADAM ? adam_coef(g.g, g.adam) : AdamCoef{1.f, 1.f}), wi(wave >> 1), wj(wave & 1), li(li_),
        lg(lg_), lane(lane_) {
    owa = ZS * 4 * lg + 16 * wi + li;
    owb = HS * 4 * lg + 32 * wj + 2 * li;
    owe = WS * (16 * wi + 4 * lg) + 32 * wj + 2 * li;
  }

  // the update's memory operands (rows and columns clamped into the
  // matrix; the stores check the edges)
  __device__ __forceinline__ void load(Update& u, int64_t wo, int i0, int j0, bool bias) const {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = min(i0 + 16 * wi + 4 * lg + r, dw.M - 1);
      const int j = min(j0 + 32 * wj + 2 * li, dw.N - 2);
      const int64_t e = wo + (int64_t)i * dw.ldw + j;
      if (LAST) u.snap[r] = *reinterpret_cast<const f32x2*>(dw.w_snap + e);
      if (ADAM) {
        u.mw[r] = *reinterpret_cast<const f32x2*>(dw.adam.mw + e);
        u.vw[r] = *reinterpret_cast<const f32x2*>(dw.adam.vw + e);
      }
    }
    if (bias && wj == 0) {
      const int64_t e = wo + min(i0 + 16 * wi + li, dw.M - 1);
      u.bsrc = dw.b_src[e];
      if (LAST) u.bsnap = dw.b_snap[e];
      if (ADAM) {
        u.mb = dw.adam.mb[e];
        u.vb = dw.adam.vb[e];
      }
    }
  }

  // the block's weight gradient from the dZ block zs and the strip hs, and
  // W_src from the W block ws
  __device__ __forceinline__ void mma(const float* zs, const float* ws, const float* hs, Update& u,
                                      bool bias) const {
    u.bsum = 0.f;
    if (bias && wj == 0)
      dw_part<true>(zs + owa, hs + owb, u.aw, u.bsum);
    else
      dw_part<false>(zs + owa, hs + owb, u.aw, u.bsum);
#pragma unroll
    for (int r = 0; r < 4; ++r) u.wsrc[r] = *reinterpret_cast<const f32x2*>(ws + owe + WS * r);
  }

  // the block's stores (past an edge into the sink)
  __device__ __forceinline__ void store(const Update& u, int64_t wo, int i0, int j0, bool bias) const {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      f32x2 d = {u.aw[0][r], u.aw[1][r]}, m = {0.f, 0.f}, v2 = {0.f, 0.f};
      if (ADAM) {
        float mx = u.mw[r].x, my = u.mw[r].y, vx = u.vw[r].x, vy = u.vw[r].y;
        d.x = adam_moments(d.x, mx, vx, dw.adam, ac);
        d.y = adam_moments(d.y, my, vy, dw.adam, ac);
        m = f32x2{mx, my};
        v2 = f32x2{vx, vy};
      }
      f32x2 v = {u.wsrc[r].x - dw.eta * d.x, u.wsrc[r].y - dw.eta * d.y};
      if (LAST) {
        v.x = (v.x - u.snap[r].x) / dw.lam;
        v.y = (v.y - u.snap[r].y) / dw.lam;
      }
      const int i = i0 + 16 * wi + 4 * lg + r, j = j0 + 32 * wj + 2 * li;
      const bool in = i < dw.M && j < dw.N;
      const int64_t e = wo + (int64_t)i * dw.ldw + j;
      f32x2* sink = reinterpret_cast<f32x2*>(dw.sink) + (lane & 31);
      f32x2* dst = in ? reinterpret_cast<f32x2*>(dw.w_dst + e) : sink;
      if (LAST)
        *dst = v;
      else
        __builtin_nontemporal_store(v, dst);
      if (ADAM) {
        __builtin_nontemporal_store(m, in ? reinterpret_cast<f32x2*>(dw.adam.mw + e) : sink);
        __builtin_nontemporal_store(v2, in ? reinterpret_cast<f32x2*>(dw.adam.vw + e) : sink);
      }
    }
    if (bias && wj == 0) {
      // lane groups 1..3 hold partial sums of the same column of dZ as
      // group 0: add them in a fixed order
      const float p1 = __shfl(u.bsum, li + 16), p2 = __shfl(u.bsum, li + 32), p3 = __shfl(u.bsum, li + 48);
      float tot = ((u.bsum + p1) + p2) + p3;
      const int i = i0 + 16 * wi + li;
      if (lg == 0 && i < dw.M) {
        const int64_t e = wo + i;
        if (ADAM) {
          float m = u.mb, v2 = u.vb;
          tot = adam_moments(tot, m, v2, dw.adam, ac);
          dw.adam.mb[e] = m;
          dw.adam.vb[e] = v2;
        }
        const float nb = u.bsrc - dw.eta * tot;
        dw.b_dst[e] = LAST ? (nb - u.bsnap) / dw.lam : nb;
      }
    }
  }
};

template <bool LAST, bool ADAM>
__global__ __launch_bounds__(NT_S) void gemm_f32_strip_bwd_kernel(GemmArgs dx, GemmArgs dw) {
  __shared__ __attribute__((aligned(16))) float hs[H_F];
  __shared__ __attribute__((aligned(16))) float zs0[Z_F];
  __shared__ __attribute__((aligned(16))) float zs1[Z_F];
  __shared__ __attribute__((aligned(16))) float ws0[W_F];
  __shared__ __attribute__((aligned(16))) float ws1[W_F];
  const int tid = threadIdx.x, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & 7;  // uniform: the roles branch per wave
  const int nstrip = (dx.N + STRIP - 1) / STRIP;
  const int logical = xcd_remap(blockIdx.x, (int)gridDim.x);
  const int worker = logical / nstrip, j0 = (logical % nstrip) * STRIP;
  const int T = (dw.M + BLK - 1) / BLK;

  StripCtx s;
  s.dz = reinterpret_cast<const float*>(dx.a.ptr) + (int64_t)worker * dx.a.wstride;
  s.w = dw.w_src + (int64_t)worker * dw.pstride;
  s.ld_z = dx.a.ld;
  s.ldw = dw.ldw;
  s.m = dx.M;
  s.mo = dw.M;
  s.j0 = j0;
  s.ncol = dx.N;
  s.zero = dx.zero;
  const float* h = reinterpret_cast<const float*>(dw.b.ptr) + (int64_t)worker * dw.b.wstride;

  // prologue: the H strip, then block 0
#pragma unroll
  for (int u = 0; u < (H_Q + 7) / 8; ++u) {
    const int q = wave + 8 * u;
    if (q < H_Q) fire(tile_src<HS>(h, dw.b.ld, 0, s.m, j0, s.ncol, q, lane, s.zero), lds_off(hs) + 1024 * q);
  }
  fire_block<8>(s, 0, zs0, ws0, wave, lane);

  const int64_t wo = (int64_t)worker * dw.pstride;
  const StripUpdate<LAST, ADAM> up(dw, wave, li, lg, lane);
  // the bias is updated by the strip at j0 == 0
  const bool bias = j0 == 0;
  // per-lane offsets of the input-gradient reads (floats from the tile's start)
  const int oxa = ZS * (16 * wave + li) + 4 * lg, oxb = WS * 4 * lg + 4 * li;
  f32x4 ax[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) ax[b] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Per block t: wait for its loads; store the update of block t-1 while
  // the memory pipeline is empty (a store issued behind the next block's
  // loads holds up the wave until they land); load the update operands of
  // block t; issue the loads of block t+1; then the weight gradient and the
  // input gradient of block t from LDS.
  Update held;  // the update of block t-1, not yet stored
  for (int t = 0; t < T; ++t) {
    const float* zs = (t & 1) ? zs1 : zs0;
    const float* ws = (t & 1) ? ws1 : ws0;
    // every memory operation of this wave so far has completed (the loads
    // of block t among them); after the barrier, those of every wave, and
    // every wave is done with the other stage buffers
    wait_lgkm0();
    wait_vm<0>();
    barrier();
    if (t > 0) up.store(held, wo, BLK * (t - 1), j0, bias);
    up.load(held, wo, BLK * t, j0, bias);
    if (t + 1 < T) fire_block<FIRE_WAVES>(s, t + 1, (t & 1) ? zs0 : zs1, (t & 1) ? ws0 : ws1, wave, lane);
    up.mma(zs, ws, hs, held, bias);
    dx_part(zs + oxa, ws + oxb, ax);
  }
  up.store(held, wo, BLK * (T - 1), j0, bias);
  // dZ_l = acc * [H_l > 0]; lane: rows 16w + 4lg + r, columns 4li + (0..3)
  wait_lgkm0();
  float* out = reinterpret_cast<float*>(dx.out) + (int64_t)worker * dx.ostride;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int m = 16 * wave + 4 * lg + r;
    const f32x4 mk = *reinterpret_cast<const f32x4*>(hs + HS * m + 4 * li);
    const f32x4 v = {mk.x > 0.f ? ax[0][r] : 0.f, mk.y > 0.f ? ax[1][r] : 0.f, mk.z > 0.f ? ax[2][r] : 0.f,
                     mk.w > 0.f ? ax[3][r] : 0.f};
    const int j = j0 + 4 * li;
    if (m < dx.M && j < dx.N) *reinterpret_cast<f32x4*>(out + (int64_t)m * dx.ldo + j) = v;
  }
}

// ---------------------------------------------------------------------------
// The first layer's weight gradient as strips of its rows: dW_0 = dZ_1^T X_b
// (X_b: the worker's mini-batch rows of the data set, K = m) fused with the
// update of W_0 and b_0 (Algorithm 1, gradient line and local step).  A
// workgroup owns one worker and one strip of 64 rows i of W_0 (64 units of
// the first hidden layer): dZ_1[:, strip] (128 x 64) stays in LDS for the
// whole launch, and the workgroup walks the blocks of 64 columns j (inputs).
// Per block only the gathered X_b[:, block] (128 x 64) travels into LDS
// (direct loads, double-buffered, issued by four waves); W_src, and on a
// round's last step W_snap, come into registers for the update.  The product
// and the update's lane layout are those of the backward strip kernel's
// weight-gradient part (dZ strip as A, X block as B), so the bias gradient
// comes from the A fragments of the first block.

// Source of this lane's 16 bytes in load instruction q of the X block whose
// row r is batch row r of worker k (data-set row k*S + (tb + r) mod S),
// columns col0 .. col0 + 63; padding, rows >= m and columns >= ncol read
// zeros.
__device__ __forceinline__ const float* xblock_src(const float* x, int64_t ldx, int64_t rowk, int64_t S, int64_t tb,
                                                   int m, int col0, int ncol, int q, int lane, const float* zero) {
  const int f = 256 * q + 4 * lane;
  const int r = f / HS, c = f - r * HS;
  const int gc = col0 + c;
  if (c >= 64 || r >= m || gc >= ncol) return zero;
  int64_t j = tb + r;
  if (j >= S) j -= S;
  return x + (rowk + j) * ldx + gc;
}

template <bool LAST, bool ADAM>
__global__ __launch_bounds__(512) void gemm_f32_strip_dw_kernel(GemmArgs dw) {
  __shared__ __attribute__((aligned(16))) float zs[Z_F];
  __shared__ __attribute__((aligned(16))) float xs0[H_F];
  __shared__ __attribute__((aligned(16))) float xs1[H_F];
  const int tid = threadIdx.x, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & 7;  // uniform: the roles branch per wave
  const int wi = wave >> 1, wj = wave & 1;
  const int nstrip = (dw.M + STRIP - 1) / STRIP;
  const int logical = xcd_remap(blockIdx.x, (int)gridDim.x);
  const int worker = logical / nstrip, i0 = (logical % nstrip) * STRIP;
  const int T = (dw.N + BLK - 1) / BLK;
  const int m = dw.K;
  const float* dz = reinterpret_cast<const float*>(dw.a.ptr) + (int64_t)worker * dw.a.wstride;
  const float* x = reinterpret_cast<const float*>(dw.b.ptr);
  const int64_t S = dw.g.S, rowk = (int64_t)worker * S;
  const int64_t tb = (gather_step(dw.g) * dw.g.mb) % S;
  // the loads of X block t into dst; instruction q is issued by wave q % NW
  auto fire_x = [&](auto nw, int t, float* dst) {
    constexpr int NW = decltype(nw)::value;
#pragma unroll
    for (int u = 0; u < (H_Q + NW - 1) / NW; ++u) {
      const int q = wave + NW * u;
      if (q < H_Q)
        fire(xblock_src(x, dw.b.ld, rowk, S, tb, m, BLK * t, dw.N, q, lane, dw.zero), lds_off(dst) + 1024 * q);
    }
  };

  // prologue: the dZ strip and X block 0, issued by every wave
#pragma unroll
  for (int u = 0; u < (Z_Q + 7) / 8; ++u) {
    const int q = wave + 8 * u;
    if (q < Z_Q) fire(tile_src<ZS>(dz, dw.a.ld, 0, m, i0, dw.M, q, lane, dw.zero), lds_off(zs) + 1024 * q);
  }
  fire_x(std::integral_constant<int, 8>{}, 0, xs0);

  const int64_t wo = (int64_t)worker * dw.pstride;
  const int owa = ZS * 4 * lg + 16 * wi + li, owb = HS * 4 * lg + 32 * wj + 2 * li;
  // this lane's rows of the update: i0 + 16wi + 4lg + r (clamped for the loads)
  int64_t rowo[4];
  bool rin[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = i0 + 16 * wi + 4 * lg + r;
    rin[r] = i < dw.M;
    rowo[r] = wo + (int64_t)min(i, dw.M - 1) * dw.ldw;
  }
  f32x4 aw[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  f32x2 wsrc[4], snap[4], mw[4], vw[4];
  float bsum = 0.f;
  const AdamCoef ac = ADAM ? adam_coef(dw.g, dw.adam) : AdamCoef{1.f, 1.f};

  // the update of block t (columns j0 = 64t + 32wj + 2li, +1): its operands
  // (UPL loads: W_src, the snapshot on the last step, Adam's two moments)
  // and its stores (UST: the weights and the moments, every lane storing,
  // past an edge into the sink)
  constexpr int UPL = 4 + (LAST ? 4 : 0) + (ADAM ? 8 : 0);
  constexpr int UST = ADAM ? 12 : 4;
  auto load_update = [&](int t) {
    const int j = min(BLK * t + 32 * wj + 2 * li, dw.N - 2);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      wsrc[r] = *reinterpret_cast<const f32x2*>(dw.w_src + rowo[r] + j);
      if (LAST) snap[r] = *reinterpret_cast<const f32x2*>(dw.w_snap + rowo[r] + j);
      if (ADAM) {
        mw[r] = *reinterpret_cast<const f32x2*>(dw.adam.mw + rowo[r] + j);
        vw[r] = *reinterpret_cast<const f32x2*>(dw.adam.vw + rowo[r] + j);
      }
    }
  };
  auto store_update = [&](int t) {
    const int j = BLK * t + 32 * wj + 2 * li;
    f32x2* sink = reinterpret_cast<f32x2*>(dw.sink) + (lane & 31);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      f32x2 d = {aw[0][r], aw[1][r]};
      if (ADAM) {
        float mx = mw[r].x, my = mw[r].y, vx = vw[r].x, vy = vw[r].y;
        d.x = adam_moments(d.x, mx, vx, dw.adam, ac);
        d.y = adam_moments(d.y, my, vy, dw.adam, ac);
        mw[r] = f32x2{mx, my};
        vw[r] = f32x2{vx, vy};
      }
      f32x2 v = {wsrc[r].x - dw.eta * d.x, wsrc[r].y - dw.eta * d.y};
      if (LAST) {
        v.x = (v.x - snap[r].x) / dw.lam;
        v.y = (v.y - snap[r].y) / dw.lam;
      }
      const bool in = rin[r] && j < dw.N;
      f32x2* dst = in ? reinterpret_cast<f32x2*>(dw.w_dst + rowo[r] + j) : sink;
      if (LAST)
        *dst = v;
      else
        __builtin_nontemporal_store(v, dst);
      if (ADAM) {
        __builtin_nontemporal_store(mw[r], in ? reinterpret_cast<f32x2*>(dw.adam.mw + rowo[r] + j) : sink);
        __builtin_nontemporal_store(vw[r], in ? reinterpret_cast<f32x2*>(dw.adam.vw + rowo[r] + j) : sink);
      }
    }
  };

  // Per block t: wait for its loads; issue the loads of block t+1 (waves
  // 0-3); the product of block t from LDS; then its update's stores and the
  // update operands of block t+1.  Those two sets of memory operations
  // (UST + UPL per wave) are younger than every direct load a wave waits for
  // at the next block, so they stay in flight across the barrier; a store
  // or load issued at the start of a block waited behind that block's
  // direct loads.
  load_update(0);
  for (int t = 0; t < T; ++t) {
    const float* xs = (t & 1) ? xs1 : xs0;
    wait_lgkm0();
    if (t == 0)
      wait_vm<UPL>();
    else
      wait_vm<UST + UPL>();
    barrier();
    if (t + 1 < T && wave < 4) fire_x(std::integral_constant<int, 4>{}, t + 1, (t & 1) ? xs0 : xs1);
    if (t == 0 && wj == 0) {
      dw_part<true>(zs + owa, xs + owb, aw, bsum);
    } else {
      float unused = 0.f;
      dw_part<false>(zs + owa, xs + owb, aw, unused);
    }
    store_update(t);
    if (t + 1 < T) load_update(t + 1);
  }
  if (wj == 0) {
    // the bias of rows i0 + 16wi + li: lane groups 1..3 hold partial sums
    // of the same column of dZ_1 as group 0, added in a fixed order
    const float p1 = __shfl(bsum, li + 16), p2 = __shfl(bsum, li + 32), p3 = __shfl(bsum, li + 48);
    float tot = ((bsum + p1) + p2) + p3;
    const int i = i0 + 16 * wi + li;
    if (lg == 0 && i < dw.M) {
      const int64_t e = wo + i;
      if (ADAM) {
        float mb = dw.adam.mb[e], vb = dw.adam.vb[e];
        tot = adam_moments(tot, mb, vb, dw.adam, ac);
        dw.adam.mb[e] = mb;
        dw.adam.vb[e] = vb;
      }
      const float nb = dw.b_src[e] - dw.eta * tot;
      dw.b_dst[e] = LAST ? (nb - dw.b_snap[e]) / dw.lam : nb;
    }
  }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

// The strip schedule applies to one float32 hidden layer whose products share
// their operands as enqueue_step builds them (input gradient: A = dZ_{l+1},
// B = W_l, mask = H_l; weight gradient: A = dZ_{l+1}, B = H_l, W_src = W_l),
// with a mini-batch of at most 128 rows, widths and row strides that allow
// 16-byte chunks (the Adam moments too), and enough strips (workers x
// column strips) to give every compute unit several workgroups.
bool gemm_f32_strip_ok(const GemmArgs& dx, const GemmArgs& dw) {
  if (dx.epi != EPI_DX_MASK || dw.epi != EPI_DW_UPDATE || !dx.zero || !dw.sink) return false;
  if (dx.M < 1 || dx.M > ROWS || dw.K != dx.M || dx.N != dw.N || dx.K != dw.M || dx.batch != dw.batch) return false;
  if (dx.N % 4 || dw.M % 4 || dx.N < 2) return false;
  if (dx.a.ptr != dw.a.ptr || dx.a.ld != dw.a.ld || dx.a.wstride != dw.a.wstride || dx.a.gather || dw.b.gather)
    return false;
  if (dx.b.ptr != dw.w_src || dx.b.ld != dw.ldw || dx.b.wstride != dw.pstride) return false;
  if (dx.mask != dw.b.ptr || dx.ldm != dw.b.ld || dx.mstride != dw.b.wstride) return false;
  const void* ptrs[] = {dx.a.ptr, dw.b.ptr, dw.w_src, dw.w_dst, dx.out, dx.zero, dw.sink};
  for (const void* p : ptrs)
    if (!aligned16(p)) return false;
  if (dw.last && !aligned16(dw.w_snap)) return false;
  if (dw.adam.on && (!aligned16(dw.adam.mw) || !aligned16(dw.adam.vw) || !dw.adam.mb || !dw.adam.vb)) return false;
  if (dx.a.ld % 4 || dx.a.wstride % 4 || dw.b.ld % 4 || dw.b.wstride % 4 || dw.ldw % 4 || dw.pstride % 4 ||
      dx.ldo % 4 || dx.ostride % 4)
    return false;
  const int64_t groups = (int64_t)dx.batch * ((dx.N + STRIP - 1) / STRIP);
  return groups >= kStripMinGroups && groups < (1 << 30);
}

hipError_t launch_gemm_f32_strip_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s) {
  if (!gemm_f32_strip_ok(dx, dw)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(dx.batch * ((dx.N + STRIP - 1) / STRIP))), block(NT_S);
  if (dw.adam.on) {
    if (dw.last)
      AGN_LAUNCH((gemm_f32_strip_bwd_kernel<true, true>), grid, block, 0, s, dx, dw);
    else
      AGN_LAUNCH((gemm_f32_strip_bwd_kernel<false, true>), grid, block, 0, s, dx, dw);
  } else if (dw.last) {
    AGN_LAUNCH((gemm_f32_strip_bwd_kernel<true, false>), grid, block, 0, s, dx, dw);
  } else {
    AGN_LAUNCH((gemm_f32_strip_bwd_kernel<false, false>), grid, block, 0, s, dx, dw);
  }
  return hipGetLastError();
}

// The strip schedule of the first layer's weight gradient: gathered data
// rows as B (a batch within a shard), dZ_1 as A, SGD or Adam as the local
// rule, a mini-batch of at most 128 rows, 16-byte rows, and enough strips
// (workers x 64-row strips of W_0) to give every compute unit several
// workgroups.
bool gemm_f32_strip_dw_ok(const GemmArgs& dw) {
  if (dw.epi != EPI_DW_UPDATE || !dw.zero || !dw.sink || dw.w_dst16) return false;
  if (dw.adam.on && (!aligned16(dw.adam.mw) || !aligned16(dw.adam.vw) || !dw.adam.mb || !dw.adam.vb)) return false;
  if (!dw.b.gather || dw.a.gather || dw.K < 1 || dw.K > ROWS || dw.K > dw.g.S) return false;
  if (dw.M % 4 || dw.N % 4 || dw.N < 2) return false;
  const void* ptrs[] = {dw.a.ptr, dw.b.ptr, dw.w_src, dw.w_dst, dw.zero, dw.sink};
  for (const void* p : ptrs)
    if (!aligned16(p)) return false;
  if (dw.last && !aligned16(dw.w_snap)) return false;
  if (dw.a.ld % 4 || dw.a.wstride % 4 || dw.b.ld % 4 || dw.ldw % 4 || dw.pstride % 4) return false;
  const int64_t groups = (int64_t)dw.batch * ((dw.M + STRIP - 1) / STRIP);
  return groups >= kStripMinGroups && groups < (1 << 30);
}

hipError_t launch_gemm_f32_strip_dw(const GemmArgs& dw, hipStream_t s) {
  if (!gemm_f32_strip_dw_ok(dw)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(dw.batch * ((dw.M + STRIP - 1) / STRIP))), block(512);
  if (dw.adam.on) {
    if (dw.last)
      AGN_LAUNCH((gemm_f32_strip_dw_kernel<true, true>), grid, block, 0, s, dw);
    else
      AGN_LAUNCH((gemm_f32_strip_dw_kernel<false, true>), grid, block, 0, s, dw);
  } else if (dw.last) {
    AGN_LAUNCH((gemm_f32_strip_dw_kernel<true, false>), grid, block, 0, s, dw);
  } else {
    AGN_LAUNCH((gemm_f32_strip_dw_kernel<false, false>), grid, block, 0, s, dw);
  }
  return hipGetLastError();
}

}  // namespace agn
