// Batched float32 products with direct global->LDS operand loads
// (global_load_lds_dwordx4 on gfx950): operand tiles travel from memory into
// LDS without passing through registers, three K steps ahead of their use,
// and the fragments of the next K step are read from LDS while the MFMAs of
// the current one run.
//
// Tile: 64x64 outputs per workgroup of 4 waves; wave (wm, wn) owns a 32x32
// block as 2x2 blocks of v_mfma_f32_16x16x4_f32; K in steps of 32.  In one
// MFMA, lane l supplies A[i = l%16][k = l/16] and B[k = l/16][j = l%16] and
// holds D[4*(l/16) + r][l%16] in accumulator register r.  A K step is eight
// MFMA slices s; lane group g = l/16 covers k = 8g + s of the step, so over
// the eight slices a lane reads 8 consecutive k of its row or column.
//
// Which tile rows (columns) a 16x16 block covers depends on the operand's
// layout in memory:
//   K-contiguous: block b covers rows 16b .. 16b+15 of the wave's 32, and a
//     lane reads its 8 k as two 16-byte LDS reads;
//   K-strided: block b covers rows 2i + b, i = 0..15 (interleaved), and one
//     8-byte LDS read gives a lane the operand of both blocks at one k.
// The epilogue maps each accumulator back to its (row, column).
//
// LDS layout of one operand tile (64 x 32 floats = 512 chunks of 16 bytes;
// a wave's load instruction fills 64 consecutive chunks, lane l chunk l):
//   K-contiguous (rows = outer index, 8 chunks of 4 k per row):
//     chunk (r, q) at r*8 + (q ^ key(r)), key(r) = (r&7) ^ ((r>>3)&1): the
//     rows of 8 consecutive lanes of a 16-byte read fall in 8 distinct
//     16-byte bank groups modulo 128 bytes, and those of 16 consecutive
//     lanes in 16 distinct groups modulo 256 bytes;
//   K-strided (rows = k, 16 chunks of 4 outer per row):
//     chunk (k, c) at k*16 + (c ^ (8*((k>>3)&1))), so rows k and k+8, read
//     together by lane groups 0 and 1, land in opposite halves of the banks.
// Each lane loads the global 16 bytes that belong in its slot; lanes past an
// edge read a zero page, so edge tiles hold exact zeros.
//
// Two schedules:
//   * forward and input-gradient products (K = layer width, tens of K
//     steps): one output tile per workgroup (the forward with eight waves
//     that split each K step between two waves per block);
//   * weight-gradient products (K = mini-batch, a few K steps per tile):
//     persistent workgroups walk a list of tiles and the operand loads run
//     on across tile boundaries, so a tile's first steps load while the
//     previous tile computes and stores.  The weight (and, on a round's last
//     step, snapshot) tile of the epilogue is loaded into LDS by the same
//     direct loads, so that every wait on the load counter has a known
//     count.
#include <cmath>
#include <type_traits>

#include "direct_load.h"
#include "head_dw_unit.h"

namespace agn {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int NT = 256, TM = 64, BKD = 32, NS = 4;  // NS: LDS stages
constexpr int TILE_F = TM * BKD;                     // floats per operand tile
constexpr int STAGE_F = 2 * TILE_F;                  // A and B
constexpr int EPI_F = TM * TM;                       // floats of one epilogue operand tile
constexpr int EPI_ADAM_F = 3 * EPI_F + 2 * 256;      // W_src, the Adam moments, the bias moments
constexpr int NWG_DW = 512;                          // persistent weight-gradient workgroups (2 per CU)
constexpr int NWG_DW_ADAM = 256;                     // with Adam's moment tiles in LDS: 1 per CU

__device__ __forceinline__ int kc_key(int r) { return (r & 7) ^ ((r >> 3) & 1); }
__device__ __forceinline__ int kc_slot(int r, int q) { return r * 8 + (q ^ kc_key(r)); }
__device__ __forceinline__ int ks_slot(int k, int c) { return k * 16 + (c ^ (((k >> 3) & 1) << 3)); }


// Slot of lane `lane` in load instruction j of a K-strided tile: k row and
// 16-byte column chunk.
__device__ __forceinline__ int ks_row(int j, int lane) { return 4 * j + lane / 16; }
__device__ __forceinline__ int ks_chunk(int j, int lane) {
  return (lane % 16) ^ (((ks_row(j, lane) >> 3) & 1) << 3);
}

// One-tile schedule: one operand's tile loads.  This wave fills slots
// [64j, 64j+64) for j = 2*wave and 2*wave+1 (two load instructions per
// operand per K step).  K-contiguous operands may be gathered (data-set rows
// of the first layer); K-strided ones are not.
template <bool KC>
struct DirectLoader {
  const float* base;
  const float* zero;
  int64_t ld;
  int outer0, outer_n, K;
  const float* rowp[2];      // KC: the lane's two rows (null past the edge)
  // steps whose loads all lie inside K ("full" steps) load from
  // fast[u] + offset(k0): the lane's row (KC) or column chunk (KS) clamped
  // into the matrix -- rows and columns past the edge feed only outputs
  // that are never stored, so any data will do there
  const float* fast[2];
  int lk[2];                 // KC: the lane's k offset inside a step

  __device__ void init(const Operand& op, const Gather& g, const float* zp, int64_t w, int o0, int on, int k,
                       int wave, int lane) {
    base = reinterpret_cast<const float*>(op.ptr) + w * op.wstride;
    zero = zp;
    ld = op.ld;
    outer0 = o0;
    outer_n = on;
    K = k;
    if (KC) {
      const int64_t t = op.gather ? gather_step(g) : 0;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int r = 8 * (2 * wave + u) + lane / 8;
        const int o = o0 + r, oc = o < on ? o : on - 1;
        const int64_t ri = op.gather ? batch_row(w, t, g.mb, g.S, oc) : oc;
        rowp[u] = o < on ? base + ri * ld : nullptr;
        fast[u] = base + ri * ld;
        lk[u] = 4 * ((lane % 8) ^ kc_key(r));
      }
    } else {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int j = 2 * wave + u;
        const int o = o0 + 4 * ks_chunk(j, lane);
        fast[u] = base + (int64_t)ks_row(j, lane) * ld + (o < on ? o : on - 4);  // (on % 4 == 0)
      }
    }
  }

  // source for a full step (every k of the step below K)
  __device__ const float* src_full(int k0, int u) const {
    return KC ? fast[u] + (k0 + lk[u]) : fast[u] + (int64_t)k0 * ld;
  }

  // source of this lane's 16 bytes in load instruction u (0, 1) of the K
  // step starting at k0; the zero page past an edge (also for k0 >= K)
  __device__ const float* src(int k0, int u, int wave, int lane) const {
    const int j = 2 * wave + u;
    if (KC) {
      const int r = 8 * j + lane / 8;
      const int q = (lane % 8) ^ kc_key(r);
      const int k = k0 + 4 * q;
      return (rowp[u] && k < K) ? rowp[u] + k : zero;
    } else {
      const int kk = k0 + ks_row(j, lane), o = outer0 + 4 * ks_chunk(j, lane);
      if (kk >= K || o >= outer_n) return zero;
      return base + (int64_t)kk * ld + o;
    }
  }
};

// Fragments of one wave for one K step: a[b][s] / b[b][s] is the operand of
// block b in slice s (k = 8g + s of the step, g = lane/16).
struct Frags {
  float a[2][8], b[2][8];
};

template <bool KC>
__device__ __forceinline__ void frag(const float* tile, int outer_off, int li, int lg, float (&f)[2][8]) {
  if (KC) {
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int r = outer_off + 16 * b + li;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(tile + 4 * kc_slot(r, 2 * lg + h));
#pragma unroll
        for (int e = 0; e < 4; ++e) f[b][4 * h + e] = v[e];
      }
    }
  } else {
    const int o = outer_off + 2 * li;  // even: blocks 0 and 1 take o and o+1
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const float2 v = *reinterpret_cast<const float2*>(tile + 4 * ks_slot(8 * lg + s, o >> 2) + (o & 3));
      f[0][s] = v.x;
      f[1][s] = v.y;
    }
  }
}

template <bool A_KC, bool B_KC>
__device__ __forceinline__ void read_frags(const float* stage, int wm, int wn, int li, int lg, Frags& f) {
  frag<A_KC>(stage, wm * 32, li, lg, f.a);
  frag<B_KC>(stage + TILE_F, wn * 32, li, lg, f.b);
}

struct Lanes {
  int wave, lane, wm, wn, li, lg;
};

// K step: the fragments of this step are in `cur`; the loads of the next
// NS-1 steps are in flight.  Wait until every wave has read `cur` and the
// next step's loads have landed (VM: load instructions this wave may leave
// in flight, those issued after the next step's), then, interleaved with the
// 32 MFMAs, read the next step's fragments from `rd` into `nxt` and start the
// loads `src` of the step NS ahead into `wr` (the stage this step came from).
// Loads past the end of K read the zero page, so every step has the same
// shape and the MFMAs, LDS reads and loads form one basic block.
template <bool A_KC, bool B_KC, int VM>
__device__ __forceinline__ void k_step(const Lanes& q, const Frags& cur, Frags& nxt, const float* rd, float* wr,
                                       const float* const (&src)[4], f32x4 (&acc)[2][2], float (&bsum)[2]) {
  wait_lgkm0();
  wait_vm<VM>();
  barrier();
  read_frags<A_KC, B_KC>(rd, q.wm, q.wn, q.li, q.lg, nxt);
  const uint32_t wa = lds_off(wr) + 4 * 256 * (2 * q.wave);
  fire(src[0], wa);
  fire(src[1], wa + 4 * 256);
  fire(src[2], wa + 4 * TILE_F);
  fire(src[3], wa + 4 * (TILE_F + 256));
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
        acc[bi][bj] = __builtin_amdgcn_mfma_f32_16x16x4f32(cur.a[bi][s], cur.b[bj][s], acc[bi][bj], 0, 0, 0);
  // bias gradient (used by the weight-gradient product, where A = dZ^T is
  // K-strided): this lane's two columns over its 8 k
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    bsum[0] += cur.a[0][s];
    bsum[1] += cur.a[1][s];
  }
  // issue order: the LDS reads spread between the MFMAs
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // LDS read
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
  }
}

// Tile row (column) of accumulator index x of block b.
template <bool KC>
__device__ __forceinline__ int tile_idx(int b, int x) { return KC ? 16 * b + x : 2 * x + b; }

__host__ __device__ inline int tiles_dl(const GemmArgs& g) { return ((g.M + TM - 1) / TM) * ((g.N + TM - 1) / TM) * g.batch; }

struct TileCoord {
  int worker, m0, n0, tile_n;
};

__device__ __forceinline__ TileCoord coord_of(const GemmArgs& g, int logical) {
  const int tm = (g.M + TM - 1) / TM, tn = (g.N + TM - 1) / TM;
  TileCoord c;
  c.worker = logical / (tm * tn);
  const int rem = logical % (tm * tn);
  c.tile_n = rem / tm;
  c.m0 = (rem % tm) * TM;
  c.n0 = c.tile_n * TM;
  return c;
}

// ---------------------------------------------------------------------------
// One-tile schedule: forward (A = H or gathered data rows, B = W, both
// K-contiguous) and input-gradient (A = dZ K-contiguous, B = W K-strided).

template <bool A_KC, bool B_KC, int EPI>
__device__ __forceinline__ void tile_dl(const GemmArgs& g, const int logical, float* st0, float* st1, float* st2,
                                        float* st3) {
  static_assert(EPI != EPI_DW_UPDATE, "weight-gradient tiles use the persistent schedule");
  const int tid = threadIdx.x;
  const TileCoord c = coord_of(g, logical);
  const int worker = c.worker, m0 = c.m0, n0 = c.n0;
  const Lanes q{tid >> 6, tid & 63, (tid >> 6) >> 1, (tid >> 6) & 1, tid & 15, (tid & 63) >> 4};
  const int rbase = m0 + q.wm * 32, cbase = n0 + q.wn * 32;
  // accumulator (bi, bj, r) sits at row rbase + tile_idx<A_KC>(bi, 4*lg + r),
  // column cbase + tile_idx<B_KC>(bj, li)

  // operands of the epilogue first, oldest in the memory queue: the
  // forward's bias of this lane's two columns, the input gradient's mask.
  // The loads are unconditional (indices clamped into the matrix; values
  // outside it are never stored), so they issue back to back
  float bpre[2] = {0.f, 0.f};
  if (EPI == EPI_FWD_RELU || EPI == EPI_FWD_LINEAR) {
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) {
      const int col = min(cbase + tile_idx<B_KC>(bj, q.li), g.N - 1);
      bpre[bj] = g.bias[(int64_t)worker * g.bstride + col];
    }
  }
  float pre[2][2][4];
  if (EPI == EPI_DX_MASK) {
    const float* mk = reinterpret_cast<const float*>(g.mask) + (int64_t)worker * g.mstride;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) {
          const int row = min(rbase + tile_idx<A_KC>(bi, 4 * q.lg + r), g.M - 1),
                    col = min(cbase + tile_idx<B_KC>(bj, q.li), g.N - 1);
          pre[bi][bj][r] = mk[(int64_t)row * g.ldm + col];
        }
  }

  DirectLoader<A_KC> la;
  DirectLoader<B_KC> lb;
  la.init(g.a, g.g, g.zero, worker, m0, g.M, g.K, q.wave, q.lane);
  lb.init(g.b, g.g, g.zero, worker, n0, g.N, g.K, q.wave, q.lane);

  float bsum[2] = {0.f, 0.f};
  f32x4 acc[2][2];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (g.K + BKD - 1) / BKD;
  // steps 0..3 in flight (4 load instructions per wave per step), then the
  // fragments of step 0
  {
    float* stg[NS] = {st0, st1, st2, st3};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const uint32_t wa = lds_off(stg[s]) + 4 * 256 * (2 * q.wave);
      fire(la.src(s * BKD, 0, q.wave, q.lane), wa);
      fire(la.src(s * BKD, 1, q.wave, q.lane), wa + 4 * 256);
      fire(lb.src(s * BKD, 0, q.wave, q.lane), wa + 4 * TILE_F);
      fire(lb.src(s * BKD, 1, q.wave, q.lane), wa + 4 * (TILE_F + 256));
    }
  }
  wait_vm<4 * (NS - 1)>();
  barrier();
  Frags f0, f1;
  read_frags<A_KC, B_KC>(st0, q.wm, q.wn, q.li, q.lg, f0);

  // step kt loads step kt + NS: from the precomputed full-step sources
  // while that step lies inside K, else through the bounds checks
  auto step = [&](auto full, int kt, const Frags& cur, Frags& nxt, const float* rd, float* wr) {
    const int k0 = (kt + NS) * BKD;
    if constexpr (decltype(full)::value) {
      const float* const src[4] = {la.src_full(k0, 0), la.src_full(k0, 1), lb.src_full(k0, 0),
                                   lb.src_full(k0, 1)};
      k_step<A_KC, B_KC, 4 * (NS - 2)>(q, cur, nxt, rd, wr, src, acc, bsum);
    } else {
      const float* const src[4] = {la.src(k0, 0, q.wave, q.lane), la.src(k0, 1, q.wave, q.lane),
                                   lb.src(k0, 0, q.wave, q.lane), lb.src(k0, 1, q.wave, q.lane)};
      k_step<A_KC, B_KC, 4 * (NS - 2)>(q, cur, nxt, rd, wr, src, acc, bsum);
    }
  };
  using Full = std::true_type;
  using Checked = std::false_type;
  // stage of step kt: kt % 4; fragment set: kt % 2
  const int nk4 = nk & ~3;
  const int nfast = (g.K / BKD - NS > 0 ? g.K / BKD - NS : 0) & ~3;  // steps kt whose step kt+NS is full
  int kt = 0;
  for (; kt < nfast && kt < nk4; kt += 4) {
    step(Full{}, kt, f0, f1, st1, st0);
    step(Full{}, kt + 1, f1, f0, st2, st1);
    step(Full{}, kt + 2, f0, f1, st3, st2);
    step(Full{}, kt + 3, f1, f0, st0, st3);
  }
  for (; kt < nk4; kt += 4) {
    step(Checked{}, kt, f0, f1, st1, st0);
    step(Checked{}, kt + 1, f1, f0, st2, st1);
    step(Checked{}, kt + 2, f0, f1, st3, st2);
    step(Checked{}, kt + 3, f1, f0, st0, st3);
  }
  if (nk4 < nk) step(Checked{}, nk4, f0, f1, st1, st0);
  if (nk4 + 1 < nk) step(Checked{}, nk4 + 1, f1, f0, st2, st1);
  if (nk4 + 2 < nk) step(Checked{}, nk4 + 2, f0, f1, st3, st2);
  // loads of the steps past the end (zero page) still write LDS
  wait_vm<0>();
  // the epilogue operands are in registers now (nothing is in flight): use
  // them here, in straight-line code, so that the compiler's own waits for
  // them land here and not between the conditional stores below (where each
  // would wait for the stores before it)
  if (EPI == EPI_FWD_RELU || EPI == EPI_FWD_LINEAR) asm volatile("" ::"v"(bpre[0]), "v"(bpre[1]));
  if (EPI == EPI_DX_MASK) {
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 4; ++r) asm volatile("" ::"v"(pre[bi][0][r]), "v"(pre[bi][1][r]));
  }

#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) {
        const int row = rbase + tile_idx<A_KC>(bi, 4 * q.lg + r), col = cbase + tile_idx<B_KC>(bj, q.li);
        if (row >= g.M || col >= g.N) continue;
        const float v = acc[bi][bj][r];
        float* out = reinterpret_cast<float*>(g.out) + (int64_t)worker * g.ostride;
        if (EPI == EPI_FWD_RELU || EPI == EPI_FWD_LINEAR) {
          float z = v + bpre[bj];
          if (EPI == EPI_FWD_RELU) z = z > 0.f ? z : 0.f;
          out[(int64_t)row * g.ldo + col] = z;
        } else {  // EPI_DX_MASK
          out[(int64_t)row * g.ldo + col] = pre[bi][bj][r] > 0.f ? v : 0.f;
        }
      }
}

// ---------------------------------------------------------------------------
// Forward product with eight waves (two per SIMD) splitting each K step:
// waves 0-3 take MFMA slices 0-3 of the step, waves 4-7 slices 4-7, each
// wave with the accumulators of its 32 x 32 block (wm, wn).  A wave waiting
// at a barrier or on its LDS reads leaves the matrix core to the other wave
// of its SIMD.  The halves are added (waves 4-7 through LDS) before the
// epilogue.  Tiles, LDS layout and loads as in the four-wave schedule; each
// wave issues one load instruction per operand and step (j = wave).
constexpr int NT8 = 512;

struct Loader1 {  // K-contiguous operand, one load instruction per wave and step
  const float* zero;
  const float* fast;  // the lane's row (clamped into the matrix)
  int lk;             // its k offset inside a step
  bool valid;         // the row lies inside the matrix
  int K;

  __device__ void init(const Operand& op, const Gather& g, const float* zp, int64_t w, int o0, int on, int k,
                       int wave, int lane) {
    const float* base = reinterpret_cast<const float*>(op.ptr) + w * op.wstride;
    const int r = 8 * wave + lane / 8;
    const int o = o0 + r, oc = o < on ? o : on - 1;
    const int64_t t = op.gather ? gather_step(g) : 0;
    const int64_t ri = op.gather ? batch_row(w, t, g.mb, g.S, oc) : oc;
    zero = zp;
    K = k;
    valid = o < on;
    fast = base + ri * op.ld;
    lk = 4 * ((lane % 8) ^ kc_key(r));
  }
  __device__ const float* src_full(int k0) const { return fast + (k0 + lk); }
  __device__ const float* src(int k0) const {
    const int k = k0 + lk;
    return (valid && k < K) ? fast + k : zero;
  }
};

// this wave's half of a K step's fragments: slices 4*kh .. 4*kh+3, i.e. the
// lane's 16-byte chunk 2*lg + kh of its row
__device__ __forceinline__ void frag_half(const float* tile, int outer_off, int li, int lg, int kh, f32x4 (&f)[2]) {
#pragma unroll
  for (int b = 0; b < 2; ++b)
    f[b] = *reinterpret_cast<const f32x4*>(tile + 4 * kc_slot(outer_off + 16 * b + li, 2 * lg + kh));
}

struct FragsH {
  f32x4 a[2], b[2];
};

__device__ __forceinline__ void k_step8(int wave, int wm, int wn, int li, int lg, int kh, const FragsH& cur,
                                        FragsH& nxt, const float* rd, float* wr, const float* sa, const float* sb,
                                        f32x4 (&acc)[2][2]) {
  wait_lgkm0();
  wait_vm<2 * (NS - 2)>();
  barrier();
  frag_half(rd, wm * 32, li, lg, kh, nxt.a);
  frag_half(rd + TILE_F, wn * 32, li, lg, kh, nxt.b);
  const uint32_t wa = lds_off(wr) + 4 * 256 * wave;
  fire(sa, wa);
  fire(sb, wa + 4 * TILE_F);
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
        acc[bi][bj] = __builtin_amdgcn_mfma_f32_16x16x4f32(cur.a[bi][s], cur.b[bj][s], acc[bi][bj], 0, 0, 0);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
  }
}

template <int EPI>
__device__ __forceinline__ void tile_fwd8(const GemmArgs& g, const int logical, float* st0, float* st1, float* st2,
                                          float* st3) {
  static_assert(EPI == EPI_FWD_RELU || EPI == EPI_FWD_LINEAR, "forward products only");
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kh = wave >> 2, wm = (wave & 3) >> 1, wn = wave & 1, li = lane & 15, lg = lane >> 4;
  const TileCoord c = coord_of(g, logical);
  const int worker = c.worker, m0 = c.m0, n0 = c.n0;
  const int rbase = m0 + wm * 32, cbase = n0 + wn * 32;
  // accumulator (bi, bj, r) sits at row rbase + 16*bi + 4*lg + r, column
  // cbase + 16*bj + li; the bias of this lane's two columns first (clamped,
  // unconditional, oldest in the memory queue)
  float bpre[2];
#pragma unroll
  for (int bj = 0; bj < 2; ++bj) bpre[bj] = g.bias[(int64_t)worker * g.bstride + min(cbase + 16 * bj + li, g.N - 1)];

  Loader1 la, lb;
  la.init(g.a, g.g, g.zero, worker, m0, g.M, g.K, wave, lane);
  lb.init(g.b, g.g, g.zero, worker, n0, g.N, g.K, wave, lane);
  f32x4 acc[2][2];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (g.K + BKD - 1) / BKD;
  {
    float* stg[NS] = {st0, st1, st2, st3};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const uint32_t wa = lds_off(stg[s]) + 4 * 256 * wave;
      fire(la.src(s * BKD), wa);
      fire(lb.src(s * BKD), wa + 4 * TILE_F);
    }
  }
  wait_vm<2 * (NS - 1)>();
  barrier();
  FragsH f0, f1;
  frag_half(st0, wm * 32, li, lg, kh, f0.a);
  frag_half(st0 + TILE_F, wn * 32, li, lg, kh, f0.b);

  auto step = [&](auto full, const FragsH& cur, FragsH& nxt, const float* rd, float* wr, int kt) {
    const int k0 = (kt + NS) * BKD;
    if constexpr (decltype(full)::value)
      k_step8(wave, wm, wn, li, lg, kh, cur, nxt, rd, wr, la.src_full(k0), lb.src_full(k0), acc);
    else
      k_step8(wave, wm, wn, li, lg, kh, cur, nxt, rd, wr, la.src(k0), lb.src(k0), acc);
  };
  using Full = std::true_type;
  using Checked = std::false_type;
  const int nk4 = nk & ~3;
  const int nfast = (g.K / BKD - NS > 0 ? g.K / BKD - NS : 0) & ~3;  // steps kt whose step kt+NS is full
  int kt = 0;
  for (; kt < nfast && kt < nk4; kt += 4) {
    step(Full{}, f0, f1, st1, st0, kt);
    step(Full{}, f1, f0, st2, st1, kt + 1);
    step(Full{}, f0, f1, st3, st2, kt + 2);
    step(Full{}, f1, f0, st0, st3, kt + 3);
  }
  for (; kt < nk4; kt += 4) {
    step(Checked{}, f0, f1, st1, st0, kt);
    step(Checked{}, f1, f0, st2, st1, kt + 1);
    step(Checked{}, f0, f1, st3, st2, kt + 2);
    step(Checked{}, f1, f0, st0, st3, kt + 3);
  }
  if (nk4 < nk) step(Checked{}, f0, f1, st1, st0, nk4);
  if (nk4 + 1 < nk) step(Checked{}, f1, f0, st2, st1, nk4 + 1);
  if (nk4 + 2 < nk) step(Checked{}, f0, f1, st3, st2, nk4 + 2);
  // every load (also those of the steps past the end) has landed and every
  // wave is done reading the stages: waves 4-7 hand their sums over in LDS
  wait_vm<0>();
  wait_lgkm0();
  barrier();
  f32x4* xfer = reinterpret_cast<f32x4*>(st0) + ((wave & 3) * 64 + lane) * 4;
  if (kh == 1) {
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) xfer[2 * bi + bj] = acc[bi][bj];
  }
  __syncthreads();
  if (kh == 1) return;
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) acc[bi][bj] += xfer[2 * bi + bj];
  asm volatile("" ::"v"(bpre[0]), "v"(bpre[1]));
  float* out = reinterpret_cast<float*>(g.out) + (int64_t)worker * g.ostride;
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) {
        const int row = rbase + 16 * bi + 4 * lg + r, col = cbase + 16 * bj + li;
        if (row >= g.M || col >= g.N) continue;
        float z = acc[bi][bj][r] + bpre[bj];
        if (EPI == EPI_FWD_RELU) z = z > 0.f ? z : 0.f;
        out[(int64_t)row * g.ldo + col] = z;
      }
}

// ---------------------------------------------------------------------------
// Persistent schedule of the weight-gradient product
//   dW = dZ^T H (A = dZ [K][M] and B = H [K][N], both K-strided; for the
//   first layer H is the gathered data rows),
// fused with the SGD update of the weights (and the bias from the column
// sums of dZ): W_dst = W_src - eta*dW, on a round's last step
// (W_src - eta*dW - W_snap) / lambda.

// Tiles of workgroup `wg` of `nwg` (nwg a multiple of 8): workgroup wg runs
// on XCD wg % 8 (round-robin dispatch); each XCD owns one contiguous range of
// logical tiles (tiles of one worker share its dZ and H in that XCD's L2),
// walked by its nwg/8 workgroups with stride nwg/8.
struct TileList {
  int first, stride, count;
  __device__ int logical(int i) const { return first + i * stride; }
};

__device__ __forceinline__ TileList tiles_of_wg(int T, int wg, int nwg) {
  const int xcd = wg % kNumXcd, slot = wg / kNumXcd, per = nwg / kNumXcd;
  const int q = (T + kNumXcd - 1) / kNumXcd;
  const int lo = xcd * q, hi = min(T, lo + q);
  TileList t;
  t.first = lo + slot;
  t.stride = per;
  t.count = t.first < hi ? (hi - t.first + per - 1) / per : 0;
  return t;
}

// Per-lane part of the K-strided operand loads of the weight-gradient tiles.
struct DwLoads {
  const float* a_base;   // dZ of worker 0
  const float* b_base;   // H of worker 0 (gathered: the data set)
  const float* zero;
  int64_t a_ld, a_ws, b_ld, b_ws;
  int M, N, K, b_gather;
  int64_t S, tb;         // gathered rows: worker*S + (tb + k) mod S
  int kl[2], cc[2];      // the lane's k row and column chunk in its two instructions
  // current issue-side tile
  int64_t a_off, b_off;  // worker offsets
  int m0, n0, worker;
  bool live;
  // Sources of the tile's steps that lie inside K, at k0 = 0: the lane's k
  // row and column chunk (clamped into the matrix: columns past the edge
  // feed only outputs that are never stored); usable when the tile is live
  // and its gathered rows do not wrap around the shard's end
  const float* fa[2];
  const float* fb[2];
  bool fast;

  __device__ void set_tile(const GemmArgs& g, const TileList& tl, int i) {
    live = i < tl.count;
    const TileCoord c = coord_of(g, live ? tl.logical(i) : 0);
    worker = c.worker;
    m0 = c.m0;
    n0 = c.n0;
    a_off = (int64_t)worker * a_ws;
    b_off = (int64_t)worker * b_ws;
    fast = live && (!b_gather || tb + K <= S);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int oa = m0 + 4 * cc[u], ob = n0 + 4 * cc[u];  // (M, N multiples of 4)
      fa[u] = a_base + a_off + (int64_t)kl[u] * a_ld + (oa < M ? oa : M - 4);
      const int64_t rb = b_gather ? (int64_t)worker * S + tb + kl[u] : (int64_t)kl[u];
      fb[u] = b_base + b_off + rb * b_ld + (ob < N ? ob : N - 4);
    }
  }
  __device__ const float* a_full(int k0, int u) const { return fa[u] + (int64_t)k0 * a_ld; }
  __device__ const float* b_full(int k0, int u) const { return fb[u] + (int64_t)k0 * b_ld; }
  __device__ const float* a_src(int k0, int u) const {
    const int kk = k0 + kl[u], o = m0 + 4 * cc[u];
    if (!live || kk >= K || o >= M) return zero;
    return a_base + a_off + (int64_t)kk * a_ld + o;
  }
  __device__ const float* b_src(int k0, int u) const {
    const int kk = k0 + kl[u], o = n0 + 4 * cc[u];
    if (!live || kk >= K || o >= N) return zero;
    int64_t row = kk;
    if (b_gather) {
      const int64_t x = tb + kk;
      row = (int64_t)worker * S + (x >= S ? x - S : x);
    }
    return b_base + b_off + row * b_ld + o;
  }
};

// Epilogue operands of tile `c`: W_src into LDS (rows m0.., columns n0..,
// row-major 64 x 64; this wave: rows 4j .. 4j+3 for j = 4*wave .. 4*wave+3,
// lane l row 4j + l/16, columns 4*(l%16) .. +3), and on a round's last step
// the lane's own W_snap pairs straight into registers (rows and columns as
// its accumulators; clamped into the matrix, never stored outside it).  The
// snapshot's loads are ordinary loads, so the compiler waits for them where
// the epilogue reads them; in LDS it would take a second tile buffer, and
// with it the second workgroup of each CU.
template <bool LAST, bool ADAM>
__device__ __forceinline__ void fire_epi(const GemmArgs& g, const TileCoord& c, float* epi, float2 (&snap)[2][4],
                                         const Lanes& q) {
  const int64_t wo = (int64_t)c.worker * g.pstride;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int j = 4 * q.wave + u;
    const int row = c.m0 + 4 * j + q.lane / 16, col = c.n0 + 4 * (q.lane % 16);
    const bool ok = row < g.M && col < g.N;
    const int64_t e = wo + (int64_t)row * g.ldw + col;
    fire(ok ? g.w_src + e : g.zero, lds_off(epi) + 4 * 256 * j);
    if constexpr (ADAM) {
      // the Adam moments of the same block, in the two tiles after it
      fire(ok ? g.adam.mw + e : g.zero, lds_off(epi) + 4 * (EPI_F + 256 * j));
      fire(ok ? g.adam.vw + e : g.zero, lds_off(epi) + 4 * (2 * EPI_F + 256 * j));
    }
  }
  if constexpr (ADAM) {
    // the bias moments of rows m0 .. m0 + 63 (lanes 0..15; every wave loads
    // the same values, so that each issues the same number of loads)
    const int row = c.m0 + 4 * q.lane;
    const bool ok = q.lane < 16 && row < g.M;
    fire(ok ? g.adam.mb + wo + row : g.zero, lds_off(epi) + 4 * 3 * EPI_F);
    fire(ok ? g.adam.vb + wo + row : g.zero, lds_off(epi) + 4 * (3 * EPI_F + 256));
  }
  if constexpr (LAST) {
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = min(c.m0 + q.wm * 32 + 2 * (4 * q.lg + r) + bi, g.M - 1);
        const int col = min(c.n0 + q.wn * 32 + 2 * q.li, g.N - 2);  // (N even)
        snap[bi][r] = *reinterpret_cast<const float2*>(g.w_snap + wo + (int64_t)row * g.ldw + col);
      }
  }
}

// ADAM: Adam as the local rule; epi then holds W_src, the two moment tiles
// and the bias moments (EPI_ADAM_F floats)
template <bool LAST, bool ADAM>
__device__ __forceinline__ void dw_tiles(const GemmArgs& g, const TileList tl, float* st0, float* st1, float* st2,
                                         float* st3, float* epi) {
  // epilogue load instructions per wave and tile
  constexpr int EPN = 4 + (LAST ? 8 : 0) + (ADAM ? 10 : 0);
  if (tl.count == 0) return;
  const int tid = threadIdx.x;
  const Lanes q{tid >> 6, tid & 63, (tid >> 6) >> 1, (tid >> 6) & 1, tid & 15, (tid & 63) >> 4};
  const int nk = (g.K + BKD - 1) / BKD;  // a multiple of NS (checked on the host)

  DwLoads ld;
  ld.a_base = reinterpret_cast<const float*>(g.a.ptr);
  ld.b_base = reinterpret_cast<const float*>(g.b.ptr);
  ld.zero = g.zero;
  ld.a_ld = g.a.ld;
  ld.a_ws = g.a.wstride;
  ld.b_ld = g.b.ld;
  ld.b_ws = g.b.wstride;
  ld.M = g.M;
  ld.N = g.N;
  ld.K = g.K;
  ld.b_gather = g.b.gather;
  ld.S = g.g.S;
  ld.tb = g.b.gather ? (gather_step(g.g) * g.g.mb) % g.g.S : 0;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    ld.kl[u] = ks_row(2 * q.wave + u, q.lane);
    ld.cc[u] = ks_chunk(2 * q.wave + u, q.lane);
  }

  // prologue: steps 0..NS-1 (all in tile 0, since nk >= NS), then the
  // epilogue operands of tile 0
  ld.set_tile(g, tl, 0);
  {
    float* stg[NS] = {st0, st1, st2, st3};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const uint32_t wa = lds_off(stg[s]) + 4 * 256 * (2 * q.wave);
      fire(ld.a_src(s * BKD, 0), wa);
      fire(ld.a_src(s * BKD, 1), wa + 4 * 256);
      fire(ld.b_src(s * BKD, 0), wa + 4 * TILE_F);
      fire(ld.b_src(s * BKD, 1), wa + 4 * (TILE_F + 256));
    }
  }
  float2 snap[2][4];
  fire_epi<LAST, ADAM>(g, coord_of(g, tl.logical(0)), epi, snap, q);
  const AdamCoef ac = ADAM ? adam_coef(g.g, g.adam) : AdamCoef{1.f, 1.f};
  wait_vm<4 * (NS - 1) + EPN>();
  barrier();
  Frags f0, f1;
  read_frags<false, false>(st0, q.wm, q.wn, q.li, q.lg, f0);

  float bsum[2] = {0.f, 0.f};
  f32x4 acc[2][2];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};

  // the issue side runs NS steps ahead of the compute side: tile i2, step kt2
  int i2 = 0, kt2 = NS;
  if (kt2 >= nk) {  // (nk == NS)
    kt2 -= nk;
    ++i2;
    ld.set_tile(g, tl, i2);
  }

  // one K step: wait for the fragments of the next step, read them, issue
  // the loads NS steps ahead, run this step's MFMAs
  auto step = [&](auto vm, const Frags& cur, Frags& nxt, const float* rd, float* wr) {
    const int k0 = kt2 * BKD;
    const float* src[4];
    if (ld.fast && k0 + BKD <= g.K) {  // (uniform) every load of the step inside K
      src[0] = ld.a_full(k0, 0);
      src[1] = ld.a_full(k0, 1);
      src[2] = ld.b_full(k0, 0);
      src[3] = ld.b_full(k0, 1);
    } else {
      src[0] = ld.a_src(k0, 0);
      src[1] = ld.a_src(k0, 1);
      src[2] = ld.b_src(k0, 0);
      src[3] = ld.b_src(k0, 1);
    }
    k_step<false, false, decltype(vm)::value>(q, cur, nxt, rd, wr, src, acc, bsum);
    if (++kt2 == nk) {
      kt2 = 0;
      ld.set_tile(g, tl, ++i2);
    }
  };
  // the epilogue loads of a tile were issued after the step loads up to
  // its step NS-1: until then they sit behind the next step's loads
  using VM_E = std::integral_constant<int, 4 * (NS - 2) + EPN>;
  using VM_0 = std::integral_constant<int, 4 * (NS - 2)>;

  for (int i = 0; i < tl.count; ++i) {
    // K steps of tile i (nk a multiple of 4: step kt uses stage kt % 4 and
    // fragment set kt % 2)
    step(VM_E{}, f0, f1, st1, st0);
    step(VM_E{}, f1, f0, st2, st1);
    step(VM_E{}, f0, f1, st3, st2);
    step(VM_0{}, f1, f0, st0, st3);
    for (int kt = 4; kt < nk; kt += 4) {
      step(VM_0{}, f0, f1, st1, st0);
      step(VM_0{}, f1, f0, st2, st1);
      step(VM_0{}, f0, f1, st3, st2);
      step(VM_0{}, f1, f0, st0, st3);
    }
    // ---- epilogue of tile i (its operands in LDS since step NS-1)
    const TileCoord c = coord_of(g, tl.logical(i));
    const int64_t wo = (int64_t)c.worker * g.pstride;
    // lane holds rows tr = wm*32 + 2*(4*lg + r) + bi, column pairs
    // tc = wn*32 + 2*li + (0, 1)
    float2 nw[2][4];
    float2 mom[2][4][2];  // Adam: the updated moments (m, v)
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int tr = q.wm * 32 + 2 * (4 * q.lg + r) + bi, tc = q.wn * 32 + 2 * q.li;
        const float2 ws = *reinterpret_cast<const float2*>(epi + tr * TM + tc);
        float dx = acc[bi][0][r], dy = acc[bi][1][r];
        if constexpr (ADAM) {
          float2 mm = *reinterpret_cast<const float2*>(epi + EPI_F + tr * TM + tc);
          float2 vv = *reinterpret_cast<const float2*>(epi + 2 * EPI_F + tr * TM + tc);
          dx = adam_moments(dx, mm.x, vv.x, g.adam, ac);
          dy = adam_moments(dy, mm.y, vv.y, g.adam, ac);
          mom[bi][r][0] = mm;
          mom[bi][r][1] = vv;
        }
        float2 v{ws.x - g.eta * dx, ws.y - g.eta * dy};
        if (LAST) {
          v.x = (v.x - snap[bi][r].x) / g.lam;
          v.y = (v.y - snap[bi][r].y) / g.lam;
        }
        nw[bi][r] = v;
      }
    const bool full = c.m0 + TM <= g.M && c.n0 + TM <= g.N;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = c.m0 + q.wm * 32 + 2 * (4 * q.lg + r) + bi, col = c.n0 + q.wn * 32 + 2 * q.li;
        // streaming stores for the updated weights (read again only by the
        // next local step's products); the last step's deltas are cached,
        // the commit reads them next
        f32x2* dst = reinterpret_cast<f32x2*>(g.w_dst + wo + (int64_t)row * g.ldw + col);
        const f32x2 v = {nw[bi][r].x, nw[bi][r].y};
        if (full || (row < g.M && col < g.N)) {  // (N even: col+1 < N too)
          if (LAST)
            *dst = v;
          else
            __builtin_nontemporal_store(v, dst);
          if constexpr (ADAM) {
            const int64_t e = wo + (int64_t)row * g.ldw + col;
            __builtin_nontemporal_store(f32x2{mom[bi][r][0].x, mom[bi][r][0].y}, reinterpret_cast<f32x2*>(g.adam.mw + e));
            __builtin_nontemporal_store(f32x2{mom[bi][r][1].x, mom[bi][r][1].y}, reinterpret_cast<f32x2*>(g.adam.vw + e));
          }
        }
      }
    if (c.tile_n == 0 && q.wn == 0) {
      // lane groups 1..3 hold partial sums of the same columns as group 0:
      // add them in a fixed order
      float tot[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const float p1 = __shfl(bsum[b], q.li + 16), p2 = __shfl(bsum[b], q.li + 32),
                    p3 = __shfl(bsum[b], q.li + 48);
        tot[b] = ((bsum[b] + p1) + p2) + p3;
      }
      if (q.lg == 0) {
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int o = c.m0 + q.wm * 32 + 2 * q.li + b;
          if (o < g.M) {
            const int64_t e = wo + o;
            float stp = tot[b];
            if constexpr (ADAM) {
              float mb = epi[3 * EPI_F + (o - c.m0)], vb = epi[3 * EPI_F + 256 + (o - c.m0)];
              stp = adam_moments(stp, mb, vb, g.adam, ac);
              g.adam.mb[e] = mb;
              g.adam.vb[e] = vb;
            }
            const float nb = g.b_src[e] - g.eta * stp;
            g.b_dst[e] = LAST ? (nb - g.b_snap[e]) / g.lam : nb;
          }
        }
      }
    }
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};
    bsum[0] = bsum[1] = 0.f;
    if (i + 1 < tl.count) {
      // every wave has read this tile's epilogue operands: load the next's
      wait_lgkm0();
      barrier();
      fire_epi<LAST, ADAM>(g, coord_of(g, tl.logical(i + 1)), epi, snap, q);
    }
  }
  // loads of the steps past the end (zero page) still write LDS
  wait_vm<0>();
}

// four LDS stages as separate objects, so that the compiler can tell the
// loads into one stage from the fragment reads of another
#define DL_STAGES                                                \
  __shared__ __attribute__((aligned(16))) float st0[STAGE_F];     \
  __shared__ __attribute__((aligned(16))) float st1[STAGE_F];     \
  __shared__ __attribute__((aligned(16))) float st2[STAGE_F];     \
  __shared__ __attribute__((aligned(16))) float st3[STAGE_F];
#define DL_EPI __shared__ __attribute__((aligned(16))) float epi[ADAM ? EPI_ADAM_F : EPI_F];

// forward products, eight waves splitting each K step
template <int EPI>
__global__ __launch_bounds__(NT8) void gemm_f32_dl_fwd8_kernel(GemmArgs g) {
  DL_STAGES
  tile_fwd8<EPI>(g, xcd_remap(blockIdx.x, tiles_dl(g)), st0, st1, st2, st3);
}

template <bool A_KC, bool B_KC, int EPI>
__global__ __launch_bounds__(NT) void gemm_f32_dl_kernel(GemmArgs g) {
  DL_STAGES
  tile_dl<A_KC, B_KC, EPI>(g, xcd_remap(blockIdx.x, tiles_dl(g)), st0, st1, st2, st3);
}

// Rank of workgroup `wg` of `nwg` by its number of weight-gradient tiles
// (tiles_of_wg: the high slots of each XCD hold one tile fewer): rank 0 is
// the last slot of XCD 0, then the last slot of XCD 1, ...  A bijection on
// [0, nwg).
__device__ __forceinline__ int fewest_tiles_rank(int wg, int nwg) {
  const int per = nwg / kNumXcd;
  return (per - 1 - wg / kNumXcd) * kNumXcd + wg % kNumXcd;
}

// The first layer's weight gradient; with HCM > 0 (the class bound of the
// fused output layer) also the output layer's weight-gradient units, which
// neither read nor write what the first layer's tiles do: unit u goes to
// the workgroup of rank u mod nwg, before its tiles (the stage buffers are
// free then, and these workgroups hold a tile fewer).
template <bool LAST, int HCM, bool ADAM>
__global__ __launch_bounds__(NT) void gemm_f32_dl_dw_kernel(GemmArgs g, HeadDwArgs h) {
  DL_STAGES
  DL_EPI
  if constexpr (HCM > 0) {
    static_assert(hdw_smem_floats<HCM>() <= STAGE_F, "an output-layer unit fits one stage buffer");
    const int units = hdw_units(h);
    bool ran = false;
    for (int u = fewest_tiles_rank(blockIdx.x, gridDim.x); u < units; u += gridDim.x) {
      if (ran) __syncthreads();  // the previous unit's LDS reads are done
      head_dw_unit<HCM>(h, u, st0);
      ran = true;
    }
    if (ran) __syncthreads();    // before the tiles' loads land in the stages
  }
  dw_tiles<LAST, ADAM>(g, tiles_of_wg(tiles_dl(g), blockIdx.x, gridDim.x), st0, st1, st2, st3, epi);
}

// Weight-gradient tiles of workgroup `pid` in the combined backward launch
// (workgroups [0, n1pad) start with an input-gradient tile, the rest are
// weight-gradient only; workgroup pid runs on XCD pid % 8).  Each XCD owns a
// contiguous range of logical tiles (one worker's dZ and H share its L2),
// handed out in contiguous runs: cb tiles to each of its weight-gradient-only
// workgroups, then ca to each of its input-gradient workgroups, so that both
// kinds finish together.
__device__ __forceinline__ TileList split_tiles(int T, int pid, int n1pad, int ca, int cb) {
  const int xcd = pid % kNumXcd, q = (T + kNumXcd - 1) / kNumXcd;
  const int lo = xcd * q, hi = min(T, lo + q);
  const int nb = ((int)gridDim.x - n1pad) / kNumXcd;
  const int first = pid >= n1pad ? lo + ((pid - n1pad) / kNumXcd) * cb : lo + nb * cb + (pid / kNumXcd) * ca;
  const int n = pid >= n1pad ? cb : ca;
  TileList t;
  t.first = first;
  t.stride = 1;
  t.count = max(0, min(hi, first + n) - first);
  return t;
}

// input-gradient tiles (one per workgroup, spread evenly over the XCDs),
// and the weight-gradient tiles of the same layer on every workgroup
template <bool LAST, bool ADAM>
__global__ __launch_bounds__(NT) void gemm_f32_dl_bwd_kernel(GemmArgs dx, GemmArgs dw, int n1, int n1pad, int ca,
                                                             int cb) {
  DL_STAGES
  DL_EPI
  const int pid = blockIdx.x;
  if (pid < n1) {
    tile_dl<true, false, EPI_DX_MASK>(dx, xcd_remap(pid, n1), st0, st1, st2, st3);
    // every wave is done with the stages before the weight-gradient tiles load into them
    wait_lgkm0();
    barrier();
  }
  dw_tiles<LAST, ADAM>(dw, split_tiles(tiles_dl(dw), pid, n1pad, ca, cb), st0, st1, st2, st3, epi);
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// the operand can be staged with 16-byte direct loads
bool operand_ok(const Operand& op, bool kc, int outer_n, int K) {
  if (!op.vec || !aligned16(op.ptr) || op.ld % 4 || op.wstride % 4 || K % 4) return false;
  return kc || (outer_n % 4 == 0 && !op.gather);
}

// weight-gradient product: K-strided operands (B may be gathered when the
// batch fits in a shard), a multiple of NS K steps, 16-byte epilogue rows
bool dw_ok(const GemmArgs& g) {
  if (g.epi != EPI_DW_UPDATE || !g.zero) return false;
  if (g.adam.on && (!aligned16(g.adam.mw) || !aligned16(g.adam.vw) || !aligned16(g.adam.mb) || !aligned16(g.adam.vb)))
    return false;
  const Operand& a = g.a;
  const Operand& b = g.b;
  if (!a.vec || !b.vec || a.gather || !aligned16(a.ptr) || !aligned16(b.ptr)) return false;
  if (a.ld % 4 || a.wstride % 4 || b.ld % 4 || b.wstride % 4) return false;
  if (g.M % 4 || g.N % 4 || ((g.K + BKD - 1) / BKD) % NS) return false;
  if (b.gather && g.K > g.g.S) return false;
  if (!aligned16(g.w_src) || !aligned16(g.w_dst) || g.ldw % 4 || g.pstride % 4) return false;
  return !g.last || aligned16(g.w_snap);
}

int dw_grid(const GemmArgs& g) {
  const int t = (tiles_dl(g) + kNumXcd - 1) / kNumXcd * kNumXcd, cap = g.adam.on ? NWG_DW_ADAM : NWG_DW;
  return t < cap ? t : cap;
}

}  // namespace

bool gemm_f32_dl_ok(int a_kc, int b_kc, const GemmArgs& g) {
  if (!a_kc && !b_kc) return dw_ok(g);
  return g.zero && a_kc && (g.epi == EPI_DX_MASK ? !b_kc : b_kc) && operand_ok(g.a, true, g.M, g.K) &&
         operand_ok(g.b, b_kc, g.N, g.K);
}

hipError_t launch_gemm_f32_dl(int a_kc, int b_kc, const GemmArgs& g, hipStream_t s) {
  const dim3 grid(tiles_dl(g)), block(NT);
  if (a_kc && b_kc && g.epi == EPI_FWD_RELU)
    AGN_LAUNCH((gemm_f32_dl_fwd8_kernel<EPI_FWD_RELU>), grid, dim3(NT8), 0, s, g);
  else if (a_kc && b_kc && g.epi == EPI_FWD_LINEAR)
    AGN_LAUNCH((gemm_f32_dl_fwd8_kernel<EPI_FWD_LINEAR>), grid, dim3(NT8), 0, s, g);
  else if (a_kc && !b_kc && g.epi == EPI_DX_MASK)
    AGN_LAUNCH((gemm_f32_dl_kernel<true, false, EPI_DX_MASK>), grid, block, 0, s, g);
  else if (!a_kc && !b_kc && g.epi == EPI_DW_UPDATE) {
    const HeadDwArgs none{};
    if (g.adam.on) {
      if (g.last)
        AGN_LAUNCH((gemm_f32_dl_dw_kernel<true, 0, true>), dim3(dw_grid(g)), block, 0, s, g, none);
      else
        AGN_LAUNCH((gemm_f32_dl_dw_kernel<false, 0, true>), dim3(dw_grid(g)), block, 0, s, g, none);
    } else if (g.last) {
      AGN_LAUNCH((gemm_f32_dl_dw_kernel<true, 0, false>), dim3(dw_grid(g)), block, 0, s, g, none);
    } else {
      AGN_LAUNCH((gemm_f32_dl_dw_kernel<false, 0, false>), dim3(dw_grid(g)), block, 0, s, g, none);
    }
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

bool gemm_f32_dl_dw_head_ok(const GemmArgs& g, const HeadDwArgs& h) {
  return dw_ok(g) && h.C >= 1 && h.C <= 10 && h.n >= 1 && h.d >= 1;
}

hipError_t launch_gemm_f32_dl_dw_head(const GemmArgs& g, const HeadDwArgs& h, hipStream_t s) {
  if (!gemm_f32_dl_dw_head_ok(g, h)) return hipErrorInvalidValue;
  if (g.adam.on) {
    if (g.last)
      AGN_LAUNCH((gemm_f32_dl_dw_kernel<true, 10, true>), dim3(dw_grid(g)), dim3(NT), 0, s, g, h);
    else
      AGN_LAUNCH((gemm_f32_dl_dw_kernel<false, 10, true>), dim3(dw_grid(g)), dim3(NT), 0, s, g, h);
  } else if (g.last) {
    AGN_LAUNCH((gemm_f32_dl_dw_kernel<true, 10, false>), dim3(dw_grid(g)), dim3(NT), 0, s, g, h);
  } else {
    AGN_LAUNCH((gemm_f32_dl_dw_kernel<false, 10, false>), dim3(dw_grid(g)), dim3(NT), 0, s, g, h);
  }
  return hipGetLastError();
}

hipError_t launch_gemm_f32_dl_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s) {
  const int n1 = tiles_dl(dx), n1pad = (n1 + kNumXcd - 1) / kNumXcd * kNumXcd;
  // as many persistent weight-gradient workgroups as input-gradient tiles
  // (an input-gradient tile of a 1000-wide layer carries the MFMA work of
  // eight weight-gradient tiles), at least 8 and at most one per
  // weight-gradient tile
  const int cap = dw.adam.on ? NWG_DW_ADAM : NWG_DW;
  int n2 = n1pad < cap ? n1pad : cap;
  const int t2 = dw_grid(dw);
  if (n2 > t2) n2 = t2;
  if (n2 < kNumXcd) n2 = kNumXcd;
  // Split each XCD's q weight-gradient tiles so that an input-gradient
  // workgroup (nkx K steps, then ca tiles) and a weight-gradient-only one
  // (cb tiles) take about the same time.  A weight-gradient tile costs about
  // three times its NS K steps (its epilogue reads and writes a 64 x 64
  // block of weights; measured on 8 x 1000 x 1000 x 128: the split 3 / 5
  // beats 1 / 7 and 4 / 4 by 4 % of the round)
  const int q = (tiles_dl(dw) + kNumXcd - 1) / kNumXcd, a = n1pad / kNumXcd, b = n2 / kNumXcd;
  const double u = 3.0 * NS, nkx = (dx.K + BKD - 1) / BKD;
  int ca = (int)std::floor((q - b * nkx / u) / (a + b) + 0.5);
  if (ca < 0) ca = 0;
  if (ca * a > q) ca = q / a;
  const int cb = (q - ca * a + b - 1) / b;
  const dim3 grid(n1pad + n2), block(NT);
  if (dw.adam.on) {
    if (dw.last)
      AGN_LAUNCH((gemm_f32_dl_bwd_kernel<true, true>), grid, block, 0, s, dx, dw, n1, n1pad, ca, cb);
    else
      AGN_LAUNCH((gemm_f32_dl_bwd_kernel<false, true>), grid, block, 0, s, dx, dw, n1, n1pad, ca, cb);
  } else if (dw.last) {
    AGN_LAUNCH((gemm_f32_dl_bwd_kernel<true, false>), grid, block, 0, s, dx, dw, n1, n1pad, ca, cb);
  } else {
    AGN_LAUNCH((gemm_f32_dl_bwd_kernel<false, false>), grid, block, 0, s, dx, dw, n1, n1pad, ca, cb);
  }
  return hipGetLastError();
}

}  // namespace agn
