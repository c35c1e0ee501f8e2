// Batched float32 products with direct global->LDS operand loads
// (global_load_lds_dwordx4 on gfx950): operand tiles travel from memory into
// LDS without passing through registers, two K steps ahead of their use, and
// the fragments of the next K step are read from LDS while the MFMAs of the
// current one run.
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
//     chunk (r, q) at r*8 + (q ^ ((r>>1)&7)), so the 16 rows that one
//     16-byte read touches per cycle cover all 64 banks once;
//   K-strided (rows = k, 16 chunks of 4 outer per row):
//     chunk (k, c) at k*16 + (c ^ (8*((k>>3)&1))), so rows k and k+8, read
//     together by lane groups 0 and 1, land in opposite halves of the banks.
// Each lane loads the global 16 bytes that belong in its slot; lanes past an
// edge read a zero page, so edge tiles hold exact zeros.
#include "device_common.h"

namespace agn {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int NT = 256, TM = 64, BKD = 32;
constexpr int TILE_F = TM * BKD;                 // floats per operand tile
constexpr int STAGE_F = 2 * TILE_F;              // A and B
constexpr int GTAB = 1024;                       // gathered K-strided rows: offset table

__device__ __forceinline__ int kc_slot(int r, int q) { return r * 8 + (q ^ ((r >> 1) & 7)); }
__device__ __forceinline__ int ks_slot(int k, int c) { return k * 16 + (c ^ (((k >> 3) & 1) << 3)); }

// vmcnt(n) without waiting on the other counters (gfx9 encoding)
#define WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 0xF) | ((((n) >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8))
// lgkmcnt(0) alone
#define WAIT_LGKM0() __builtin_amdgcn_s_waitcnt(0xC07F)

// One operand's tile loads: this wave issues slots [64j, 64j+64) for
// j = 2*wave and 2*wave+1 (two load instructions per operand per K step).
template <bool KC>
struct DirectLoader {
  const float* base;
  const float* zero;
  int64_t ld;
  int outer0, outer_n, K;
  const float* rowp[2];      // KC: the lane's two rows (null past the edge)
  const int64_t* tab;        // KS gathered: row offsets (elements) in LDS, or null
  int gather;
  int64_t worker, t, mb, S;

  __device__ void init(const Operand& op, const Gather& g, const float* zp, int64_t w, int o0, int on, int k,
                       int wave, int lane, const int64_t* table) {
    base = reinterpret_cast<const float*>(op.ptr) + w * op.wstride;
    zero = zp;
    ld = op.ld;
    outer0 = o0;
    outer_n = on;
    K = k;
    gather = op.gather;
    worker = w;
    mb = g.mb;
    S = g.S;
    t = gather ? gather_step(g) : 0;
    tab = table;
    if (KC) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int r = 8 * (2 * wave + u) + lane / 8;
        const int o = o0 + r;
        int64_t ri = o;
        if (gather && o < on) ri = batch_row(worker, t, mb, S, o);
        rowp[u] = o < on ? base + ri * ld : nullptr;
      }
    }
  }

  __device__ void issue(int k0, float* stage_tile, int wave, int lane) const {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int j = 2 * wave + u;
      const float* src;
      if (KC) {
        const int r = 8 * j + lane / 8;
        const int q = (lane % 8) ^ ((r >> 1) & 7);
        const int k = k0 + 4 * q;
        src = (rowp[u] && k < K) ? rowp[u] + k : zero;
      } else {
        const int kl = 4 * j + lane / 16;
        const int c = (lane % 16) ^ (((kl >> 3) & 1) << 3);
        const int kk = k0 + kl, o = outer0 + 4 * c;
        if (kk < K && o < outer_n) {
          const int64_t roff = gather ? (tab ? tab[kk] : batch_row(worker, t, mb, S, kk) * ld) : (int64_t)kk * ld;
          src = base + roff + o;
        } else {
          src = zero;
        }
      }
      __builtin_amdgcn_global_load_lds(src, (lds_ptr_t)(stage_tile + 256 * j), 16, 0, 0);
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

__device__ __forceinline__ void mfmas(const Frags& f, f32x4 (&acc)[2][2]) {
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
        acc[bi][bj] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.a[bi][s], f.b[bj][s], acc[bi][bj], 0, 0, 0);
}

template <bool A_KC, bool B_KC>
struct Pipe {
  const DirectLoader<A_KC>* la;
  const DirectLoader<B_KC>* lb;
  int nk, wave, lane, wm, wn, li, lg;
  bool do_bias;
};

// K step kt: the fragments of step kt are in `cur`.  Wait until every wave
// has read them and the loads of step kt+1 have landed, read step kt+1's
// fragments from `rd` into `nxt`, start the loads of step kt+3 into `wr`
// (the stage step kt came from), then run step kt's MFMAs.
template <bool A_KC, bool B_KC>
__device__ __forceinline__ void k_step(const Pipe<A_KC, B_KC>& p, int kt, const Frags& cur, Frags& nxt,
                                       const float* rd, float* wr, f32x4 (&acc)[2][2], float (&bsum)[2]) {
  // (unconditional, so that `cur` counts as landed on every path into the
  // MFMAs and the compiler adds no wait of its own there)
  WAIT_LGKM0();
  if (kt + 1 < p.nk) {
    if (kt + 2 < p.nk)
      WAIT_VM(4);
    else
      WAIT_VM(0);
    __builtin_amdgcn_s_barrier();
    read_frags<A_KC, B_KC>(rd, p.wm, p.wn, p.li, p.lg, nxt);
    if (kt + 3 < p.nk) {
      p.la->issue((kt + 3) * BKD, wr, p.wave, p.lane);
      p.lb->issue((kt + 3) * BKD, wr + TILE_F, p.wave, p.lane);
    }
  }
  mfmas(cur, acc);
  if (p.do_bias) {  // A is dZ^T (K-strided): this lane's two columns over its 8 k
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      bsum[0] += cur.a[0][s];
      bsum[1] += cur.a[1][s];
    }
  }
}

// Tile row (column) of accumulator index x of block b.
template <bool KC>
__device__ __forceinline__ int tile_idx(int b, int x) { return KC ? 16 * b + x : 2 * x + b; }

template <bool A_KC, bool B_KC, int EPI>
__device__ __forceinline__ void tile_dl(const GemmArgs& g, const int logical, float* st0, float* st1, float* st2,
                                        int64_t* tab) {
  const int tid = threadIdx.x;
  const int tm = (g.M + TM - 1) / TM, tn = (g.N + TM - 1) / TM;
  const int worker = logical / (tm * tn);
  const int rem = logical % (tm * tn);
  const int tile_n = rem / tm, tile_m = rem % tm;
  const int m0 = tile_m * TM, n0 = tile_n * TM;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 15, lg = lane >> 4;
  const int64_t wo = (int64_t)worker * g.pstride;
  const int rbase = m0 + wm * 32, cbase = n0 + wn * 32;
  // accumulator (bi, bj, r) sits at row rbase + tile_idx<A_KC>(bi, 4*lg + r),
  // column cbase + tile_idx<B_KC>(bj, li)

  // operands of the epilogue first (oldest in the memory queue), so the K
  // loop's counted waits cover them
  float pre[2][2][4], pre2[2][2][4];
  if (EPI == EPI_DX_MASK || EPI == EPI_DW_UPDATE) {
    const float* mk = EPI == EPI_DX_MASK ? reinterpret_cast<const float*>(g.mask) + (int64_t)worker * g.mstride
                                         : nullptr;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) {
          const int row = rbase + tile_idx<A_KC>(bi, 4 * lg + r), col = cbase + tile_idx<B_KC>(bj, li);
          const bool ok = row < g.M && col < g.N;
          if (EPI == EPI_DX_MASK) {
            pre[bi][bj][r] = ok ? mk[(int64_t)row * g.ldm + col] : 0.f;
          } else {
            const int64_t e = wo + (int64_t)row * g.ldw + col;
            pre[bi][bj][r] = ok ? g.w_src[e] : 0.f;
            pre2[bi][bj][r] = (ok && g.last) ? g.w_snap[e] : 0.f;
          }
        }
  }

  // gathered K-strided operand (data rows of the first layer's weight
  // gradient): row offsets once per workgroup
  const bool tabA = !A_KC && g.a.gather && g.K <= GTAB, tabB = !B_KC && g.b.gather && g.K <= GTAB;
  if (tabA || tabB) {
    const Operand& op = tabA ? g.a : g.b;
    const int64_t ts = gather_step(g.g);
    for (int k = tid; k < g.K; k += NT) tab[k] = batch_row(worker, ts, g.g.mb, g.g.S, k) * op.ld;
    __syncthreads();
  }

  DirectLoader<A_KC> la;
  DirectLoader<B_KC> lb;
  la.init(g.a, g.g, g.zero, worker, m0, g.M, g.K, wave, lane, tabA ? tab : nullptr);
  lb.init(g.b, g.g, g.zero, worker, n0, g.N, g.K, wave, lane, tabB ? tab : nullptr);

  // bias gradient of the weight-gradient product: the waves of the first
  // column tile with wn = 0 sum their A fragments (A = dZ^T)
  const bool do_bias = (EPI == EPI_DW_UPDATE) && tile_n == 0 && wn == 0;
  float bsum[2] = {0.f, 0.f};
  f32x4 acc[2][2];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (g.K + BKD - 1) / BKD;
  // steps 0..2 in flight (4 load instructions per wave per step), then the
  // fragments of step 0
  la.issue(0, st0, wave, lane);
  lb.issue(0, st0 + TILE_F, wave, lane);
  if (nk > 1) {
    la.issue(BKD, st1, wave, lane);
    lb.issue(BKD, st1 + TILE_F, wave, lane);
  }
  if (nk > 2) {
    la.issue(2 * BKD, st2, wave, lane);
    lb.issue(2 * BKD, st2 + TILE_F, wave, lane);
    WAIT_VM(8);
  } else if (nk > 1) {
    WAIT_VM(4);
  } else {
    WAIT_VM(0);
  }
  __builtin_amdgcn_s_barrier();
  Frags f0, f1;
  read_frags<A_KC, B_KC>(st0, wm, wn, li, lg, f0);

  // stage of step kt: kt % 3; fragment set: kt % 2
  const Pipe<A_KC, B_KC> p{&la, &lb, nk, wave, lane, wm, wn, li, lg, do_bias};
  for (int kt = 0; kt < nk; kt += 6) {
    k_step(p, kt, f0, f1, st1, st0, acc, bsum);
    if (kt + 1 < nk) k_step(p, kt + 1, f1, f0, st2, st1, acc, bsum);
    if (kt + 2 < nk) k_step(p, kt + 2, f0, f1, st0, st2, acc, bsum);
    if (kt + 3 < nk) k_step(p, kt + 3, f1, f0, st1, st0, acc, bsum);
    if (kt + 4 < nk) k_step(p, kt + 4, f0, f1, st2, st1, acc, bsum);
    if (kt + 5 < nk) k_step(p, kt + 5, f1, f0, st0, st2, acc, bsum);
  }

  if (EPI == EPI_DW_UPDATE && do_bias) {
    // lane groups 1..3 hold partial sums of the same columns as group 0:
    // add them in a fixed order
    float tot[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const float p1 = __shfl(bsum[b], li + 16), p2 = __shfl(bsum[b], li + 32), p3 = __shfl(bsum[b], li + 48);
      tot[b] = ((bsum[b] + p1) + p2) + p3;
    }
    if (lg == 0) {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int o = rbase + 2 * li + b;
        if (o < g.M) {
          const int64_t e = wo + o;
          const float nb = g.b_src[e] - g.eta * tot[b];
          g.b_dst[e] = g.last ? (nb - g.b_snap[e]) / g.lam : nb;
        }
      }
    }
  }

#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) {
        const int row = rbase + tile_idx<A_KC>(bi, 4 * lg + r), col = cbase + tile_idx<B_KC>(bj, li);
        if (row >= g.M || col >= g.N) continue;
        const float v = acc[bi][bj][r];
        if (EPI == EPI_FWD_RELU || EPI == EPI_FWD_LINEAR) {
          float* out = reinterpret_cast<float*>(g.out) + (int64_t)worker * g.ostride;
          float z = v + g.bias[(int64_t)worker * g.bstride + col];
          if (EPI == EPI_FWD_RELU) z = z > 0.f ? z : 0.f;
          out[(int64_t)row * g.ldo + col] = z;
        } else if (EPI == EPI_DX_MASK) {
          float* out = reinterpret_cast<float*>(g.out) + (int64_t)worker * g.ostride;
          out[(int64_t)row * g.ldo + col] = pre[bi][bj][r] > 0.f ? v : 0.f;
        } else {  // EPI_DW_UPDATE: rows are output units o, columns input units i
          const int64_t e = wo + (int64_t)row * g.ldw + col;
          const float nw = pre[bi][bj][r] - g.eta * v;
          g.w_dst[e] = g.last ? (nw - pre2[bi][bj][r]) / g.lam : nw;
        }
      }
}

__host__ __device__ inline int tiles_dl(const GemmArgs& g) { return ((g.M + TM - 1) / TM) * ((g.N + TM - 1) / TM) * g.batch; }

// three LDS stages as separate objects, so that the compiler can tell the
// loads into one stage from the fragment reads of another
#define DL_LDS                                                   \
  __shared__ __attribute__((aligned(16))) float st0[STAGE_F];     \
  __shared__ __attribute__((aligned(16))) float st1[STAGE_F];     \
  __shared__ __attribute__((aligned(16))) float st2[STAGE_F];     \
  __shared__ __attribute__((aligned(16))) int64_t tab[GTAB];

template <bool A_KC, bool B_KC, int EPI>
__global__ __launch_bounds__(NT) void gemm_f32_dl_kernel(GemmArgs g) {
  DL_LDS
  tile_dl<A_KC, B_KC, EPI>(g, xcd_remap(blockIdx.x, tiles_dl(g)), st0, st1, st2, tab);
}

// input-gradient tiles, then weight-gradient tiles of one layer (see the
// register-staged kernel for the layout over the XCDs)
__global__ __launch_bounds__(NT) void gemm_f32_dl_bwd_kernel(GemmArgs dx, GemmArgs dw, int n1, int n1pad) {
  DL_LDS
  const int pid = blockIdx.x;
  if (pid < n1pad) {
    if (pid < n1) tile_dl<true, false, EPI_DX_MASK>(dx, xcd_remap(pid, n1), st0, st1, st2, tab);
  } else {
    tile_dl<false, false, EPI_DW_UPDATE>(dw, xcd_remap(pid - n1pad, tiles_dl(dw)), st0, st1, st2, tab);
  }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// the operand can be staged with 16-byte direct loads
bool operand_ok(const Operand& op, bool kc, int outer_n, int K) {
  if (!op.vec || !aligned16(op.ptr) || op.ld % 4 || op.wstride % 4 || K % 4) return false;
  return kc || outer_n % 4 == 0;
}

}  // namespace

bool gemm_f32_dl_ok(int a_kc, int b_kc, const GemmArgs& g) {
  return g.zero && operand_ok(g.a, a_kc, g.M, g.K) && operand_ok(g.b, b_kc, g.N, g.K);
}

hipError_t launch_gemm_f32_dl(int a_kc, int b_kc, const GemmArgs& g, hipStream_t s) {
  const dim3 grid(tiles_dl(g)), block(NT);
  if (a_kc && b_kc && g.epi == EPI_FWD_RELU)
    hipLaunchKernelGGL((gemm_f32_dl_kernel<true, true, EPI_FWD_RELU>), grid, block, 0, s, g);
  else if (a_kc && b_kc && g.epi == EPI_FWD_LINEAR)
    hipLaunchKernelGGL((gemm_f32_dl_kernel<true, true, EPI_FWD_LINEAR>), grid, block, 0, s, g);
  else if (a_kc && !b_kc && g.epi == EPI_DX_MASK)
    hipLaunchKernelGGL((gemm_f32_dl_kernel<true, false, EPI_DX_MASK>), grid, block, 0, s, g);
  else if (!a_kc && !b_kc && g.epi == EPI_DW_UPDATE)
    hipLaunchKernelGGL((gemm_f32_dl_kernel<false, false, EPI_DW_UPDATE>), grid, block, 0, s, g);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_gemm_f32_dl_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s) {
  const int n1 = tiles_dl(dx), n1pad = (n1 + kNumXcd - 1) / kNumXcd * kNumXcd;
  hipLaunchKernelGGL(gemm_f32_dl_bwd_kernel, dim3(n1pad + tiles_dl(dw)), dim3(NT), 0, s, dx, dw, n1, n1pad);
  return hipGetLastError();
}

}  // namespace agn
