// Batched bf16 products (bf16 operands, float32 accumulation) with direct
// global->LDS operand loads (global_load_lds_dwordx4 on gfx950): operand
// tiles travel from memory into LDS without passing through registers,
// three K steps ahead of their use, and the fragments of the next K step
// are read from LDS while the MFMAs of the current one run.
//
// Tile: 128x128 outputs per workgroup of 4 waves; wave (wm, wn) owns a
// 64x64 quarter as 2x2 blocks of v_mfma_f32_32x32x16_bf16; K in steps of 32
// (two MFMA slices of 16).  In one MFMA, lane (li = l%32, lh = l/32)
// supplies A[i = li][k = 8*lh .. 8*lh+7] and B[k = 8*lh .. 8*lh+7][j = li],
// 16 bytes each; the accumulators are laid out as the shared epilogues
// expect.
//
// LDS layout of one operand tile (128 x 32 bf16 = 512 chunks of 16 bytes; a
// wave's load instruction fills 64 consecutive chunks, lane l chunk l):
//   K-contiguous (rows = outer index, 4 chunks of 8 k per row): chunk
//     (r, q) at 4r + (q ^ key(r)), key(r) = ((r >> 1) ^ (r >> 3)) & 3.  A
//     fragment is one 16-byte read; the rows of 8 consecutive lanes land in
//     8 distinct 16-byte bank groups modulo 128 bytes, those of 16
//     consecutive lanes in 16 distinct groups modulo 256 bytes.
//   K-strided (rows = k, 16 chunks of 8 outer per row): chunk (k, c) at
//     16k + (c ^ key(k)), key(k) = 0, 6, 12, 10 for k % 4 = 0, 1, 2, 3.  A
//     fragment is two transposing 8-byte reads (ds_read_b64_tr_b16), each
//     over four consecutive k rows; the key puts those rows in distinct
//     bank windows (32 bytes modulo 128, 64 bytes modulo 256).
// Each lane loads the global 16 bytes that belong in its slot.  Lanes past
// an edge read a zero page, so edge tiles hold exact zeros; chunks never
// straddle an edge (K of a K-contiguous operand and the outer size of a
// K-strided one are multiples of 8, checked on the host).
//
// One output tile per workgroup for all three products: forward (A = H or
// the gathered data rows, B = W, both K-contiguous), input gradient (A = dZ
// K-contiguous, B = W K-strided) and weight gradient (A = dZ^T and B = H,
// both K-strided; H may be the gathered data rows).  The epilogues go
// through LDS (16-byte row chunks of outputs, masks and master weights).
#include <type_traits>

#include "bf16_epilogue.h"
#include "direct_load.h"

namespace agn {
namespace {

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int BK = 32, NS = 4;       // k per step, LDS stages
constexpr int TILE_B = TB * BK * 2;  // bytes of one operand tile
constexpr int STAGE_B = 2 * TILE_B;  // A and B
constexpr int LDS_DL = NS * STAGE_B > EPI_BYTES ? NS * STAGE_B : EPI_BYTES;

__device__ __forceinline__ int kc_key(int r) { return ((r >> 1) ^ (r >> 3)) & 3; }
__device__ __forceinline__ int ks_key(int k) { return (0xAC60 >> (4 * (k & 3))) & 15; }
__device__ __forceinline__ int kc_byte(int r, int q) { return (4 * r + (q ^ kc_key(r))) * 16; }
__device__ __forceinline__ int ks_byte(int k, int c) { return (16 * k + (c ^ ks_key(k))) * 16; }

// Per-lane sources of one operand's two load instructions per K step
// (instruction j = 2*wave + u, u = 0, 1; lane l fills chunk 64j + l):
//   K-contiguous: row r = 16j + l/4 (rows may be gathered data-set rows),
//     k chunk (l%4) ^ key(r);
//   K-strided: k row 4j + l/16, column chunk (l%16) ^ key(k) (k rows may be
//     gathered data-set rows: batch index kk of worker w is row
//     w*S + (tb + kk) mod S, tb = t*m mod S, with K <= S).
template <bool KC>
struct Loader {
  const uint16_t* zero;
  const uint16_t* row[2];   // KC: the lane's row; KS: its column chunk at k row 0 (null past the edge)
  // steps whose loads all lie inside K ("full" steps) load from
  // fast[u] + offset(k0): the lane's row or column chunk clamped into the
  // matrix (rows and columns past the edge feed only outputs that are never
  // stored, so any data will do there)
  const uint16_t* fast[2];
  int lk[2];                // KC: the lane's k offset in a step; KS: its k row in a step
  int64_t ld, rbase, tb, S;
  int K, gather;
  bool full_ok;             // false: a gathered mini-batch wraps round the shard's end

  __device__ void init(const Operand& op, const Gather& g, const void* zp, int64_t w, int o0, int on, int k,
                       int wave, int lane) {
    const uint16_t* base = reinterpret_cast<const uint16_t*>(op.ptr) + w * op.wstride;
    zero = reinterpret_cast<const uint16_t*>(zp);
    ld = op.ld;
    K = k;
    gather = op.gather;
    if (KC) {
      const int64_t t = op.gather ? gather_step(g) : 0;
      rbase = tb = S = 0;
      full_ok = true;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int r = 16 * (2 * wave + u) + lane / 4;
        const int o = o0 + r, oc = o < on ? o : on - 1;
        const int64_t ri = op.gather ? batch_row(w, t, g.mb, g.S, oc) : oc;
        row[u] = o < on ? base + ri * ld : nullptr;
        fast[u] = base + ri * ld;
        lk[u] = 8 * ((lane % 4) ^ kc_key(r));
      }
    } else {
      S = g.S;
      tb = op.gather ? (gather_step(g) * g.mb) % g.S : 0;
      rbase = op.gather ? w * g.S : 0;
      full_ok = !op.gather || tb + K <= S;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int kr = 4 * (2 * wave + u) + lane / 16;
        const int o = o0 + 8 * ((lane % 16) ^ ks_key(kr));
        row[u] = o < on ? base + o : nullptr;
        fast[u] = base + (op.gather ? rbase + tb + kr : kr) * ld + (o < on ? o : on - 8);
        lk[u] = kr;
      }
    }
  }

  // source for a full step
  __device__ const uint16_t* src_full(int k0, int u) const {
    return KC ? fast[u] + (k0 + lk[u]) : fast[u] + (int64_t)k0 * ld;
  }

  // source of this lane's 16 bytes in load instruction u of the K step
  // starting at k0; the zero page past an edge (also for k0 >= K)
  __device__ const uint16_t* src(int k0, int u) const {
    const int kk = k0 + lk[u];
    if (!row[u] || kk >= K) return zero;
    if (KC) return row[u] + kk;
    int64_t r = kk;
    if (gather) {
      const int64_t x = tb + kk;
      r = rbase + (x >= S ? x - S : x);
    }
    return row[u] + r * ld;
  }
};

// Fragments of one wave for one K step: a[b][s] / b[b][s] is the operand of
// block b in slice s (k = 16s + 8*lh + 0..7 of the step).
struct Frags {
  bf16x8 a[2][2], b[2][2];
};

template <bool KC>
__device__ __forceinline__ void frag(const char* tile, int outer_off, int li, int lh, bf16x8 (&f)[2][2]) {
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      if (KC) {
        f[b][s] = *reinterpret_cast<const bf16x8*>(tile + kc_byte(outer_off + 32 * b + li, 2 * s + lh));
      } else {
        // read c covers k = 16s + 8lh + 4c + e: within each group of 16
        // lanes, lane i receives element e from the 4 bf16 at the address
        // that lane 4e + i/4 supplies, offset i%4; so lane j supplies row
        // 16s + 8lh + 4c + j/4 at column (block start) + 16*(li/16) + 4*(j%4),
        // j = li % 16, and lane i ends up with column (block start) + li
        const int col = outer_off + 32 * b + 16 * (li / 16) + 4 * (li % 4);
        bf16x4 h[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int k = 16 * s + 8 * lh + 4 * c + (li % 16) / 4;
          const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4*)(tile + ks_byte(k, col / 8) + 2 * (col % 8)));
          h[c] = __builtin_bit_cast(bf16x4, v);
        }
        f[b][s] = __builtin_shufflevector(h[0], h[1], 0, 1, 2, 3, 4, 5, 6, 7);
      }
    }
}

struct Lanes {
  int wave, lane, wm, wn, li, lh;
};

template <bool A_KC, bool B_KC>
__device__ __forceinline__ void read_frags(const char* stage, const Lanes& q, Frags& f) {
  frag<A_KC>(stage, q.wm * 64, q.li, q.lh, f.a);
  frag<B_KC>(stage + TILE_B, q.wn * 64, q.li, q.lh, f.b);
}

__device__ __forceinline__ float sum8(const bf16x8& v) {
  const uint4 w = __builtin_bit_cast(uint4, v);
  const uint32_t x[4] = {w.x, w.y, w.z, w.w};
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) s += __uint_as_float(x[i] << 16) + __uint_as_float(x[i] & 0xFFFF0000u);
  return s;
}

// K step: the fragments of this step are in `cur`; the loads of the next
// NS-1 steps are in flight.  Wait until every wave has read `cur`'s stage
// and the next step's loads have landed (at most the 4*(NS-2) load
// instructions issued after the next step's may remain), start the loads
// `src` of the step NS ahead into `wr` (the stage this step came from), read
// the next step's fragments from `rd` into `nxt`, run this step's MFMAs.
// Loads past the end of K read the zero page, so every step has the same
// shape.  BSUM: add this step's A operands (dZ^T of the weight-gradient
// product) to the lane's two bias-gradient partial sums.
template <bool A_KC, bool B_KC, bool BSUM>
__device__ __forceinline__ void k_step(const Lanes& q, const Frags& cur, Frags& nxt, const char* rd, char* wr,
                                       const uint16_t* const (&src)[4], f32x16 (&acc)[2][2], float (&bsum)[2]) {
  // the scheduler keeps each step's work between its waits: it would
  // otherwise pull the next step's MFMAs up against the reads they need
  __builtin_amdgcn_sched_barrier(0);
  wait_lgkm0();
  wait_vm<4 * (NS - 2)>();
  barrier();
  const uint32_t wa = lds_off(wr) + 2048 * q.wave;
  fire(src[0], wa);
  fire(src[1], wa + 1024);
  fire(src[2], wa + TILE_B);
  fire(src[3], wa + TILE_B + 1024);
  read_frags<A_KC, B_KC>(rd, q, nxt);
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
        acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur.a[bi][s], cur.b[bj][s], acc[bi][bj], 0, 0, 0);
  if (BSUM) {
#pragma unroll
    for (int b = 0; b < 2; ++b) bsum[b] += sum8(cur.a[b][0]) + sum8(cur.a[b][1]);
  }
  // issue order: the next step's LDS reads spread between the MFMAs
  constexpr int NR = (A_KC ? 4 : 8) + (B_KC ? 4 : 8);  // LDS read instructions per step
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);       // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, NR / 4, 0);  // LDS read
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);       // MFMA
  }
  __builtin_amdgcn_sched_barrier(0);
}

__host__ __device__ inline int tiles16(const GemmArgs& g) {
  return ((g.M + TB - 1) / TB) * ((g.N + TB - 1) / TB) * g.batch;
}

// One 128x128 output tile (logical tile id `logical`) of one product;
// lds: LDS_DL bytes.
template <bool A_KC, bool B_KC, int EPI>
__device__ __forceinline__ void tile_dl16(const GemmArgs& g, const int logical, char* lds) {
  constexpr bool DW = EPI == EPI_DW_UPDATE;
  const int tid = threadIdx.x;
  const Lanes q{tid >> 6, tid & 63, (tid >> 6) >> 1, (tid >> 6) & 1, tid & 31, (tid & 63) >> 5};
  const int tm = (g.M + TB - 1) / TB, tn = (g.N + TB - 1) / TB;
  const int worker = logical / (tm * tn), rem = logical % (tm * tn);
  const int tile_n = rem / tm, m0 = (rem % tm) * TB, n0 = tile_n * TB;
  char* const st0 = lds;
  char* const st1 = lds + STAGE_B;
  char* const st2 = lds + 2 * STAGE_B;
  char* const st3 = lds + 3 * STAGE_B;

  Loader<A_KC> la;
  Loader<B_KC> lb;
  la.init(g.a, g.g, g.zero, worker, m0, g.M, g.K, q.wave, q.lane);
  lb.init(g.b, g.g, g.zero, worker, n0, g.N, g.K, q.wave, q.lane);

  float bsum[2] = {0.f, 0.f};
  f32x16 acc[2][2];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[bi][bj][r] = 0.f;

  const int nk = (g.K + BK - 1) / BK;
  // steps 0..NS-1 in flight (4 load instructions per wave per step), then
  // the fragments of step 0
  {
    char* const stg[NS] = {st0, st1, st2, st3};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const uint32_t wa = lds_off(stg[s]) + 2048 * q.wave;
      fire(la.src(s * BK, 0), wa);
      fire(la.src(s * BK, 1), wa + 1024);
      fire(lb.src(s * BK, 0), wa + TILE_B);
      fire(lb.src(s * BK, 1), wa + TILE_B + 1024);
    }
  }
  wait_vm<4 * (NS - 1)>();
  barrier();
  Frags f0, f1;
  read_frags<A_KC, B_KC>(st0, q, f0);

  // step kt loads step kt + NS: from the precomputed full-step sources
  // while that step lies inside K, else through the bounds checks
  auto step = [&](auto full, const Frags& cur, Frags& nxt, const char* rd, char* wr, int kt) {
    const int k0 = (kt + NS) * BK;
    if constexpr (decltype(full)::value) {
      const uint16_t* const src[4] = {la.src_full(k0, 0), la.src_full(k0, 1), lb.src_full(k0, 0),
                                      lb.src_full(k0, 1)};
      k_step<A_KC, B_KC, DW>(q, cur, nxt, rd, wr, src, acc, bsum);
    } else {
      const uint16_t* const src[4] = {la.src(k0, 0), la.src(k0, 1), lb.src(k0, 0), lb.src(k0, 1)};
      k_step<A_KC, B_KC, DW>(q, cur, nxt, rd, wr, src, acc, bsum);
    }
  };
  using Full = std::true_type;
  using Checked = std::false_type;
  // stage of step kt: kt % 4; fragment set: kt % 2
  const int nk4 = nk & ~3;
  int nfast = (la.full_ok && lb.full_ok) ? g.K / BK - NS : 0;  // steps kt whose step kt+NS is full
  nfast = nfast > 0 ? nfast & ~3 : 0;
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
  // wave is done reading the stages: the LDS is free for the epilogue
  wait_vm<0>();
  wait_lgkm0();
  barrier();

  if constexpr (!DW) {
    out_epilogue_lds<EPI>(g, worker, m0, n0, acc, reinterpret_cast<float*>(lds));
  } else {
    const AdamCoef ac = g.adam.on ? adam_coef(g.g, g.adam) : AdamCoef{1.f, 1.f};
    if (g.last)
      dw_epilogue_lds<true>(g, worker, m0, n0, acc, reinterpret_cast<float*>(lds), ac);
    else
      dw_epilogue_lds<false>(g, worker, m0, n0, acc, reinterpret_cast<float*>(lds), ac);
    // bias gradient: the first column tile; lanes lh = 0 and 1 of a wave
    // hold the sums over the two halves of each k slice of the same column
    // of dZ (waves wn = 0 and 1 hold the same sums)
    if (tile_n == 0 && q.wn == 0) {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const float tot = bsum[b] + __shfl_xor(bsum[b], 32);
        const int o = m0 + q.wm * 64 + 32 * b + q.li;
        if (q.lh == 0 && o < g.M) {
          const int64_t e = (int64_t)worker * g.pstride + o;
          const float stp = g.adam.on ? adam_dir(tot, g.adam.mb, g.adam.vb, e, g.adam, ac) : tot;
          const float nb = g.b_src[e] - g.eta * stp;
          g.b_dst[e] = g.last ? (nb - g.b_snap[e]) / g.lam : nb;
        }
      }
    }
  }
}

template <bool A_KC, bool B_KC, int EPI>
__global__ __launch_bounds__(NT) void gemm_bf16_dl_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) char lds[LDS_DL];
  tile_dl16<A_KC, B_KC, EPI>(g, xcd_remap(blockIdx.x, tiles16(g)), lds);
}

// The backward products of one layer in one launch: input-gradient tiles
// (workgroups [0, n1), the range padded to a multiple of 8 workgroups),
// then the weight-gradient tiles; each range laid out over the XCDs on its
// own.  Both read dZ_{l+1}; the first reads W_l from the step's source
// parameters, the second writes the destination parameters.
__global__ __launch_bounds__(NT) void gemm_bf16_dl_bwd_kernel(GemmArgs dx, GemmArgs dw, int n1, int n1pad) {
  __shared__ __attribute__((aligned(16))) char lds[LDS_DL];
  const int pid = blockIdx.x;
  if (pid < n1pad) {
    if (pid < n1) tile_dl16<true, false, EPI_DX_MASK>(dx, xcd_remap(pid, n1), lds);
  } else {
    tile_dl16<false, false, EPI_DW_UPDATE>(dw, xcd_remap(pid - n1pad, tiles16(dw)), lds);
  }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// the operand can be staged in 16-byte chunks (8 bf16) that never straddle
// an edge; a K-strided operand may be gathered only where the caller says so
bool operand_ok(const Operand& op, bool kc, int outer_n, int K, bool gather_ok) {
  if (!op.vec || !aligned16(op.ptr) || op.ld % 8 || op.wstride % 8) return false;
  if (kc) return K % 8 == 0;
  return outer_n % 8 == 0 && (!op.gather || gather_ok);
}

}  // namespace

bool gemm_bf16_dl_ok(int a_kc, int b_kc, const GemmArgs& g) {
  if (!g.zero || g.M <= 0 || g.N <= 0 || g.K <= 0) return false;
  if (a_kc && b_kc)
    return (g.epi == EPI_FWD_RELU || g.epi == EPI_FWD_LINEAR) && operand_ok(g.a, true, g.M, g.K, false) &&
           operand_ok(g.b, true, g.N, g.K, false) && out_vec_ok(g);
  if (a_kc && !b_kc)
    return g.epi == EPI_DX_MASK && operand_ok(g.a, true, g.M, g.K, false) &&
           operand_ok(g.b, false, g.N, g.K, false) && out_vec_ok(g);
  if (!a_kc && !b_kc)
    return g.epi == EPI_DW_UPDATE && operand_ok(g.a, false, g.M, g.K, false) &&
           operand_ok(g.b, false, g.N, g.K, g.K <= g.g.S) && dw_vec_ok(g);
  return false;
}

hipError_t launch_gemm_bf16_dl(int a_kc, int b_kc, const GemmArgs& g, hipStream_t s) {
  const dim3 grid(tiles16(g)), block(NT);
  if (a_kc && b_kc && g.epi == EPI_FWD_RELU)
    hipLaunchKernelGGL((gemm_bf16_dl_kernel<true, true, EPI_FWD_RELU>), grid, block, 0, s, g);
  else if (a_kc && b_kc && g.epi == EPI_FWD_LINEAR)
    hipLaunchKernelGGL((gemm_bf16_dl_kernel<true, true, EPI_FWD_LINEAR>), grid, block, 0, s, g);
  else if (a_kc && !b_kc && g.epi == EPI_DX_MASK)
    hipLaunchKernelGGL((gemm_bf16_dl_kernel<true, false, EPI_DX_MASK>), grid, block, 0, s, g);
  else if (!a_kc && !b_kc && g.epi == EPI_DW_UPDATE)
    hipLaunchKernelGGL((gemm_bf16_dl_kernel<false, false, EPI_DW_UPDATE>), grid, block, 0, s, g);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_gemm_bf16_dl_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s) {
  const int n1 = tiles16(dx), n1pad = (n1 + kNumXcd - 1) / kNumXcd * kNumXcd;
  hipLaunchKernelGGL(gemm_bf16_dl_bwd_kernel, dim3(n1pad + tiles16(dw)), dim3(NT), 0, s, dx, dw, n1, n1pad);
  return hipGetLastError();
}

}  // namespace agn
