// Batched bf16 products (bf16 operands, float32 accumulation) with direct
// global->LDS operand loads (global_load_lds_dwordx4 on gfx950): operand
// tiles travel from memory into LDS without passing through registers,
// three K steps ahead of their use, and the fragments of the next K step
// are read from LDS while the MFMAs of the current one run.
//
// Tile: TR x TR outputs per workgroup, TR = 128 (4 waves, two workgroups
// per CU; wave (wm, wn) owns a 64 x 64 quarter) or 256 (forward products
// with a whole 256-row mini-batch per tile, one workgroup of 8 waves per
// CU; wave (wm, wn) owns 128 x 64), as blocks of v_mfma_f32_32x32x16_bf16;
// K in steps of 32 (two MFMA slices of 16).  In one MFMA, lane (li = l%32,
// lh = l/32) supplies
// A[i = li][k = 8*lh .. 8*lh+7] and B[k = 8*lh .. 8*lh+7][j = li], 16 bytes
// each; the 128-tile accumulators are laid out as the shared epilogues
// expect.
//
// LDS layout of one operand tile (TR x 32 bf16 = TR*4 chunks of 16 bytes; a
// wave's load instruction fills 64 consecutive chunks, lane l chunk l):
//   K-contiguous (rows = outer index, 4 chunks of 8 k per row): chunk
//     (r, q) at 4r + (q ^ key(r)), key(r) = ((r >> 1) ^ (r >> 3)) & 3.  A
//     fragment is one 16-byte read; the rows of 8 consecutive lanes land in
//     8 distinct 16-byte bank groups modulo 128 bytes, those of 16
//     consecutive lanes in 16 distinct groups modulo 256 bytes.
//   K-strided (rows = k, TR/8 chunks of 8 outer per row): chunk (k, c) at
//     (TR/8)k + (c ^ key(k)), key(k) = 0, 6, 12, 10 for k % 4 = 0..3.  A
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

constexpr int BK = 32, NS = 4;  // k per step, LDS stages

// Geometry of a TR x TR output tile (TR = 128 or 256): four waves of
// TR/2 x TR/2, each as NB x NB blocks of 32 x 32.
template <int TR>
struct Geo {
  static constexpr int NB = TR / 64;        // blocks per wave and dimension
  static constexpr int IPW = TR / 64;       // load instructions per wave, operand and K step
  static constexpr int TILE = TR * BK * 2;  // bytes of one operand tile
  static constexpr int STAGE = 2 * TILE;    // A and B
  static constexpr int CPK = TR / 8;        // 16-byte chunks per k row of a K-strided tile
  static constexpr int RPI = 512 / TR;      // k rows per load instruction of a K-strided tile
};
constexpr int LDS_DL = NS * Geo<128>::STAGE > EPI_BYTES ? NS * Geo<128>::STAGE : EPI_BYTES;
// 256 x 256 tiles: the epilogue stages 128 rows at a time
constexpr int EPI_BIG_LD = 256 + 4;
constexpr int EPI_BIG_BYTES = 128 * EPI_BIG_LD * 4;
constexpr int LDS_BIG = NS * Geo<256>::STAGE > EPI_BIG_BYTES ? NS * Geo<256>::STAGE : EPI_BIG_BYTES;

__device__ __forceinline__ int kc_key(int r) { return ((r >> 1) ^ (r >> 3)) & 3; }
__device__ __forceinline__ int ks_key(int k) { return (0xAC60 >> (4 * (k & 3))) & 15; }
__device__ __forceinline__ int kc_byte(int r, int q) { return (4 * r + (q ^ kc_key(r))) * 16; }
template <int TR>
__device__ __forceinline__ int ks_byte(int k, int c) { return (Geo<TR>::CPK * k + (c ^ ks_key(k))) * 16; }

// Per-lane sources of one operand's IPW load instructions per K step
// (instruction j = IPW*wave + u, u < IPW; lane l fills chunk 64j + l):
//   K-contiguous: row r = 16j + l/4 (rows may be gathered data-set rows),
//     k chunk (l%4) ^ key(r);
//   K-strided: k row RPI*j + l/CPK, column chunk (l%CPK) ^ key(k) (k rows
//     may be gathered data-set rows: batch index kk of worker w is row
//     w*S + (tb + kk) mod S, tb = t*m mod S, with K <= S).
template <bool KC, int TR, int IPW_ = Geo<TR>::IPW>
struct Loader {
  static constexpr int IPW = IPW_, CPK = Geo<TR>::CPK, RPI = Geo<TR>::RPI;
  const uint16_t* zero;
  // the lane's source at k0 = 0 in instruction u: its row (KC) or column
  // chunk (KS), clamped into the matrix -- rows and columns past the edge
  // feed only outputs that are never stored, so steps whose loads all lie
  // inside K ("full" steps) load from fast[u] + offset(k0) whatever the lane
  const uint16_t* fast[IPW];
  int lk[IPW];     // KC: the lane's k offset in a step; KS: its k row in a step
  uint32_t valid;  // bit u: instruction u's row / column chunk lies inside the matrix
  int64_t ld, tb, S;
  int K, gather;
  bool full_ok;    // false: a gathered mini-batch wraps round the shard's end

  __device__ void init(const Operand& op, const Gather& g, const void* zp, int64_t w, int o0, int on, int k,
                       int wave, int lane) {
    const uint16_t* base = reinterpret_cast<const uint16_t*>(op.ptr) + w * op.wstride;
    zero = reinterpret_cast<const uint16_t*>(zp);
    ld = op.ld;
    K = k;
    gather = op.gather;
    valid = 0;
    if (KC) {
      const int64_t t = op.gather ? gather_step(g) : 0;
      tb = S = 0;
      full_ok = true;
#pragma unroll
      for (int u = 0; u < IPW; ++u) {
        const int r = 16 * (IPW * wave + u) + lane / 4;
        const int o = o0 + r, oc = o < on ? o : on - 1;
        const int64_t ri = op.gather ? batch_row(w, t, g.mb, g.S, oc) : oc;
        valid |= (o < on ? 1u : 0u) << u;
        fast[u] = base + ri * ld;
        lk[u] = 8 * ((lane % 4) ^ kc_key(r));
      }
    } else {
      S = g.S;
      tb = op.gather ? (gather_step(g) * g.mb) % g.S : 0;
      const int64_t rbase = op.gather ? w * g.S + tb : 0;
      full_ok = !op.gather || tb + K <= S;
#pragma unroll
      for (int u = 0; u < IPW; ++u) {
        const int kr = RPI * (IPW * wave + u) + lane / CPK;
        const int o = o0 + 8 * ((lane % CPK) ^ ks_key(kr));
        valid |= (o < on ? 1u : 0u) << u;
        fast[u] = base + (rbase + kr) * ld + (o < on ? o : on - 8);
        lk[u] = kr;
      }
    }
  }

  // source for a full step
  __device__ const uint16_t* src_full(int k0, int u) const {
    return KC ? fast[u] + (k0 + lk[u]) : fast[u] + (int64_t)k0 * ld;
  }

  // source of this lane's 16 bytes in load instruction u of the K step
  // starting at k0; the zero page past an edge (also for k0 >= K).  A
  // gathered k row past the shard's end wraps round to its start.
  __device__ const uint16_t* src(int k0, int u) const {
    const int kk = k0 + lk[u];
    if (!((valid >> u) & 1u) || kk >= K) return zero;
    if (KC) return fast[u] + kk;
    return fast[u] + (int64_t)(gather && tb + kk >= S ? k0 - S : k0) * ld;
  }
};

// Fragments of one wave for one K step: a[b][s] / b[b][s] is the operand of
// block b in slice s (k = 16s + 8*lh + 0..7 of the step).
template <int TR>
struct Frags {
  bf16x8 a[Geo<TR>::NB][2], b[Geo<TR>::NB][2];
};

template <bool KC, int TR, int NBLK = Geo<TR>::NB>
__device__ __forceinline__ void frag(const char* tile, int outer_off, int li, int lh, bf16x8 (&f)[NBLK][2]) {
#pragma unroll
  for (int b = 0; b < NBLK; ++b)
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
              (lds_i16x4*)(tile + ks_byte<TR>(k, col / 8) + 2 * (col % 8)));
          h[c] = __builtin_bit_cast(bf16x4, v);
        }
        f[b][s] = __builtin_shufflevector(h[0], h[1], 0, 1, 2, 3, 4, 5, 6, 7);
      }
    }
}

struct Lanes {
  int wave, lane, wm, wn, li, lh;
};

template <bool A_KC, bool B_KC, int TR>
__device__ __forceinline__ void read_frags(const char* stage, const Lanes& q, Frags<TR>& f) {
  frag<A_KC, TR>(stage, q.wm * (TR / 2), q.li, q.lh, f.a);
  frag<B_KC, TR>(stage + Geo<TR>::TILE, q.wn * (TR / 2), q.li, q.lh, f.b);
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
// and the next step's loads have landed (at most the 2*IPW*(NS-2) load
// instructions issued after the next step's may remain), start the loads
// `src` of the step NS ahead into `wr` (the stage this step came from), read
// the next step's fragments from `rd` into `nxt`, run this step's MFMAs.
// Loads past the end of K read the zero page, so every step has the same
// shape.  BSUM: add this step's A operands (dZ^T of the weight-gradient
// product) to the lane's bias-gradient partial sums.
template <bool A_KC, bool B_KC, int TR, bool BSUM>
__device__ __forceinline__ void k_step(const Lanes& q, const Frags<TR>& cur, Frags<TR>& nxt, const char* rd,
                                       char* wr, const uint16_t* const (&src)[2 * Geo<TR>::IPW],
                                       f32x16 (&acc)[Geo<TR>::NB][Geo<TR>::NB], float (&bsum)[Geo<TR>::NB]) {
  constexpr int NB = Geo<TR>::NB, IPW = Geo<TR>::IPW;
  // the scheduler keeps each step's work between its waits: it would
  // otherwise pull the next step's MFMAs up against the reads they need
  __builtin_amdgcn_sched_barrier(0);
  wait_lgkm0();
  wait_vm<2 * IPW * (NS - 2)>();
  barrier();
  const uint32_t wa = lds_off(wr) + 1024 * IPW * q.wave;
#pragma unroll
  for (int u = 0; u < IPW; ++u) fire(src[u], wa + 1024 * u);
#pragma unroll
  for (int u = 0; u < IPW; ++u) fire(src[IPW + u], wa + Geo<TR>::TILE + 1024 * u);
  read_frags<A_KC, B_KC, TR>(rd, q, nxt);
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int bi = 0; bi < NB; ++bi)
#pragma unroll
      for (int bj = 0; bj < NB; ++bj)
        acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur.a[bi][s], cur.b[bj][s], acc[bi][bj], 0, 0, 0);
  if (BSUM) {
#pragma unroll
    for (int b = 0; b < NB; ++b) bsum[b] += sum8(cur.a[b][0]) + sum8(cur.a[b][1]);
  }
  // issue order: the next step's LDS reads spread between the MFMAs
  constexpr int NR = NB * ((A_KC ? 2 : 4) + (B_KC ? 2 : 4));  // LDS read instructions per step
  constexpr int NM = 2 * NB * NB;                               // MFMAs per step
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, NM / 8, 0);  // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, NR / 4, 0);  // LDS read
    __builtin_amdgcn_sched_group_barrier(0x008, NM / 8, 0);  // MFMA
  }
  __builtin_amdgcn_sched_barrier(0);
}

template <int TR>
__host__ __device__ inline int tiles16(const GemmArgs& g) {
  return ((g.M + TR - 1) / TR) * ((g.N + TR - 1) / TR) * g.batch;
}

// One TR x TR output tile (logical tile id `logical`) of one product (TR =
// 128; the 256 x 256 forward tiles have a kernel of their own below); lds:
// LDS_DL bytes.
template <bool A_KC, bool B_KC, int EPI, int TR>
__device__ __forceinline__ void tile_dl16(const GemmArgs& g, const int logical, char* lds) {
  constexpr bool DW = EPI == EPI_DW_UPDATE;
  constexpr int NB = Geo<TR>::NB, IPW = Geo<TR>::IPW, STAGE = Geo<TR>::STAGE;
  static_assert(TR == 128, "four-wave tiles are 128 x 128");
  const int tid = threadIdx.x;
  const Lanes q{tid >> 6, tid & 63, (tid >> 6) >> 1, (tid >> 6) & 1, tid & 31, (tid & 63) >> 5};
  const int tm = (g.M + TR - 1) / TR, tn = (g.N + TR - 1) / TR;
  const int worker = logical / (tm * tn), rem = logical % (tm * tn);
  const int tile_n = rem / tm, m0 = (rem % tm) * TR, n0 = tile_n * TR;
  char* const st0 = lds;
  char* const st1 = lds + STAGE;
  char* const st2 = lds + 2 * STAGE;
  char* const st3 = lds + 3 * STAGE;

  Loader<A_KC, TR> la;
  Loader<B_KC, TR> lb;
  la.init(g.a, g.g, g.zero, worker, m0, g.M, g.K, q.wave, q.lane);
  lb.init(g.b, g.g, g.zero, worker, n0, g.N, g.K, q.wave, q.lane);

  float bsum[NB];
  f32x16 acc[NB][NB];
#pragma unroll
  for (int bi = 0; bi < NB; ++bi) {
    bsum[bi] = 0.f;
#pragma unroll
    for (int bj = 0; bj < NB; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[bi][bj][r] = 0.f;
  }

  const int nk = (g.K + BK - 1) / BK;
  // steps 0..NS-1 in flight (2*IPW load instructions per wave per step),
  // then the fragments of step 0
  {
    char* const stg[NS] = {st0, st1, st2, st3};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const uint32_t wa = lds_off(stg[s]) + 1024 * IPW * q.wave;
#pragma unroll
      for (int u = 0; u < IPW; ++u) fire(la.src(s * BK, u), wa + 1024 * u);
#pragma unroll
      for (int u = 0; u < IPW; ++u) fire(lb.src(s * BK, u), wa + Geo<TR>::TILE + 1024 * u);
    }
  }
  wait_vm<2 * IPW * (NS - 1)>();
  barrier();
  Frags<TR> f0, f1;
  read_frags<A_KC, B_KC, TR>(st0, q, f0);

  // step kt loads step kt + NS: from the precomputed full-step sources
  // while that step lies inside K, else through the bounds checks
  auto step = [&](auto full, const Frags<TR>& cur, Frags<TR>& nxt, const char* rd, char* wr, int kt) {
    const int k0 = (kt + NS) * BK;
    const uint16_t* src[2 * IPW];
#pragma unroll
    for (int u = 0; u < IPW; ++u) {
      if constexpr (decltype(full)::value) {
        src[u] = la.src_full(k0, u);
        src[IPW + u] = lb.src_full(k0, u);
      } else {
        src[u] = la.src(k0, u);
        src[IPW + u] = lb.src(k0, u);
      }
    }
    k_step<A_KC, B_KC, TR, DW>(q, cur, nxt, rd, wr, src, acc, bsum);
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
      for (int b = 0; b < NB; ++b) {
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
  tile_dl16<A_KC, B_KC, EPI, 128>(g, xcd_remap(blockIdx.x, tiles16<128>(g)), lds);
}

// ---------------------------------------------------------------------------
// Forward product in 256 x 256 tiles with eight waves (two per SIMD): wave
// (wm, wn) = (w / 4, w % 4) owns rows 128wm .. +127 and columns 64wn .. +63
// of the tile as 4 x 2 blocks of 32 x 32, and issues two load instructions
// per operand and K step (instruction j = 2w + u).  With one wave per SIMD
// a wave held up in instruction issue (waiting for room in the memory
// pipeline), on its LDS reads or at the barrier left the matrix core idle;
// with two, the other wave of the SIMD runs its MFMAs meanwhile.
constexpr int NT_BIG = 512;
constexpr int IPW_BIG = 2;

struct FragsBig {
  bf16x8 a[4][2], b[2][2];
};

// the wave's fragments of one K step, slice 0's reads first
__device__ __forceinline__ void read_frags_big(const char* stage, int wm, int wn, int li, int lh, FragsBig& f) {
  const char* tb = stage + Geo<256>::TILE;
#pragma unroll
  for (int sl = 0; sl < 2; ++sl) {
#pragma unroll
    for (int b = 0; b < 4; ++b)
      f.a[b][sl] = *reinterpret_cast<const bf16x8*>(stage + kc_byte(wm * 128 + 32 * b + li, 2 * sl + lh));
#pragma unroll
    for (int b = 0; b < 2; ++b)
      f.b[b][sl] = *reinterpret_cast<const bf16x8*>(tb + kc_byte(wn * 64 + 32 * b + li, 2 * sl + lh));
  }
}

// K step kt: wait until step kt's loads have landed (at most the loads of
// steps kt+1 and kt+2 still in flight) and every wave is done reading the
// stage of step kt-1; start the loads of step kt+3 into that stage; read
// this step's fragments and run its MFMAs.  The fragments are read in the
// step that uses them (one set of registers: the other wave of the SIMD
// runs its MFMAs meanwhile); slice 0's MFMAs start while slice 1's reads
// are in flight.
__device__ __forceinline__ void k_step_big(int wave, int wm, int wn, int li, int lh, const char* rd, char* wr,
                                           const uint16_t* const (&src)[2 * IPW_BIG], f32x16 (&acc)[4][2]) {
  __builtin_amdgcn_sched_barrier(0);
  wait_lgkm0();
  wait_vm<2 * IPW_BIG * (NS - 2)>();
  barrier();
  const uint32_t wa = lds_off(wr) + 1024 * IPW_BIG * wave;
#pragma unroll
  for (int u = 0; u < IPW_BIG; ++u) fire(src[u], wa + 1024 * u);
#pragma unroll
  for (int u = 0; u < IPW_BIG; ++u) fire(src[IPW_BIG + u], wa + Geo<256>::TILE + 1024 * u);
  FragsBig f;
  read_frags_big(rd, wm, wn, li, lh, f);
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
        acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[bi][s], f.b[bj][s], acc[bi][bj], 0, 0, 0);
  __builtin_amdgcn_sched_barrier(0);
}

// Epilogue of the eight-wave tile: two passes of 128 rows; in pass h the
// four waves with wm == h stage their accumulators in LDS, then every
// thread stores 16-byte row chunks (8 bf16 or 4 float32 columns) with the
// bias loaded up front from indices clamped into the matrix (element by
// element only where a chunk crosses the matrix edge).
template <int EPI>
__device__ __forceinline__ void out_epilogue_big8(const GemmArgs& g, int worker, int m0, int n0,
                                                  const f32x16 (&acc)[4][2], float* et) {
  static_assert(EPI == EPI_FWD_RELU || EPI == EPI_FWD_LINEAR, "forward products only");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3, li = lane & 31, lh = lane >> 5;
  constexpr bool F32 = EPI == EPI_FWD_LINEAR;
  constexpr int CW = F32 ? 4 : 8;         // columns per chunk
  constexpr int CPR = 256 / CW;           // chunks per row
  constexpr int NC = 128 * CPR / NT_BIG;  // chunks per thread and pass
  const int colc = (tid % CPR) * CW;      // this thread's chunk column (the same for all its chunks)
  const int cbase = n0 + colc;
  float bv[CW];
#pragma unroll
  for (int j = 0; j < CW; ++j) bv[j] = g.bias[(int64_t)worker * g.bstride + min(cbase + j, g.N - 1)];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (h == 1) __syncthreads();  // every thread is done reading pass 0's rows
    if (wm == h) {
#pragma unroll
      for (int bi = 0; bi < 4; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            et[(32 * bi + 8 * (r >> 2) + 4 * lh + (r & 3)) * EPI_BIG_LD + wn * 64 + 32 * bj + li] = acc[bi][bj][r];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < CW; j += 2) asm volatile("" ::"v"(bv[j]), "v"(bv[j + 1]));
    if (cbase >= g.N) continue;
    const bool whole = cbase + CW <= g.N;
#pragma unroll
    for (int u = 0; u < NC; ++u) {
      const int rl = (tid + NT_BIG * u) / CPR, row = m0 + 128 * h + rl;
      if (row >= g.M) continue;
      float v[CW];
#pragma unroll
      for (int j = 0; j < CW; j += 4) {
        const float4 a = *reinterpret_cast<const float4*>(et + rl * EPI_BIG_LD + colc + j);
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
#pragma unroll
        for (int j = 0; j < CW; ++j) {
          const float z = v[j] + bv[j];
          hv[j] = f32_to_bf16_rne(z > 0.f ? z : 0.f);
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
}

// 256 x 256 tiles, one workgroup per CU (LDS)
template <int EPI>
__global__ __launch_bounds__(NT_BIG) void gemm_bf16_dl_big_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) char lds[LDS_BIG];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & 7;
  const int wm = wave >> 2, wn = wave & 3, li = lane & 31, lh = lane >> 5;
  const int logical = xcd_remap(blockIdx.x, tiles16<256>(g));
  const int tm = (g.M + 255) / 256, tn = (g.N + 255) / 256;
  const int worker = logical / (tm * tn), rem = logical % (tm * tn);
  const int m0 = (rem % tm) * 256, n0 = (rem / tm) * 256;
  constexpr int STAGE = Geo<256>::STAGE;
  char* const st0 = lds;
  char* const st1 = lds + STAGE;
  char* const st2 = lds + 2 * STAGE;
  char* const st3 = lds + 3 * STAGE;

  Loader<true, 256, IPW_BIG> la, lb;
  la.init(g.a, g.g, g.zero, worker, m0, g.M, g.K, wave, lane);
  lb.init(g.b, g.g, g.zero, worker, n0, g.N, g.K, wave, lane);
  f32x16 acc[4][2];
#pragma unroll
  for (int bi = 0; bi < 4; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[bi][bj][r] = 0.f;

  const int nk = (g.K + BK - 1) / BK;
  {
    // steps 0 .. NS-2 in flight (2*IPW_BIG load instructions per wave and step)
    char* const stg[NS - 1] = {st0, st1, st2};
#pragma unroll
    for (int s = 0; s < NS - 1; ++s) {
      const uint32_t wa = lds_off(stg[s]) + 1024 * IPW_BIG * wave;
#pragma unroll
      for (int u = 0; u < IPW_BIG; ++u) fire(la.src(s * BK, u), wa + 1024 * u);
#pragma unroll
      for (int u = 0; u < IPW_BIG; ++u) fire(lb.src(s * BK, u), wa + Geo<256>::TILE + 1024 * u);
    }
  }

  // step kt reads stage kt % 4 and loads step kt + 3 into stage (kt + 3) % 4:
  // from the precomputed full-step sources while that step lies inside K,
  // else through the bounds checks (the zero page past K)
  auto step = [&](auto full, const char* rd, char* wr, int kt) {
    const int k0 = (kt + NS - 1) * BK;
    const uint16_t* src[2 * IPW_BIG];
#pragma unroll
    for (int u = 0; u < IPW_BIG; ++u) {
      if constexpr (decltype(full)::value) {
        src[u] = la.src_full(k0, u);
        src[IPW_BIG + u] = lb.src_full(k0, u);
      } else {
        src[u] = la.src(k0, u);
        src[IPW_BIG + u] = lb.src(k0, u);
      }
    }
    k_step_big(wave, wm, wn, li, lh, rd, wr, src, acc);
  };
  using Full = std::true_type;
  using Checked = std::false_type;
  const int nk4 = nk & ~3;
  int nfast = (la.full_ok && lb.full_ok) ? g.K / BK - (NS - 1) : 0;  // steps kt whose step kt+3 is full
  nfast = nfast > 0 ? nfast & ~3 : 0;
  int kt = 0;
  for (; kt < nfast && kt < nk4; kt += 4) {
    step(Full{}, st0, st3, kt);
    step(Full{}, st1, st0, kt + 1);
    step(Full{}, st2, st1, kt + 2);
    step(Full{}, st3, st2, kt + 3);
  }
  for (; kt < nk4; kt += 4) {
    step(Checked{}, st0, st3, kt);
    step(Checked{}, st1, st0, kt + 1);
    step(Checked{}, st2, st1, kt + 2);
    step(Checked{}, st3, st2, kt + 3);
  }
  if (nk4 < nk) step(Checked{}, st0, st3, nk4);
  if (nk4 + 1 < nk) step(Checked{}, st1, st0, nk4 + 1);
  if (nk4 + 2 < nk) step(Checked{}, st2, st1, nk4 + 2);
  // every load (also those of the steps past the end) has landed and every
  // wave is done reading the stages: the LDS is free for the epilogue
  wait_vm<0>();
  wait_lgkm0();
  barrier();
  out_epilogue_big8<EPI>(g, worker, m0, n0, acc, reinterpret_cast<float*>(lds));
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
    if (pid < n1) tile_dl16<true, false, EPI_DX_MASK, 128>(dx, xcd_remap(pid, n1), lds);
  } else {
    tile_dl16<false, false, EPI_DW_UPDATE, 128>(dw, xcd_remap(pid - n1pad, tiles16<128>(dw)), lds);
  }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// the operand can be staged in 16-byte chunks (8 bf16).  A chunk may cross
// an edge only inside the row's padding: past K of a K-contiguous operand
// when that padding is zero (it meets the other operand's zero-page rows,
// so it adds nothing), past the outer size of a K-strided one in any case
// (those columns feed only outputs that are never stored).  A K-strided
// operand may be gathered only where the caller says so.
bool operand_ok(const Operand& op, bool kc, int outer_n, int K, bool gather_ok) {
  if (!op.vec || !aligned16(op.ptr) || op.ld % 8 || op.wstride % 8) return false;
  if (kc) return K % 8 == 0 || (op.padded && op.ld >= (K + 7) / 8 * 8);
  return (outer_n % 8 == 0 || op.ld >= (outer_n + 7) / 8 * 8) && (!op.gather || gather_ok);
}

}  // namespace

bool gemm_bf16_dl_ok(int a_kc, int b_kc, const GemmArgs& g) {
  if (!g.zero || g.M <= 0 || g.N <= 0 || g.K <= 0) return false;
  if (a_kc && b_kc)  // (both K-contiguous: no chunk past K, it would meet the other's padding)
    return (g.epi == EPI_FWD_RELU || g.epi == EPI_FWD_LINEAR) && g.K % 8 == 0 &&
           operand_ok(g.a, true, g.M, g.K, false) && operand_ok(g.b, true, g.N, g.K, false) && out_vec_ok(g);
  if (a_kc && !b_kc)
    return g.epi == EPI_DX_MASK && operand_ok(g.a, true, g.M, g.K, false) &&
           operand_ok(g.b, false, g.N, g.K, false) && out_vec_ok(g);
  if (!a_kc && !b_kc)
    return g.epi == EPI_DW_UPDATE && operand_ok(g.a, false, g.M, g.K, false) &&
           operand_ok(g.b, false, g.N, g.K, g.K <= g.g.S) && dw_vec_ok(g);
  return false;
}

// 256 x 256 tiles for the forward product where they fill the chip (the
// workgroups hold a whole 256-row mini-batch: each weight tile is read once)
static bool use_big(int a_kc, int b_kc, const GemmArgs& g) {
  return a_kc && b_kc && g.M >= 256 && g.N >= 256 && tiles16<256>(g) >= 256;
}

hipError_t launch_gemm_bf16_dl(int a_kc, int b_kc, const GemmArgs& g, hipStream_t s) {
  const dim3 block(NT);
  if (use_big(a_kc, b_kc, g)) {
    const dim3 grid(tiles16<256>(g));
    if (g.epi == EPI_FWD_RELU)
      AGN_LAUNCH((gemm_bf16_dl_big_kernel<EPI_FWD_RELU>), grid, dim3(NT_BIG), 0, s, g);
    else
      AGN_LAUNCH((gemm_bf16_dl_big_kernel<EPI_FWD_LINEAR>), grid, dim3(NT_BIG), 0, s, g);
    return hipGetLastError();
  }
  const dim3 grid(tiles16<128>(g));
  if (a_kc && b_kc && g.epi == EPI_FWD_RELU)
    AGN_LAUNCH((gemm_bf16_dl_kernel<true, true, EPI_FWD_RELU>), grid, block, 0, s, g);
  else if (a_kc && b_kc && g.epi == EPI_FWD_LINEAR)
    AGN_LAUNCH((gemm_bf16_dl_kernel<true, true, EPI_FWD_LINEAR>), grid, block, 0, s, g);
  else if (a_kc && !b_kc && g.epi == EPI_DX_MASK)
    AGN_LAUNCH((gemm_bf16_dl_kernel<true, false, EPI_DX_MASK>), grid, block, 0, s, g);
  else if (!a_kc && !b_kc && g.epi == EPI_DW_UPDATE)
    AGN_LAUNCH((gemm_bf16_dl_kernel<false, false, EPI_DW_UPDATE>), grid, block, 0, s, g);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_gemm_bf16_dl_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s) {
  const int n1 = tiles16<128>(dx), n1pad = (n1 + kNumXcd - 1) / kNumXcd * kNumXcd;
  AGN_LAUNCH(gemm_bf16_dl_bwd_kernel, dim3(n1pad + tiles16<128>(dw)), dim3(NT), 0, s, dx, dw, n1,
                     n1pad);
  return hipGetLastError();
}

}  // namespace agn
