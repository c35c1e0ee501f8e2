// Batched bf16 products of the local SGD step (bf16 operands, float32
// accumulation) on the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// A workgroup of 4 waves owns a 128x128 output tile of one worker; each wave
// owns a 64x64 quarter as 2x2 MFMA blocks (64 accumulator registers).  K is
// consumed 32 at a time through double-buffered LDS tiles, each operand in
// the layout it has in memory.  An MFMA operand fragment is 16 bytes per
// lane: one 16-byte LDS read from a K-contiguous tile ([outer][k]), two
// transposing LDS reads (ds_read_b64_tr_b16) from a K-strided one
// ([k][outer]: the N-contiguous weights of the input-gradient product and
// both operands of the weight-gradient product).
//
// Epilogues: forward  H = bf16(relu(acc + b)) (logits stay float32);
//            input gradient  dZ = bf16(acc * [H > 0]);
//            weight gradient  W <- W - eta * acc on the float32 master, with
//            the bf16 shadow of the new W written alongside (the operand of
//            the next step's products); b <- b - eta * sum over rows of the
//            bf16 dZ.  On a round's last step the normalized displacement
//            (W_new - W_pulled) / lambda is stored instead.  Epilogues go
//            through LDS so that outputs, masks and master weights move in
//            16-byte row chunks.
#include "bf16_epilogue.h"

namespace agn {
namespace {

constexpr int BKH = 32;          // k per step
constexpr int LDK = BKH + 8;     // LDS row stride (bf16 elements) of a K-contiguous [outer][k] tile
constexpr int LDS_KS = TB + 32;  // LDS row stride (bf16 elements) of a K-strided [k][outer] tile
constexpr int TILE = TB * LDK;   // bf16 elements per operand tile (either layout)
static_assert(BKH * LDS_KS <= TILE, "K-strided tile fits the tile buffer");
// LDS per workgroup: the two double-buffered operand tiles, or (after the
// K loop) the 128x128 float32 accumulator tile of the epilogue
constexpr int LDS_BYTES = (4 * TILE * 2 > TB * EPI_LD * 4) ? 4 * TILE * 2 : TB * EPI_LD * 4;

__device__ __forceinline__ uint4 load8(const uint16_t* p, int valid, int vec) {
  if (valid >= 8 && vec) return *reinterpret_cast<const uint4*>(p);
  uint16_t e[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) e[i] = i < valid ? p[i] : (uint16_t)0;
  uint4 v;
  v.x = e[0] | ((uint32_t)e[1] << 16);
  v.y = e[2] | ((uint32_t)e[3] << 16);
  v.z = e[4] | ((uint32_t)e[5] << 16);
  v.w = e[6] | ((uint32_t)e[7] << 16);
  return v;
}

// Staging of one 128 (outer) x 32 (k) operand tile, 2 chunks of 8 bf16 per thread.
// K-contiguous: chunk = (outer row tid/4 + 64p, k offset 8*(tid%4)).
// K-strided:    chunk = (k row tid/16 + 16p, outer offset 8*(tid%16)).
template <bool KC>
struct Loader16 {
  const uint16_t* rowp[2];
  const uint16_t* base;
  int64_t ld;
  int outer0, outer_n, K;
  int vec, gather;
  int64_t worker, t, mb, S;

  __device__ void init(const Operand& op, const Gather& g, int64_t w, int o0, int on, int k, int tid) {
    base = reinterpret_cast<const uint16_t*>(op.ptr) + w * op.wstride;
    ld = op.ld;
    outer0 = o0;
    outer_n = on;
    K = k;
    vec = op.vec;
    gather = op.gather;
    worker = w;
    mb = g.mb;
    S = g.S;
    t = gather ? gather_step(g) : 0;
    if (KC) {
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int o = o0 + tid / 4 + 64 * p;
        int64_t r = o;
        if (gather && o < on) r = batch_row(worker, t, mb, S, o);
        rowp[p] = o < on ? base + r * ld : nullptr;
      }
    }
  }

  __device__ void load(int k0, int tid, uint4 (&v)[2]) const {
    if (KC) {
      const int kk = k0 + 8 * (tid % 4);
#pragma unroll
      for (int p = 0; p < 2; ++p) v[p] = rowp[p] ? load8(rowp[p] + kk, K - kk, vec) : make_uint4(0, 0, 0, 0);
    } else {
      const int cc = outer0 + 8 * (tid % 16);
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int kr = k0 + tid / 16 + 16 * p;
        if (kr < K) {
          const int64_t r = gather ? batch_row(worker, t, mb, S, kr) : kr;
          v[p] = load8(base + r * ld + cc, outer_n - cc, vec);
        } else {
          v[p] = make_uint4(0, 0, 0, 0);
        }
      }
    }
  }

  __device__ static void store(uint16_t* lds, int tid, const uint4 (&v)[2]) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      if (KC)
        *reinterpret_cast<uint4*>(lds + (tid / 4 + 64 * p) * LDK + 8 * (tid % 4)) = v[p];
      else  // as stored: row k, 8 outer elements
        *reinterpret_cast<uint4*>(lds + (tid / 16 + 16 * p) * LDS_KS + 8 * (tid % 16)) = v[p];
    }
  }
};

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// MFMA operand of lane (li, lh) for outer index `outer` (its row or column)
// and k = k0 + 8*lh + e, e = 0..7.
// K-contiguous tile: one 16-byte read.
// K-strided tile ([k][outer]): two transposing reads (ds_read_b64_tr_b16).
// Within each group of 16 lanes, lane i of such a read receives element e
// from mem[A(4e + i/4) + i%4], A(j) being the address lane j supplies; so
// for read c (e = 4c .. 4c+3) lane j supplies row k0 + 8*lh + 4c + j/4 at
// column (outer - li) + 16*(li/16) + 4*(j%4), j = li % 16.
template <bool KC>
__device__ __forceinline__ bf16x8 frag(const uint16_t* lds, int outer, int k0, int li, int lh) {
  if (KC) return *reinterpret_cast<const bf16x8*>(lds + outer * LDK + k0 + 8 * lh);
  const int col = (outer - li) + 16 * (li / 16) + 4 * (li % 4);
  bf16x4 h[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int row = k0 + 8 * lh + 4 * c + (li % 16) / 4;
    const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(lds + row * LDS_KS + col));
    h[c] = __builtin_bit_cast(bf16x4, v);
  }
  return __builtin_shufflevector(h[0], h[1], 0, 1, 2, 3, 4, 5, 6, 7);
}

__host__ __device__ inline int tiles_of(const GemmArgs& g) { return ((g.M + TB - 1) / TB) * ((g.N + TB - 1) / TB) * g.batch; }

// One 128x128 output tile (logical tile id `logical`) of one product.
// lds: LDS_BYTES of LDS.
template <bool A_KC, bool B_KC, int EPI>
__device__ __forceinline__ void gemm_tile16(const GemmArgs& g, const int logical, char* lds) {
  uint16_t (*lds_a)[TILE] = reinterpret_cast<uint16_t (*)[TILE]>(lds);
  uint16_t (*lds_b)[TILE] = reinterpret_cast<uint16_t (*)[TILE]>(lds + 2 * TILE * 2);
  const int tid = threadIdx.x;
  const int tm = (g.M + TB - 1) / TB, tn = (g.N + TB - 1) / TB;
  const int worker = logical / (tm * tn);
  const int rem = logical % (tm * tn);
  const int tile_n = rem / tm, tile_m = rem % tm;
  const int m0 = tile_m * TB, n0 = tile_n * TB;

  Loader16<A_KC> la;
  Loader16<B_KC> lb;
  la.init(g.a, g.g, worker, m0, g.M, g.K, tid);
  lb.init(g.b, g.g, worker, n0, g.N, g.K, tid);

  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 31, lh = lane >> 5;

  // bias gradient: the first column tile sums each of its 128 dZ rows
  const bool do_bias = (EPI == EPI_DW_UPDATE) && tile_n == 0 && tid < TB;
  float bsum = 0.f;

  f32x16 acc[2][2];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[bi][bj][r] = 0.f;

  const int nk = (g.K + BKH - 1) / BKH;
  uint4 va[2], vb[2];
  la.load(0, tid, va);
  lb.load(0, tid, vb);
  Loader16<A_KC>::store(lds_a[0], tid, va);
  Loader16<B_KC>::store(lds_b[0], tid, vb);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      la.load((kt + 1) * BKH, tid, va);
      lb.load((kt + 1) * BKH, tid, vb);
    }
    // two MFMA k-steps of 16; lane (i, h) supplies k = 16s + 8h + e
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      bf16x8 af[2], bfr[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        af[b] = frag<A_KC>(lds_a[cur], wm * 64 + 32 * b + li, 16 * s, li, lh);
        bfr[b] = frag<B_KC>(lds_b[cur], wn * 64 + 32 * b + li, 16 * s, li, lh);
      }
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[bi], bfr[bj], acc[bi][bj], 0, 0, 0);
    }
    if (do_bias) {  // A = dZ^T, K-strided: column tid of the [k][outer] tile
#pragma unroll 8
      for (int k = 0; k < BKH; ++k) bsum += bf16_to_f32(lds_a[cur][k * LDS_KS + tid]);
    }
    if (kt + 1 < nk) {
      Loader16<A_KC>::store(lds_a[cur ^ 1], tid, va);
      Loader16<B_KC>::store(lds_b[cur ^ 1], tid, vb);
    }
    __syncthreads();
  }

  const AdamCoef ac = (EPI == EPI_DW_UPDATE && g.adam.on) ? adam_coef(g.g, g.adam) : AdamCoef{1.f, 1.f};
  if (EPI == EPI_DW_UPDATE && dw_vec_ok(g)) {
    // (the K loop ended with a barrier: the operand tiles are free)
    if (g.last)
      dw_epilogue_lds<true>(g, worker, m0, n0, acc, reinterpret_cast<float*>(lds), ac);
    else
      dw_epilogue_lds<false>(g, worker, m0, n0, acc, reinterpret_cast<float*>(lds), ac);
  } else if (EPI != EPI_DW_UPDATE && out_vec_ok(g)) {
    out_epilogue_lds<EPI>(g, worker, m0, n0, acc, reinterpret_cast<float*>(lds));
  } else {
  // epilogue: block (bi, bj) lane holds D[i][j], j = lane%32,
  // i = 8*(r/4) + 4*(lane/32) + r%4 within the 32x32 block
#pragma unroll
  for (int bj = 0; bj < 2; ++bj) {
    const int col = n0 + wn * 64 + 32 * bj + li;
    if (col >= g.N) continue;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + 32 * bi + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (row >= g.M) continue;
        const float v = acc[bi][bj][r];
        if (EPI == EPI_FWD_RELU) {
          const float h = v + g.bias[(int64_t)worker * g.bstride + col];
          reinterpret_cast<uint16_t*>(g.out)[(int64_t)worker * g.ostride + (int64_t)row * g.ldo + col] =
              f32_to_bf16_rne(h > 0.f ? h : 0.f);
        } else if (EPI == EPI_FWD_LINEAR) {
          reinterpret_cast<float*>(g.out)[(int64_t)worker * g.ostride + (int64_t)row * g.ldo + col] =
              v + g.bias[(int64_t)worker * g.bstride + col];
        } else if (EPI == EPI_DX_MASK) {
          const uint16_t hm =
              reinterpret_cast<const uint16_t*>(g.mask)[(int64_t)worker * g.mstride + (int64_t)row * g.ldm + col];
          const bool on = bf16_to_f32(hm) > 0.f;
          reinterpret_cast<uint16_t*>(g.out)[(int64_t)worker * g.ostride + (int64_t)row * g.ldo + col] =
              f32_to_bf16_rne(on ? v : 0.f);
        } else {  // EPI_DW_UPDATE
          const int64_t e = (int64_t)worker * g.pstride + (int64_t)row * g.ldw + col;
          const float step = g.adam.on ? adam_dir(v, g.adam.mw, g.adam.vw, e, g.adam, ac) : v;
          const float nw = g.w_src[e] - g.eta * step;
          if (g.last) {
            g.w_dst[e] = (nw - g.w_snap[e]) / g.lam;
          } else {
            g.w_dst[e] = nw;
            g.w_dst16[e] = f32_to_bf16_rne(nw);
          }
        }
      }
    }
  }
  }
  if (do_bias) {
    const int o = m0 + tid;
    if (o < g.M) {
      const int64_t e = (int64_t)worker * g.pstride + o;
      const float step = g.adam.on ? adam_dir(bsum, g.adam.mb, g.adam.vb, e, g.adam, ac) : bsum;
      const float nb = g.b_src[e] - g.eta * step;
      g.b_dst[e] = g.last ? (nb - g.b_snap[e]) / g.lam : nb;
    }
  }
}

template <bool A_KC, bool B_KC, int EPI>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) char lds[LDS_BYTES];
  gemm_tile16<A_KC, B_KC, EPI>(g, xcd_remap(blockIdx.x, tiles_of(g)), lds);
}

// Input-gradient tiles and weight-gradient tiles of one layer in one launch
// (see the float32 version).
__global__ __launch_bounds__(NT) void gemm_bf16_bwd_kernel(GemmArgs dx, GemmArgs dw, int n1, int n1pad) {
  __shared__ __attribute__((aligned(16))) char lds[LDS_BYTES];
  const int pid = blockIdx.x;
  if (pid < n1pad) {
    if (pid < n1) gemm_tile16<true, false, EPI_DX_MASK>(dx, xcd_remap(pid, n1), lds);
  } else {
    gemm_tile16<false, false, EPI_DW_UPDATE>(dw, xcd_remap(pid - n1pad, tiles_of(dw)), lds);
  }
}

template <bool A_KC, bool B_KC, int EPI>
hipError_t go(const GemmArgs& g, hipStream_t s) {
  AGN_LAUNCH((gemm_bf16_kernel<A_KC, B_KC, EPI>), dim3(tiles_of(g)), dim3(NT), 0, s, g);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s) {
  if (dx.epi != EPI_DX_MASK || dw.epi != EPI_DW_UPDATE) return hipErrorInvalidValue;
  if (gemm_bf16_dl_ok(1, 0, dx) && gemm_bf16_dl_ok(0, 0, dw)) return launch_gemm_bf16_dl_bwd(dx, dw, s);
  const int n1 = tiles_of(dx), n1pad = (n1 + kNumXcd - 1) / kNumXcd * kNumXcd;
  AGN_LAUNCH(gemm_bf16_bwd_kernel, dim3(n1pad + tiles_of(dw)), dim3(NT), 0, s, dx, dw, n1, n1pad);
  return hipGetLastError();
}

hipError_t launch_gemm_bf16(int a_kc, int b_kc, const GemmArgs& g, hipStream_t s) {
  if (gemm_bf16_dl_ok(a_kc, b_kc, g)) return launch_gemm_bf16_dl(a_kc, b_kc, g, s);
  if (a_kc && b_kc && g.epi == EPI_FWD_RELU) return go<true, true, EPI_FWD_RELU>(g, s);
  if (a_kc && b_kc && g.epi == EPI_FWD_LINEAR) return go<true, true, EPI_FWD_LINEAR>(g, s);
  if (a_kc && !b_kc && g.epi == EPI_DX_MASK) return go<true, false, EPI_DX_MASK>(g, s);
  if (!a_kc && !b_kc && g.epi == EPI_DW_UPDATE) return go<false, false, EPI_DW_UPDATE>(g, s);
  return hipErrorInvalidValue;
}

}  // namespace agn
