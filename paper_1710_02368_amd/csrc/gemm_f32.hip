// Batched float32 products of the local SGD step on the fp32 matrix cores
// of gfx950 (v_mfma_f32_32x32x2_f32), one launch per layer for all workers.
//
// A workgroup of 4 waves owns a 64x64 output tile of one worker; each wave
// owns a 32x32 quarter held in 16 accumulator registers per lane.  K is
// consumed in steps of 32 through double-buffered LDS tiles, with the next
// step's global loads in flight while the current step's 16 MFMAs run.
//
// Operands are read as stored, with no transposition pass:
//   forward          H_{l+1} = relu(H_l W_l^T + b_l)   A = H_l [m][d_l]      (K-contiguous)
//                                                      B = W_l [d_{l+1}][d_l] (K-contiguous)
//   input gradient   dZ_l = (dZ_{l+1} W_l) * [H_l > 0]  A = dZ  (K-contiguous)
//                                                      B = W_l (N-contiguous)
//   weight gradient  dW_l = dZ_{l+1}^T H_l             A = dZ  (M-contiguous)
//                                                      B = H_l (N-contiguous)
// For the first layer the rows of H_0 are gathered straight from the data
// set by the mini-batch index (no copy of the batch is made).  The weight-
// gradient product carries the SGD update of Algorithm 1 in its epilogue,
// so gradients are never written to memory: W <- W - eta*dW (and the bias
// from the column sums of dZ, which the row-block's first tile forms from
// the same LDS tiles).  On a round's last step the epilogue stores the
// normalized displacement (W_new - W_pulled) / lambda, which equals the
// accumulated update a / lambda of Algorithm 1.
#include "device_common.h"

namespace agn {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 64, BN = 64, BK = 32, NT = 256;
constexpr int KC_LD = BK + 4;            // LDS row stride of a K-contiguous tile
constexpr int KS_LD = 64 + 4;            // LDS row stride of a K-strided tile
constexpr int KS_SKEW = 32;              // extra offset of K-strided rows 16..31
constexpr int KC_TILE = 64 * KC_LD;
constexpr int KS_TILE = BK * KS_LD + KS_SKEW;

// LDS offset of element (k, outer) of a K-strided tile.  Rows k and k+16 are
// read by the two halves of a wave in the same instruction; the skew puts
// them 32 banks apart.
__device__ __forceinline__ int ks_off(int k, int o) { return k * KS_LD + o + (k >> 4) * KS_SKEW; }

__device__ __forceinline__ float4 load4(const float* p, int valid, int vec) {
  if (valid >= 4 && vec) return *reinterpret_cast<const float4*>(p);
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (valid > 0) v.x = p[0];
  if (valid > 1) v.y = p[1];
  if (valid > 2) v.z = p[2];
  if (valid > 3) v.w = p[3];
  return v;
}

// Global->register staging of one operand tile.
// K-contiguous tile: 64 outer rows x 32 k; thread loads rows tid/8 and
// tid/8+32 at k offset 4*(tid%8).  K-strided tile: 32 k rows x 64 outer;
// thread loads k rows tid/16 and tid/16+16 at outer offset 4*(tid%16).
template <bool KC>
struct TileLoader {
  const float* rowp[2];  // KC: fixed row pointers (null past the edge)
  const float* base;     // KS: worker base
  int64_t ld;
  int outer0, outer_n, K;
  int vec, gather;
  int64_t worker, t, mb, S;

  __device__ void init(const Operand& op, const Gather& g, int64_t w, int o0, int on, int k, int tid) {
    base = reinterpret_cast<const float*>(op.ptr) + w * op.wstride;
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
        const int o = o0 + tid / 8 + 32 * p;
        int64_t r = o;
        if (gather && o < on) r = batch_row(worker, t, mb, S, o);
        rowp[p] = o < on ? base + r * ld : nullptr;
      }
    }
  }

  __device__ void load(int k0, int tid, float4 (&v)[2]) const {
    if (KC) {
      const int kk = k0 + 4 * (tid % 8);
#pragma unroll
      for (int p = 0; p < 2; ++p)
        v[p] = rowp[p] ? load4(rowp[p] + kk, K - kk, vec) : make_float4(0.f, 0.f, 0.f, 0.f);
    } else {
      const int cc = outer0 + 4 * (tid % 16);
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int kr = k0 + tid / 16 + 16 * p;
        if (kr < K) {
          int64_t r = gather ? batch_row(worker, t, mb, S, kr) : kr;
          v[p] = load4(base + r * ld + cc, outer_n - cc, vec);
        } else {
          v[p] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
    }
  }

  __device__ static void store(float* lds, int tid, const float4 (&v)[2]) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      if (KC) {
        *reinterpret_cast<float4*>(lds + (tid / 8 + 32 * p) * KC_LD + 4 * (tid % 8)) = v[p];
      } else {
        *reinterpret_cast<float4*>(lds + ks_off(tid / 16 + 16 * p, 4 * (tid % 16))) = v[p];
      }
    }
  }
};

// Fragment of one wave for 16 MFMAs: lane (i = lane%32, h = lane/32)
// supplies element k = 16h + s of its row/column i for MFMA number s, so
// that MFMA s contracts over k in {s, 16+s}.
template <bool KC>
__device__ __forceinline__ void read_frag(const float* lds, int outer_off, int li, int lh, float (&f)[16]) {
  if (KC) {
    const float* p = lds + (outer_off + li) * KC_LD + lh * 16;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float4 v = *reinterpret_cast<const float4*>(p + 4 * q);
      f[4 * q] = v.x;
      f[4 * q + 1] = v.y;
      f[4 * q + 2] = v.z;
      f[4 * q + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int s = 0; s < 16; ++s) f[s] = lds[ks_off(lh * 16 + s, outer_off + li)];
  }
}

constexpr int LDS_FLOATS = 2 * (KC_TILE > KS_TILE ? KC_TILE : KS_TILE);

// One 64x64 output tile (logical tile id `logical`) of one product.
// lds_a / lds_b: LDS_FLOATS each (two buffers of one operand tile).
template <bool A_KC, bool B_KC, int EPI>
__device__ __forceinline__ void gemm_tile(const GemmArgs& g, const int logical, float* lds_a_base,
                                          float* lds_b_base) {
  constexpr int TA = A_KC ? KC_TILE : KS_TILE;
  constexpr int TB_ = B_KC ? KC_TILE : KS_TILE;
#define LDS_A(i) (lds_a_base + (i) * TA)
#define LDS_B(i) (lds_b_base + (i) * TB_)

  const int tid = threadIdx.x;
  const int tm = (g.M + BM - 1) / BM, tn = (g.N + BN - 1) / BN;
  const int worker = logical / (tm * tn);
  const int rem = logical % (tm * tn);
  const int tile_n = rem / tm, tile_m = rem % tm;
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  TileLoader<A_KC> la;
  TileLoader<B_KC> lb;
  la.init(g.a, g.g, worker, m0, g.M, g.K, tid);
  lb.init(g.b, g.g, worker, n0, g.N, g.K, tid);

  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 31, lh = lane >> 5;

  // bias gradient (weight-gradient epilogue): the first column tile of each
  // row block sums its dZ tile columns (A is dZ^T, stored K-strided)
  const bool do_bias = (EPI == EPI_DW_UPDATE) && tile_n == 0 && tid < 64;
  float bsum = 0.f;

  // operands of the epilogue, loaded before the K loop so that their latency
  // hides behind it: lane holds D[i][j], j = lane%32,
  // i = 8*(r/4) + 4*(lane/32) + r%4
  const int col = n0 + wn * 32 + li;
  const int64_t wo = (int64_t)worker * g.pstride;
  float pre[16], pre2[16];
  if (EPI == EPI_DX_MASK || EPI == EPI_DW_UPDATE) {
    const float* mk = EPI == EPI_DX_MASK ? reinterpret_cast<const float*>(g.mask) + (int64_t)worker * g.mstride
                                         : nullptr;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = m0 + wm * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
      const bool ok = row < g.M && col < g.N;
      if (EPI == EPI_DX_MASK) {
        pre[r] = ok ? mk[(int64_t)row * g.ldm + col] : 0.f;
      } else {
        const int64_t e = wo + (int64_t)row * g.ldw + col;
        pre[r] = ok ? g.w_src[e] : 0.f;
        pre2[r] = (ok && g.last) ? g.w_snap[e] : 0.f;
      }
    }
  }

  // two independent accumulation chains (even / odd MFMA of each step)
  f32x16 acc0, acc1;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    acc0[r] = 0.f;
    acc1[r] = 0.f;
  }

  // K loop: the next tile's global loads are in flight while the current
  // tile's 16 MFMAs run; LDS is double-buffered, one barrier per step.
  const int nk = (g.K + BK - 1) / BK;
  float4 va[2], vb[2];
  la.load(0, tid, va);
  lb.load(0, tid, vb);
  TileLoader<A_KC>::store(LDS_A(0), tid, va);
  TileLoader<B_KC>::store(LDS_B(0), tid, vb);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      la.load((kt + 1) * BK, tid, va);
      lb.load((kt + 1) * BK, tid, vb);
    }
    float af[16], bf[16];
    read_frag<A_KC>(LDS_A(cur), wm * 32, li, lh, af);
    read_frag<B_KC>(LDS_B(cur), wn * 32, li, lh, bf);
#pragma unroll
    for (int s = 0; s < 16; s += 2) {
      acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(af[s], bf[s], acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(af[s + 1], bf[s + 1], acc1, 0, 0, 0);
    }
    if (do_bias) {
#pragma unroll 8
      for (int k = 0; k < BK; ++k) bsum += LDS_A(cur)[ks_off(k, tid)];
    }
    if (kt + 1 < nk) {
      TileLoader<A_KC>::store(LDS_A(cur ^ 1), tid, va);
      TileLoader<B_KC>::store(LDS_B(cur ^ 1), tid, vb);
    }
    __syncthreads();
  }
  f32x16 acc = acc0 + acc1;

  if (EPI == EPI_FWD_RELU || EPI == EPI_FWD_LINEAR) {
    if (col < g.N) {
      float* out = reinterpret_cast<float*>(g.out) + (int64_t)worker * g.ostride;
      const float bcol = g.bias[(int64_t)worker * g.bstride + col];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (row < g.M) {
          float v = acc[r] + bcol;
          if (EPI == EPI_FWD_RELU) v = v > 0.f ? v : 0.f;
          out[(int64_t)row * g.ldo + col] = v;
        }
      }
    }
  } else if (EPI == EPI_DX_MASK) {
    if (col < g.N) {
      float* out = reinterpret_cast<float*>(g.out) + (int64_t)worker * g.ostride;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (row < g.M) out[(int64_t)row * g.ldo + col] = pre[r] > 0.f ? acc[r] : 0.f;
      }
    }
  } else {  // EPI_DW_UPDATE: rows are output units o, columns input units i
    const AdamCoef ac = g.adam.on ? adam_coef(g.g, g.adam) : AdamCoef{1.f, 1.f};
    if (col < g.N) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (row < g.M) {
          const int64_t e = wo + (int64_t)row * g.ldw + col;
          const float step = g.adam.on ? adam_dir(acc[r], g.adam.mw, g.adam.vw, e, g.adam, ac) : acc[r];
          const float nw = pre[r] - g.eta * step;
          g.w_dst[e] = g.last ? (nw - pre2[r]) / g.lam : nw;
        }
      }
    }
    if (do_bias) {
      const int o = m0 + tid;
      if (o < g.M) {
        const int64_t e = wo + o;
        const float step = g.adam.on ? adam_dir(bsum, g.adam.mb, g.adam.vb, e, g.adam, ac) : bsum;
        const float nb = g.b_src[e] - g.eta * step;
        g.b_dst[e] = g.last ? (nb - g.b_snap[e]) / g.lam : nb;
      }
    }
  }
}

#undef LDS_A
#undef LDS_B

__host__ __device__ inline int tiles_of(const GemmArgs& g) { return ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN) * g.batch; }

template <bool A_KC, bool B_KC, int EPI>
__global__ __launch_bounds__(NT) void gemm_f32_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) float lds_a[LDS_FLOATS];
  __shared__ __attribute__((aligned(16))) float lds_b[LDS_FLOATS];
  gemm_tile<A_KC, B_KC, EPI>(g, xcd_remap(blockIdx.x, tiles_of(g)), lds_a, lds_b);
}

// The backward products of one layer in one launch: the input-gradient tiles
// (long K) first, then the weight-gradient tiles.  Both read dZ_{l+1}; the
// first reads W_l from the step's source parameters, the second writes the
// destination parameters, so they are independent.  Each range is laid out
// over the XCDs on its own (the first range is padded to a multiple of 8
// workgroups, the pad workgroups exit at once).
__global__ __launch_bounds__(NT) void gemm_f32_bwd_kernel(GemmArgs dx, GemmArgs dw, int n1, int n1pad) {
  __shared__ __attribute__((aligned(16))) float lds_a[LDS_FLOATS];
  __shared__ __attribute__((aligned(16))) float lds_b[LDS_FLOATS];
  const int pid = blockIdx.x;
  if (pid < n1pad) {
    if (pid < n1) gemm_tile<true, false, EPI_DX_MASK>(dx, xcd_remap(pid, n1), lds_a, lds_b);
  } else {
    const int p2 = pid - n1pad;
    gemm_tile<false, false, EPI_DW_UPDATE>(dw, xcd_remap(p2, tiles_of(dw)), lds_a, lds_b);
  }
}

}  // namespace

template <bool A_KC, bool B_KC, int EPI>
static hipError_t go(const GemmArgs& g, hipStream_t s) {
  AGN_LAUNCH((gemm_f32_kernel<A_KC, B_KC, EPI>), dim3(tiles_of(g)), dim3(NT), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_gemm_f32_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s) {
  if (dx.epi != EPI_DX_MASK || dw.epi != EPI_DW_UPDATE) return hipErrorInvalidValue;
  if (gemm_f32_strip_ok(dx, dw)) return launch_gemm_f32_strip_bwd(dx, dw, s);
  if (gemm_f32_dl_ok(1, 0, dx) && gemm_f32_dl_ok(0, 0, dw)) return launch_gemm_f32_dl_bwd(dx, dw, s);
  const int n1 = tiles_of(dx), n1pad = (n1 + kNumXcd - 1) / kNumXcd * kNumXcd;
  AGN_LAUNCH(gemm_f32_bwd_kernel, dim3(n1pad + tiles_of(dw)), dim3(NT), 0, s, dx, dw, n1, n1pad);
  return hipGetLastError();
}

hipError_t launch_gemm_f32(int a_kc, int b_kc, const GemmArgs& g, hipStream_t s) {
  if (gemm_f32_dl_ok(a_kc, b_kc, g)) return launch_gemm_f32_dl(a_kc, b_kc, g, s);
  if (a_kc && b_kc && g.epi == EPI_FWD_RELU) return go<true, true, EPI_FWD_RELU>(g, s);
  if (a_kc && b_kc && g.epi == EPI_FWD_LINEAR) return go<true, true, EPI_FWD_LINEAR>(g, s);
  if (a_kc && !b_kc && g.epi == EPI_DX_MASK) return go<true, false, EPI_DX_MASK>(g, s);
  if (!a_kc && !b_kc && g.epi == EPI_DW_UPDATE) return go<false, false, EPI_DW_UPDATE>(g, s);
  return hipErrorInvalidValue;
}

}  // namespace agn
