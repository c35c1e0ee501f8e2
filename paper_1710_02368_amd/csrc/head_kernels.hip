// Output layer of the local step for few classes (C <= 32): one fused
// kernel for the logits, the softmax cross-entropy with its gradient and
// the output layer's input gradient, and one kernel for the output layer's
// weight gradient with the SGD update.  These layers are skinny (C rows or
// C columns), so tile products leave most of a matrix-core tile empty; the
// work is vector FMAs from LDS-resident weights.
//
// Per row j of a worker's mini-batch (softmax cross-entropy, Eq. 1's loss):
//   z_c = b_c + sum_i H[j][i] W[c][i]
//   loss_j = logsumexp(z) - z_{y_j};   dZ[j][c] = (softmax(z)_c - [c == y_j]) / m
//   dZ_prev[j][i] = (sum_c dZ[j][c] W[c][i]) * [H[j][i] > 0]
// Weight gradient (summed over the m rows) fused with the update:
//   W[c][i] <- W[c][i] - eta * sum_j dZ[j][c] H[j][i];  b[c] <- b[c] - eta * sum_j dZ[j][c]
// The evaluation variant (EVAL) computes the same logits for rows of a
// held-out set and, instead of the gradients, the loss, the predicted class
// and the block's partial sums.
#include <math.h>

#include "device_common.h"
#include "head_dw_unit.h"

namespace agn {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int HEAD_WAVE_ROWS = 1;                  // rows a wave processes together
constexpr int HEAD_DMAX = 2048;                     // hidden width limit
// dynamic LDS a workgroup may use (160 KB per CU on gfx950, less the
// kernel's static LDS)
constexpr int HEAD_LDS_CAP = 160 * 1024 - 2048;

// Rows of W in LDS trimmed to the width (instances whose padded rows would
// take more than half of the cap), and the floats per row
__host__ __device__ constexpr bool head_trim(int cmax, int q4) { return cmax * 256 * q4 * 4 > HEAD_LDS_CAP / 2; }
__host__ __device__ constexpr int head_pitch(int cmax, int q4, int d) {
  return head_trim(cmax, q4) ? (d + 3) & ~3 : 256 * q4;
}

// Argmax order of the evaluation: a NaN beats any number, a larger value a
// smaller one, and among equals (or NaNs) the lower class index wins.
__device__ __forceinline__ bool beats_h(float v, int i, float bv, int bi) {
  const bool vn = v != v, bn = bv != bv;
  if (vn != bn) return vn;
  if (vn) return i < bi;
  return v > bv || (v == bv && i < bi);
}

constexpr int EVAL_WAVE_ROWS = 4;                   // rows per wave in the evaluation variant
__host__ __device__ constexpr int head_rows(bool eval) { return 4 * (eval ? EVAL_WAVE_ROWS : HEAD_WAVE_ROWS); }
// Waves per row: the training variant splits each row's columns over two
// waves when each lane holds at least two groups of them (its latency is
// one row per wave; the evaluation variant runs many rows per wave instead)
__host__ __device__ constexpr int head_split(int q4, bool eval) { return !eval && q4 >= 2 ? 2 : 1; }

// LDS: W as CMAX rows (zeros outside C x d), then b.  Lane l owns the
// columns 4l + 256q .. +3 of every row, for the groups q of its wave's share
// (all Q4 of them, or half when SP = 2 waves share a row): it keeps them of
// its wave's rows of H in registers (all loaded at once, 16 bytes at a time
// when the rows allow it) and reads W and writes the input gradient 16 bytes
// at a time.  A row holds the 256*Q4 columns the lanes span (padding zero),
// so the loops are static and branch-free -- except where that would take
// more than half of a compute unit's LDS (head_trim): there a row holds d
// rounded up to 4 floats, and a group past the row's end reads the row's
// last four columns instead (its H is zero and its outputs are not stored).
// At d = 2000, C <= 10 that makes 80 KB, two workgroups per compute unit.
template <int CMAX, int Q4, bool EVAL>
__global__ __launch_bounds__(256 * head_split(Q4, EVAL)) void head_kernel(HeadArgs a) {
  extern __shared__ float smem[];
  __shared__ double epart[EVAL ? 8 : 1];
  constexpr int SP = head_split(Q4, EVAL), QH = Q4 / SP, NTH = 256 * SP;
  __shared__ float xch[SP > 1 ? 4 * SP * CMAX : 1];  // the halves' logits
  constexpr int LW = 256 * Q4;
  constexpr int WR = EVAL ? EVAL_WAVE_ROWS : HEAD_WAVE_ROWS;  // rows per wave
  constexpr int RB = 4 * WR;                                     // rows per workgroup
  const int tid = threadIdx.x, lane = tid & 63, wave = (tid >> 6) / SP, half = (tid >> 6) % SP;
  const int qb = QH * half;  // this wave's first column group
  const int blocks_per_worker = (a.m + RB - 1) / RB;
  const int k = blockIdx.x / blocks_per_worker;
  const int r0 = (blockIdx.x % blocks_per_worker) * RB;
  constexpr bool TRIM = head_trim(CMAX, Q4);
  const int d = a.d, C = a.C, pitch = head_pitch(CMAX, Q4, d);
  const float* W = a.w + (int64_t)k * a.pstride;
  const float* bias = a.b + (int64_t)k * a.pstride;
  float* Ws = smem;
  float* bs = smem + CMAX * pitch;
  const int64_t t = gather_step(a.g);

  // rows of this wave: issue every load of H (and the labels) before
  // anything waits
  int jr[WR];
  int label[WR];
  const float* hp[WR];
  f32x4 hv[WR][QH];
#pragma unroll
  for (int r = 0; r < WR; ++r) {
    jr[r] = r0 + wave * WR + r;
    const int j = jr[r] < a.m ? jr[r] : a.m - 1;   // rows past m compute a copy, store nothing
    label[r] = EVAL ? a.y[j] : a.y[batch_row(k, t, a.g.mb, a.g.S, j)];
    hp[r] = a.gather ? a.h + batch_row(k, t, a.g.mb, a.g.S, j) * a.ldh
                     : a.h + (int64_t)k * a.hstride + (int64_t)j * a.ldh;
#pragma unroll
    for (int q = 0; q < QH; ++q) {
      const int i = 4 * lane + 256 * (qb + q);
      if (a.vec) {  // (d a multiple of 4: a group lies inside the row or past it)
        hv[r][q] = *reinterpret_cast<const f32x4*>(hp[r] + (i < d ? i : d - 4));
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) hv[r][q][e] = hp[r][i + e < d ? i + e : d - 1];
      }
    }
  }
  // W and b into LDS, float4 at a time (W rows are 16-byte aligned).  All
  // loads first, unconditionally (row and column clamped into the padded W:
  // rows are ldw >= d floats, ldw a multiple of 8), then the LDS writes with
  // the parts outside C x d zeroed: the loads are in flight together
  if constexpr (TRIM) {
    // thread tid takes the chunks tid + NTH*u of every row (at most the
    // pitch's: NTH*CPT >= LW/4)
    constexpr int CPT = (LW / 4 + NTH - 1) / NTH;
    float4 wv[CMAX][CPT];
#pragma unroll
    for (int c = 0; c < CMAX; ++c)
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const int i = min(4 * (tid + NTH * u), (int)a.ldw - 4);
        wv[c][u] = *reinterpret_cast<const float4*>(W + (int64_t)min(c, C - 1) * a.ldw + i);
      }
#pragma unroll
    for (int c = 0; c < CMAX; ++c)
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const int i = 4 * (tid + NTH * u);
        if (i >= pitch) continue;
        float4 v = wv[c][u];
        if (c >= C || i >= d) v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (i + 1 >= d) v.y = 0.f;
        if (i + 2 >= d) v.z = 0.f;
        if (i + 3 >= d) v.w = 0.f;
        *reinterpret_cast<float4*>(Ws + c * pitch + i) = v;
      }
  } else {
    // the padded CMAX x LW block in row-major chunks, spread over the threads
    constexpr int NW4 = CMAX * LW / 4, WIT = (NW4 + NTH - 1) / NTH;
    float4 wv[WIT];
#pragma unroll
    for (int it = 0; it < WIT; ++it) {
      const int e4 = min(tid + NTH * it, NW4 - 1);
      const int c = min(e4 / (LW / 4), C - 1), i = min(4 * (e4 % (LW / 4)), (int)a.ldw - 4);
      wv[it] = *reinterpret_cast<const float4*>(W + (int64_t)c * a.ldw + i);
    }
#pragma unroll
    for (int it = 0; it < WIT; ++it) {
      const int e4 = tid + NTH * it;
      if (NW4 % NTH != 0 && e4 >= NW4) break;
      const int c = e4 / (LW / 4), i = 4 * (e4 % (LW / 4));
      float4 v = wv[it];
      if (c >= C || i >= d) v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (i + 1 >= d) v.y = 0.f;
      if (i + 2 >= d) v.z = 0.f;
      if (i + 3 >= d) v.w = 0.f;
      *reinterpret_cast<float4*>(Ws + c * LW + i) = v;
    }
  }
  {
    const float bv = bias[min(tid, C - 1)];  // (unconditional: clamped into the bias)
    if (tid < CMAX) bs[tid] = tid < C ? bv : 0.f;
  }
#pragma unroll
  for (int r = 0; r < WR; ++r)
#pragma unroll
    for (int q = 0; q < QH; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) hv[r][q][e] = 4 * lane + 256 * (qb + q) + e < d ? hv[r][q][e] : 0.f;
  __syncthreads();

  // this lane's column group q in a row of W (clamped into a trimmed row)
  const auto wcol = [&](int q) {
    const int i = 4 * lane + 256 * (qb + q);
    return TRIM ? min(i, pitch - 4) : i;
  };

  // logits: lane-partial dot products, then one wave reduction per (row, class)
  float p[WR][CMAX];
#pragma unroll
  for (int r = 0; r < WR; ++r)
#pragma unroll
    for (int c = 0; c < CMAX; ++c) p[r][c] = 0.f;
#pragma unroll
  for (int q = 0; q < QH; ++q) {
#pragma unroll
    for (int c = 0; c < CMAX; ++c) {
      const f32x4 w = *reinterpret_cast<const f32x4*>(Ws + c * pitch + wcol(q));
#pragma unroll
      for (int r = 0; r < WR; ++r)
#pragma unroll
        for (int e = 0; e < 4; ++e) p[r][c] += hv[r][q][e] * w[e];
    }
  }
  if constexpr (SP == 1) {
#pragma unroll
    for (int r = 0; r < WR; ++r)
#pragma unroll
      for (int c = 0; c < CMAX; ++c) p[r][c] = wave_sum(p[r][c]) + bs[c];
  } else {
    // each wave's partial logits to LDS; then both waves of a row add the
    // halves in the same order and hold the same logits
    static_assert(WR == 1, "one row per wave pair");
#pragma unroll
    for (int c = 0; c < CMAX; ++c) p[0][c] = wave_sum(p[0][c]);
    if (lane < CMAX) {
      float mine = 0.f;
#pragma unroll
      for (int c = 0; c < CMAX; ++c) mine = lane == c ? p[0][c] : mine;
      xch[(wave * SP + half) * CMAX + lane] = mine;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < CMAX; ++c) {
      float z = xch[wave * SP * CMAX + c];
#pragma unroll
      for (int h = 1; h < SP; ++h) z += xch[(wave * SP + h) * CMAX + c];
      p[0][c] = z + bs[c];
    }
  }

  if constexpr (EVAL) {
    // loss, predicted class and the block's partial sums (fixed order)
    double ls = 0.0, cs = 0.0;
#pragma unroll
    for (int r = 0; r < WR; ++r) {
      const int lb = label[r];
      float mx = -INFINITY, bv = -INFINITY;
      int bi = 0x7fffffff;
#pragma unroll
      for (int c = 0; c < CMAX; ++c) {
        if (c < C) {
          mx = fmaxf(mx, p[r][c]);
          if (beats_h(p[r][c], c, bv, bi)) bv = p[r][c], bi = c;
        }
      }
      float s = 0.f, zy = 0.f;
#pragma unroll
      for (int c = 0; c < CMAX; ++c) {
        s += c < C ? expf(p[r][c] - mx) : 0.f;
        zy = c == lb ? p[r][c] : zy;
      }
      const bool in_range = lb >= 0 && lb < C;
      const float loss = in_range ? mx + logf(s) - zy : NAN;
      if (jr[r] < a.m) {
        if (lane == 0) {
          if (a.row_loss) a.row_loss[jr[r]] = loss;
          if (a.row_pred) a.row_pred[jr[r]] = bi;
        }
        ls += (double)loss;
        cs += (in_range && bi == lb) ? 1.0 : 0.0;
      }
    }
    if (lane == 0) {
      epart[2 * wave] = ls;
      epart[2 * wave + 1] = cs;
    }
    __syncthreads();
    if (tid == 0) {
      double l = 0.0, c = 0.0;
      for (int w = 0; w < 4; ++w) l += epart[2 * w], c += epart[2 * w + 1];
      a.part[2 * blockIdx.x] = l;
      a.part[2 * blockIdx.x + 1] = c;
    }
    return;
  }

  // softmax cross-entropy per row; p becomes dZ
  const float inv_m = 1.f / (float)a.m;
#pragma unroll
  for (int r = 0; r < WR; ++r) {
    const int lb = label[r];
    float mx = -INFINITY;
#pragma unroll
    for (int c = 0; c < CMAX; ++c) mx = c < C ? fmaxf(mx, p[r][c]) : mx;
    float s = 0.f, zy = 0.f;
#pragma unroll
    for (int c = 0; c < CMAX; ++c) {
      const float e = c < C ? expf(p[r][c] - mx) : 0.f;
      zy = c == lb ? p[r][c] : zy;
      s += e;
      p[r][c] = e;
    }
    const float inv_s = 1.f / s;
#pragma unroll
    for (int c = 0; c < CMAX; ++c)
      p[r][c] = c < C ? (p[r][c] * inv_s - (c == lb ? 1.f : 0.f)) * inv_m : 0.f;
    if (jr[r] < a.m && half == 0) {
      float* dzo = a.dz + (int64_t)k * a.dzstride + (int64_t)jr[r] * a.lddz;
      float mine = 0.f;
#pragma unroll
      for (int c = 0; c < CMAX; ++c) mine = lane == c ? p[r][c] : mine;
      if (lane < C) dzo[lane] = mine;
      if (lane == 0) a.loss[((int64_t)k * a.lam + a.step) * a.m + jr[r]] = mx + logf(s) - zy;
    }
  }

  // input gradient of the output layer, masked by the ReLU of H_{L-1}
  if (a.dprev) {
    // a trimmed row's pitch made opaque, so that the logits' LDS addresses
    // are recomputed here rather than held in registers across the softmax
    int pitch2 = pitch;
    if constexpr (TRIM) asm volatile("" : "+s"(pitch2));
#pragma unroll
    for (int q = 0; q < QH; ++q) {
      const int i = 4 * lane + 256 * (qb + q);
      f32x4 acc[WR];
#pragma unroll
      for (int r = 0; r < WR; ++r) acc[r] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < CMAX; ++c) {
        const f32x4 w = *reinterpret_cast<const f32x4*>(Ws + c * pitch2 + wcol(q));
#pragma unroll
        for (int r = 0; r < WR; ++r)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[r][e] += p[r][c] * w[e];
      }
#pragma unroll
      for (int r = 0; r < WR; ++r) {
        if (jr[r] < a.m && i < d) {
          float* dp = a.dprev + (int64_t)k * a.hstride + (int64_t)jr[r] * a.ldh;
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = hv[r][q][e] > 0.f ? acc[r][e] : 0.f;
          if (a.vec) {
            *reinterpret_cast<f32x4*>(dp + i) = v;
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (i + e < d) dp[i + e] = v[e];
          }
        }
      }
    }
  }
}

// Output-layer weight gradient + update on its own: one unit per workgroup.
template <int CMAX>
__global__ __launch_bounds__(64 * HDW_WAVES) void head_dw_kernel(HeadDwArgs a) {
  __shared__ float smem[hdw_smem_floats<CMAX>()];
  head_dw_unit<CMAX>(a, blockIdx.x, smem);
}

}  // namespace

static int head_cmax(int C) { return C <= 10 ? 10 : C <= 16 ? 16 : 32; }
static int head_q4(int d) { return d <= 256 ? 1 : d <= 512 ? 2 : d <= 1024 ? 4 : 8; }

size_t head_lds_bytes(int C, int d) {
  const int cm = head_cmax(C);
  return ((size_t)cm * head_pitch(cm, head_q4(d), d) + cm) * sizeof(float);
}

// 16-byte accesses to the rows of H (and of the input gradient): d and the
// row pitches multiples of 4 floats, the bases 16-byte aligned
static bool head_vec(const HeadArgs& a) {
  const auto al = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  return a.d % 4 == 0 && a.ldh % 4 == 0 && (a.gather || a.hstride % 4 == 0) && al(a.h) &&
         (!a.dprev || al(a.dprev));
}

template <int CM, int QM, bool EVAL>
static hipError_t head_go(const HeadArgs& a, hipStream_t s, bool prepare) {
  const size_t lds = head_lds_bytes(a.C, a.d);
  if (prepare) {  // (the cap, not lds: contexts of other widths share the instance)
    if (lds <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute((const void*)head_kernel<CM, QM, EVAL>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, HEAD_LDS_CAP);
  }
  const int blocks = a.n * ((a.m + head_rows(EVAL) - 1) / head_rows(EVAL));
  HeadArgs v = a;
  v.vec = head_vec(a);
  AGN_LAUNCH((head_kernel<CM, QM, EVAL>), dim3(blocks), dim3(256 * head_split(QM, EVAL)), lds, s, v);
  return hipGetLastError();
}

template <int CM, bool EVAL>
static hipError_t head_dispatch_q(const HeadArgs& a, hipStream_t s, bool prepare) {
  switch (head_q4(a.d)) {
    case 1: return head_go<CM, 1, EVAL>(a, s, prepare);
    case 2: return head_go<CM, 2, EVAL>(a, s, prepare);
    case 4: return head_go<CM, 4, EVAL>(a, s, prepare);
    default: return head_go<CM, 8, EVAL>(a, s, prepare);
  }
}

template <bool EVAL>
static hipError_t head_dispatch(const HeadArgs& a, hipStream_t s, bool prepare) {
  switch (head_cmax(a.C)) {
    case 10: return head_dispatch_q<10, EVAL>(a, s, prepare);
    case 16: return head_dispatch_q<16, EVAL>(a, s, prepare);
    default: return head_dispatch_q<32, EVAL>(a, s, prepare);
  }
}

// The fused output layer applies when C <= 32, the hidden width is at most
// 2048 and the padded W fits in the LDS a workgroup may use (160 KB per CU
// on gfx950; beyond 64 KB the kernel's dynamic-LDS limit is raised first).
bool head_prepare(int C, int d) {
  if (C > 32 || d > HEAD_DMAX) return false;
  if (head_lds_bytes(C, d) > HEAD_LDS_CAP) return false;
  HeadArgs a{};
  a.C = C;
  a.d = d;
  return head_dispatch<false>(a, nullptr, true) == hipSuccess &&
         head_dispatch<true>(a, nullptr, true) == hipSuccess;
}

hipError_t launch_head(const HeadArgs& a, hipStream_t s) { return head_dispatch<false>(a, s, false); }

int64_t head_eval_blocks(int64_t rows) { return (rows + head_rows(true) - 1) / head_rows(true); }

hipError_t launch_head_eval(const HeadArgs& a, hipStream_t s) { return head_dispatch<true>(a, s, false); }

hipError_t launch_head_dw(const HeadDwArgs& a, hipStream_t s) {
  const int blocks = hdw_units(a);
  switch (head_cmax(a.C)) {
    case 10: AGN_LAUNCH(head_dw_kernel<10>, dim3(blocks), dim3(64 * HDW_WAVES), 0, s, a); break;
    case 16: AGN_LAUNCH(head_dw_kernel<16>, dim3(blocks), dim3(64 * HDW_WAVES), 0, s, a); break;
    default: AGN_LAUNCH(head_dw_kernel<32>, dim3(blocks), dim3(64 * HDW_WAVES), 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace agn
