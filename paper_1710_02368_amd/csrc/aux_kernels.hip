// Bandwidth kernels of the AGN round: softmax cross-entropy with its
// gradient, the fused normalize/commit/pull over the parameters, and small
// helpers (per-worker loss reduction, parameter packing, commit order,
// batch indices).
#include <math.h>

#include "device_common.h"

namespace agn {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Softmax cross-entropy of one mini-batch row per wave (the loss of Eq. 1).
// loss_j = logsumexp(z_j) - z_{j,y_j};  dZ_j = (softmax(z_j) - onehot(y_j)) / m,
// the gradient of the batch-mean loss with respect to the logits.
__global__ __launch_bounds__(256) void softmax_ce_kernel(SoftmaxArgs a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t rg = (int64_t)blockIdx.x * 4 + wave;
  if (rg >= (int64_t)a.n * a.m) return;
  const int k = (int)(rg / a.m), j = (int)(rg % a.m);
  const float* z = a.z + (int64_t)k * a.zstride + (int64_t)j * a.ldz;
  const int64_t t = gather_step(a.g);
  const int label = a.y[batch_row(k, t, a.g.mb, a.g.S, j)];

  float mx = -INFINITY;
  for (int c = lane; c < a.C; c += 64) mx = fmaxf(mx, z[c]);
  mx = wave_max(mx);
  float s = 0.f;
  for (int c = lane; c < a.C; c += 64) s += expf(z[c] - mx);
  s = wave_sum(s);
  const float inv_s = 1.f / s;
  const float inv_m = 1.f / (float)a.m;
  for (int c = lane; c < a.C; c += 64) {
    const float p = expf(z[c] - mx) * inv_s;
    const float d = (p - (c == label ? 1.f : 0.f)) * inv_m;
    const int64_t e = (int64_t)k * a.dstride + (int64_t)j * a.ldd + c;
    if (a.dz_bf16)
      reinterpret_cast<uint16_t*>(a.dz)[e] = f32_to_bf16_rne(d);
    else
      reinterpret_cast<float*>(a.dz)[e] = d;
  }
  if (lane == 0) {
    const float lse = mx + logf(s);
    a.loss[((int64_t)k * a.lam + a.step) * a.m + j] = lse - z[label];
  }
}

// Normalize + commit + pull (Eq. 2; Algorithm 1, Commit and Pull).
// The deltas already carry the 1/lambda normalization (stored by the last
// local step).  In commit order j = 0..n-1, worker k = order[j]:
// c <- c + delta_k;  pulled_k <- c.  Finally central <- c.  Elements are
// independent, so the sequential order per element is exact and needs no
// atomics.  SCALED: c <- c + scale[j] * delta_k, the staleness factor of
// the j-th commit (the DynSGD comparison of Section 4).
//
// Each wave owns EPT runs of 64 float4 (a contiguous 1 KB run of every
// stream per float4 a lane holds), and loads the deltas of CH workers before
// adding and storing them.  The commit reads n+1 and writes n+1 streams at
// once; longer runs per stream and fewer streams in flight keep the HBM
// pages open longer.  NT: streaming stores of the pulled copies and the
// central variable, for rounds whose buffers exceed the last-level cache.
__device__ __forceinline__ u32x2 bf16x4(f32x4 c) {
  u32x2 h;
  h.x = (uint32_t)f32_to_bf16_rne(c.x) | ((uint32_t)f32_to_bf16_rne(c.y) << 16);
  h.y = (uint32_t)f32_to_bf16_rne(c.z) | ((uint32_t)f32_to_bf16_rne(c.w) << 16);
  return h;
}

template <bool NT, class T>
__device__ __forceinline__ void put(T* p, T v) {
  if (NT)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
}

template <bool SCALED, int EPT, int CH, bool NT>
__global__ __launch_bounds__(256) void commit_kernel(CommitArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t n4 = a.count / 4, ps4 = a.pstride / 4;
  const int64_t e0 = wave * 64 * EPT + lane;  // float4 u of this lane: e0 + 64u
  f32x4* __restrict__ central = reinterpret_cast<f32x4*>(a.central);
  f32x4* __restrict__ snap = reinterpret_cast<f32x4*>(a.snap);
  u32x2* __restrict__ snap16 = reinterpret_cast<u32x2*>(a.snap16);
  const f32x4* __restrict__ delta = reinterpret_cast<const f32x4*>(a.delta);
  f32x4 c[EPT];
  bool ok[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    ok[u] = e0 + 64 * u < n4;
    c[u] = ok[u] ? __builtin_nontemporal_load(&central[e0 + 64 * u]) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int j = 0; j < a.n; j += CH) {
    f32x4 d[CH][EPT];
    int64_t ko[CH];  // worker offset of the commit (-1 past the end)
#pragma unroll
    for (int v = 0; v < CH; ++v) {
      ko[v] = j + v < a.n ? (int64_t)a.order[j + v] * ps4 : -1;
#pragma unroll
      for (int u = 0; u < EPT; ++u)
        if (ko[v] >= 0 && ok[u]) d[v][u] = __builtin_nontemporal_load(&delta[ko[v] + e0 + 64 * u]);
    }
#pragma unroll
    for (int v = 0; v < CH; ++v)
#pragma unroll
      for (int u = 0; u < EPT; ++u)
        if (ko[v] >= 0 && ok[u]) {
          if (SCALED)
            c[u] += a.scale[j + v] * d[v][u];
          else
            c[u] += d[v][u];
          const int64_t e = ko[v] + e0 + 64 * u;
          put<NT>(&snap[e], c[u]);
          if (snap16) put<NT>(&snap16[e], bf16x4(c[u]));
        }
  }
#pragma unroll
  for (int u = 0; u < EPT; ++u)
    if (ok[u]) put<NT>(&central[e0 + 64 * u], c[u]);
  if (blockIdx.x == 0 && threadIdx.x == 0) *a.round += 1;
}

// packed (W_0, b_0, W_1, ...) <-> padded internal layout
__device__ __forceinline__ int find_tensor(const PackArgs& pa, int64_t e) {
  int t = 0;
  while (t + 1 < pa.ntensors && e >= pa.t[t + 1].packed_off) ++t;
  return t;
}

__global__ void pack_kernel(PackArgs pa, const float* padded, float* packed) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= pa.P) return;
  const TensorDesc& d = pa.t[find_tensor(pa, e)];
  const int64_t i = e - d.packed_off;
  const int64_t r = i / d.cols, c = i % d.cols;
  packed[e] = padded[d.padded_off + r * d.ld + c];
}

__global__ void unpack_kernel(PackArgs pa, const float* packed, float* padded, uint16_t* padded16,
                              int32_t copies, int64_t pstride) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= pa.P) return;
  const TensorDesc& d = pa.t[find_tensor(pa, e)];
  const int64_t i = e - d.packed_off;
  const int64_t r = i / d.cols, c = i % d.cols;
  const int64_t o = d.padded_off + r * d.ld + c;
  const float v = packed[e];
  for (int k = 0; k < copies; ++k) {
    padded[(int64_t)k * pstride + o] = v;
    if (padded16) padded16[(int64_t)k * pstride + o] = f32_to_bf16_rne(v);
  }
}

// per-worker mean of the per-row losses, accumulated in float64 in a fixed order
__global__ __launch_bounds__(256) void loss_reduce_kernel(const float* loss, int64_t per_worker,
                                                          float* out) {
  __shared__ double part[256];
  const int k = blockIdx.x;
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < per_worker; i += 256) s += (double)loss[(int64_t)k * per_worker + i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[k] = (float)(part[0] / (double)per_worker);
}

struct OrderArg {
  int32_t v[256];
  float sc[256];
};
__global__ void set_order_kernel(OrderArg o, int32_t n, int32_t* dst, float* dst_scale) {
  const int j = threadIdx.x;
  if (j < n) {
    dst[j] = o.v[j];
    if (dst_scale) dst_scale[j] = o.sc[j];
  }
}

__global__ void batch_indices_kernel(int32_t worker, int64_t t, int32_t mb, int64_t S, int64_t* out) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < mb) out[j] = batch_row(worker, t, mb, S, j);
}

__global__ void copy_bf16_kernel(const float* src, uint16_t* dst, int64_t count) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < count) dst[e] = f32_to_bf16_rne(src[e]);
}

// Evaluation of one row per wave: loss = logsumexp(z) - z_y and the
// predicted class argmax z.  Argmax order: a NaN beats any number, a larger
// value beats a smaller one, and among equals (or among NaNs) the lower
// class index wins; the order is total, so the wave reduction gives the
// same class whatever the lanes' pairing.
__device__ __forceinline__ bool beats(float v, int i, float bv, int bi) {
  const bool vn = v != v, bn = bv != bv;
  if (vn != bn) return vn;
  if (vn) return i < bi;
  return v > bv || (v == bv && i < bi);
}

constexpr int EVAL_ROWS_PER_BLOCK = 4;

__global__ __launch_bounds__(256) void eval_rows_kernel(EvalArgs a) {
  __shared__ double lsum[EVAL_ROWS_PER_BLOCK];
  __shared__ double csum[EVAL_ROWS_PER_BLOCK];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * EVAL_ROWS_PER_BLOCK + wave;
  double l = 0.0, ok = 0.0;
  if (row < a.rows) {
    const float* z = a.z + row * a.ldz;
    float mx = -INFINITY, bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int c = lane; c < a.C; c += 64) {
      const float v = z[c];
      mx = fmaxf(mx, v);
      if (beats(v, c, bv, bi)) bv = v, bi = c;
    }
    mx = wave_max(mx);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float ov = __shfl_xor(bv, off, 64);
      const int oi = __shfl_xor(bi, off, 64);
      if (beats(ov, oi, bv, bi)) bv = ov, bi = oi;
    }
    float s = 0.f;
    for (int c = lane; c < a.C; c += 64) s += expf(z[c] - mx);
    s = wave_sum(s);
    const int label = a.y[row];
    const bool in_range = label >= 0 && label < a.C;
    const float loss = in_range ? mx + logf(s) - z[in_range ? label : 0] : NAN;
    l = (double)loss;
    ok = (in_range && bi == label) ? 1.0 : 0.0;
    if (lane == 0) {
      if (a.row_loss) a.row_loss[row] = loss;
      if (a.row_pred) a.row_pred[row] = bi;
    }
  }
  if (lane == 0) {
    lsum[wave] = l;
    csum[wave] = ok;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double ls = 0.0, cs = 0.0;
    for (int w = 0; w < EVAL_ROWS_PER_BLOCK; ++w) ls += lsum[w], cs += csum[w];
    a.part[2 * blockIdx.x] = ls;
    a.part[2 * blockIdx.x + 1] = cs;
  }
}

// acc (=, or += when !first) the column sums of part[blocks][2], each
// thread summing a strided subset in increasing order, then a fixed tree
__global__ __launch_bounds__(256) void eval_reduce_kernel(const double* part, int64_t blocks,
                                                          double* acc, int32_t first) {
  __shared__ double sl[256], sc[256];
  double l = 0.0, c = 0.0;
  for (int64_t b = threadIdx.x; b < blocks; b += 256) l += part[2 * b], c += part[2 * b + 1];
  sl[threadIdx.x] = l;
  sc[threadIdx.x] = c;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      sl[threadIdx.x] += sl[threadIdx.x + w];
      sc[threadIdx.x] += sc[threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    acc[0] = (first ? 0.0 : acc[0]) + sl[0];
    acc[1] = (first ? 0.0 : acc[1]) + sc[0];
  }
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

hipError_t launch_softmax_ce(const SoftmaxArgs& a, hipStream_t s) {
  const int64_t rows = (int64_t)a.n * a.m;
  AGN_LAUNCH(softmax_ce_kernel, dim3(blocks_for(rows, 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

// Commits whose traffic exceeds this stream from HBM (the last-level
// cache of MI355X is 256 MB): longer runs per wave and streaming stores
constexpr double kCommitStreamBytes = 256.0 * 1024 * 1024;

template <bool SCALED, int EPT, int CH, bool NT>
hipError_t commit_go(const CommitArgs& a, hipStream_t s) {
  const int64_t n4 = a.count / 4;
  const int64_t waves = (n4 + 64 * EPT - 1) / (64 * EPT);
  AGN_LAUNCH((commit_kernel<SCALED, EPT, CH, NT>), dim3(blocks_for(waves > 0 ? waves : 1, 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_commit(const CommitArgs& a, hipStream_t s) {
  const double bytes = (8.0 + (a.snap16 ? 2.0 : 0.0)) * (double)(a.n + 1) * (double)a.count;
  const bool stream = bytes > kCommitStreamBytes;
  if (a.scale)
    return stream ? commit_go<true, 2, 2, true>(a, s) : commit_go<true, 1, 8, false>(a, s);
  return stream ? commit_go<false, 2, 2, true>(a, s) : commit_go<false, 1, 8, false>(a, s);
}

hipError_t launch_pack(const PackArgs& pa, const float* padded, float* packed, hipStream_t s) {
  AGN_LAUNCH(pack_kernel, dim3(blocks_for(pa.P, 256)), dim3(256), 0, s, pa, padded, packed);
  return hipGetLastError();
}

hipError_t launch_unpack(const PackArgs& pa, const float* packed, float* padded, uint16_t* padded16,
                         int32_t copies, int64_t pstride, hipStream_t s) {
  AGN_LAUNCH(unpack_kernel, dim3(blocks_for(pa.P, 256)), dim3(256), 0, s, pa, packed, padded,
                     padded16, copies, pstride);
  return hipGetLastError();
}

hipError_t launch_loss_reduce(const float* loss, int32_t n, int64_t per_worker, float* out,
                              hipStream_t s) {
  AGN_LAUNCH(loss_reduce_kernel, dim3(n), dim3(256), 0, s, loss, per_worker, out);
  return hipGetLastError();
}

hipError_t launch_set_order(const int32_t* host_order, const float* host_scale, int32_t n,
                            int32_t* dev_order, float* dev_scale, hipStream_t s) {
  OrderArg o;
  for (int j = 0; j < 256; ++j) {
    o.v[j] = j < n ? host_order[j] : 0;
    o.sc[j] = (j < n && host_scale) ? host_scale[j] : 1.f;
  }
  AGN_LAUNCH(set_order_kernel, dim3(1), dim3(256), 0, s, o, n, dev_order,
                     host_scale ? dev_scale : nullptr);
  return hipGetLastError();
}

hipError_t launch_batch_indices(int32_t worker, int64_t t, int32_t mb, int64_t S, int64_t* out,
                                hipStream_t s) {
  AGN_LAUNCH(batch_indices_kernel, dim3(blocks_for(mb, 256)), dim3(256), 0, s, worker, t, mb,
                     S, out);
  return hipGetLastError();
}

int64_t eval_blocks(int64_t rows) { return (rows + EVAL_ROWS_PER_BLOCK - 1) / EVAL_ROWS_PER_BLOCK; }

hipError_t launch_eval_rows(const EvalArgs& a, hipStream_t s) {
  AGN_LAUNCH(eval_rows_kernel, dim3((unsigned)eval_blocks(a.rows)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_eval_reduce(const double* part, int64_t blocks, double* acc, int32_t first,
                              hipStream_t s) {
  AGN_LAUNCH(eval_reduce_kernel, dim3(1), dim3(256), 0, s, part, blocks, acc, first);
  return hipGetLastError();
}

hipError_t launch_copy_bf16(const float* src, uint16_t* dst, int64_t count, hipStream_t s) {
  AGN_LAUNCH(copy_bf16_kernel, dim3(blocks_for(count, 256)), dim3(256), 0, s, src, dst, count);
  return hipGetLastError();
}

}  // namespace agn
