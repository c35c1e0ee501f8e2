// Internal declarations shared by the host code and the kernels of libagn.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace agn {

// Kernel timing: while set, the next kernel launched on this thread records
// these two events at its own start and end (hipExtLaunchKernel), so that a
// timed launch measures the kernel and not the gaps around it.  Set by the
// timing bracket of the host API, taken (and cleared) by AGN_LAUNCH.
struct LaunchEvents {
  hipEvent_t start, stop;
};
extern thread_local LaunchEvents g_launch_events;

#define AGN_LAUNCH(kernel, grid, block, shmem, stream, ...)                                              \
  do {                                                                                                  \
    if (::agn::g_launch_events.start) {                                                                 \
      const ::agn::LaunchEvents ev_ = ::agn::g_launch_events;                                           \
      ::agn::g_launch_events = ::agn::LaunchEvents{nullptr, nullptr};                                   \
      hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ev_.start, ev_.stop, 0, __VA_ARGS__);  \
    } else {                                                                                            \
      hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);                              \
    }                                                                                                   \
  } while (0)

// An operand of a batched product, as the matrix is stored in memory.
struct Operand {
  const void* ptr;  // element (0,0) of worker 0's matrix
  int64_t ld;       // elements between consecutive stored rows
  int64_t wstride;  // elements between consecutive workers' matrices (0: shared)
  int32_t gather;   // 1: stored rows are data-set rows picked by the batch index
  int32_t vec;      // 1: ld % 4 == 0 and ptr 16-byte aligned (vector loads allowed)
  int32_t padded = 0;  // 1: the elements between a row's last column and ld are zero
};

// Batch index of a gathered operand: worker k, local step t = round*lam + step,
// row j -> k*S + ((t*m + j) mod S)  (FetchNextMiniBatch, Algorithm 1).
struct Gather {
  const int64_t* round;  // device round counter
  int32_t lam;
  int32_t step;
  int32_t mb;
  int64_t S;
};

enum Epilogue : int32_t {
  EPI_FWD_RELU = 0,    // out = relu(acc + bias)
  EPI_FWD_LINEAR = 1,  // out = acc + bias (logits)
  EPI_DX_MASK = 2,     // out = acc * (mask > 0)
  EPI_DW_UPDATE = 3,   // W_dst = W_src - eta*acc, b_dst = b_src - eta*colsum(dZ)
                       // (last step: store (new - snapshot) / lambda instead)
};

// Adam as the local rule (weight-gradient epilogues): moment estimates of
// the layer's weights (mw, vw) and bias (mb, vb), laid out like the
// parameters ([n][P_pad], worker stride pstride), updated in place; the
// bias corrections use the worker's local step t = round*lambda + step + 1.
struct AdamArgs {
  float* mw;
  float* vw;
  float* mb;
  float* vb;
  float beta1, beta2, eps;
  int32_t on;
};

struct GemmArgs {
  int32_t M, N, K, batch;
  Operand a;  // A[M][K]: stored [M][K] when a_kc, else [K][M]
  Operand b;  // B[K][N]: stored [N][K] when b_kc, else [K][N]
  Gather g;
  int32_t epi;
  // forward / input-gradient output
  void* out;
  int64_t ldo, ostride;
  const void* mask;
  int64_t ldm, mstride;
  const float* bias;
  int64_t bstride;
  // weight-gradient update (one layer of every worker; stride pstride)
  const float* w_src;
  float* w_dst;
  const float* w_snap;
  const float* b_src;
  float* b_dst;
  const float* b_snap;
  uint16_t* w_dst16;  // bf16 shadow of the updated weights (bf16 mode, not last step)
  int64_t ldw, pstride;
  float eta, lam;
  int32_t last;
  const float* zero;  // a zeroed page (operand reads past an edge)
  AdamArgs adam;      // EPI_DW_UPDATE: Adam instead of SGD when adam.on
  float* sink = nullptr;  // at least 256 writable bytes that absorb stores past an edge (never read)
};

// launchers (return hipError_t of the launch)
hipError_t launch_gemm_f32(int a_kc, int b_kc, const GemmArgs& g, hipStream_t s);
hipError_t launch_gemm_bf16(int a_kc, int b_kc, const GemmArgs& g, hipStream_t s);
// input-gradient (EPI_DX_MASK) and weight-gradient (EPI_DW_UPDATE) products of
// one layer in one launch
hipError_t launch_gemm_f32_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s);
hipError_t launch_gemm_bf16_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s);
// direct global->LDS variants of the float32 products (used when both
// operands qualify, see gemm_f32_dl_ok)
bool gemm_f32_dl_ok(int a_kc, int b_kc, const GemmArgs& g);
hipError_t launch_gemm_f32_dl(int a_kc, int b_kc, const GemmArgs& g, hipStream_t s);
hipError_t launch_gemm_f32_dl_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s);
// the backward launch of a float32 hidden layer as column strips of its
// weights (input gradient and weight gradient + update sharing each weight
// block in LDS), used when gemm_f32_strip_ok
bool gemm_f32_strip_ok(const GemmArgs& dx, const GemmArgs& dw);
hipError_t launch_gemm_f32_strip_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s);
// the first layer's weight gradient + update as 64-row strips of W_0 (the
// dZ_1 strip in LDS, the gathered data rows streamed), used when
// gemm_f32_strip_dw_ok
bool gemm_f32_strip_dw_ok(const GemmArgs& dw);
hipError_t launch_gemm_f32_strip_dw(const GemmArgs& dw, hipStream_t s);
struct HeadDwArgs;
// the first layer's direct-load weight gradient with the output layer's
// weight gradient + update (C <= 10) folded into the same launch
bool gemm_f32_dl_dw_head_ok(const GemmArgs& g, const HeadDwArgs& h);
hipError_t launch_gemm_f32_dl_dw_head(const GemmArgs& g, const HeadDwArgs& h, hipStream_t s);
// direct global->LDS variants of the bf16 products (used when the operands
// and outputs qualify, see gemm_bf16_dl_ok)
bool gemm_bf16_dl_ok(int a_kc, int b_kc, const GemmArgs& g);
hipError_t launch_gemm_bf16_dl(int a_kc, int b_kc, const GemmArgs& g, hipStream_t s);
hipError_t launch_gemm_bf16_dl_bwd(const GemmArgs& dx, const GemmArgs& dw, hipStream_t s);

struct SoftmaxArgs {
  const float* z;      // logits [n][m][ldz]
  int64_t ldz, zstride;
  const int32_t* y;    // labels of the data set
  Gather g;
  int32_t n, m, C;
  void* dz;            // output gradient [n][m][ldd] (float or bf16)
  int64_t ldd, dstride;
  int32_t dz_bf16;
  float* loss;         // [n][lam][m] per-row losses
  int32_t lam, step;
};
hipError_t launch_softmax_ce(const SoftmaxArgs& a, hipStream_t s);

// Fused output layer (C <= 32): logits, softmax cross-entropy, output
// gradient dZ_L and the previous layer's input gradient dZ_{L-1}.
struct HeadArgs {
  const float* h;          // H_{L-1} [n][m][ldh] (or the data set, gathered, when L == 1)
  int64_t ldh, hstride;
  int32_t gather;
  const float* w;          // W_{L-1} of worker 0 in the step's source parameters
  const float* b;          // b_{L-1}
  int64_t ldw, pstride;
  const int32_t* y;
  Gather g;
  int32_t n, m, d, C;
  float* dz;               // dZ_L [n][m][lddz]
  int64_t lddz, dzstride;
  float* dprev;            // dZ_{L-1}, same layout as h (null when L == 1)
  float* loss;             // [n][lam][m]
  int32_t lam, step;
  // evaluation variant (n = 1, rows not gathered, y = the rows' labels)
  float* row_loss;         // [m] or null
  int32_t* row_pred;       // [m] or null
  double* part;            // [2 * head_eval_blocks(m)]
  int32_t vec;             // (set by the launch: rows of h and dprev allow 16-byte accesses)
};
struct HeadDwArgs {        // output-layer weight gradient + update (M = C <= 32)
  const float* h;
  int64_t ldh, hstride;
  int32_t gather;
  Gather g;
  const float* dz;
  int64_t lddz, dzstride;
  int32_t n, m, d, C;
  const float* w_src;
  float* w_dst;
  const float* w_snap;
  const float* b_src;
  float* b_dst;
  const float* b_snap;
  int64_t ldw, pstride;
  float eta, lam;
  int32_t last;
  AdamArgs adam;
};
bool head_prepare(int C, int d);
hipError_t launch_head(const HeadArgs& a, hipStream_t s);
hipError_t launch_head_dw(const HeadDwArgs& a, hipStream_t s);
int64_t head_eval_blocks(int64_t rows);
hipError_t launch_head_eval(const HeadArgs& a, hipStream_t s);

struct CommitArgs {
  float* central;          // [P_pad]
  float* snap;             // [n][P_pad] pulled copies (written)
  const float* delta;      // [n][P_pad] normalized deltas of the round
  uint16_t* snap16;        // bf16 shadow of the pulled copies (or null)
  const int32_t* order;    // device, n entries
  const float* scale;      // device, n factors by commit position (null: unscaled commits)
  int64_t* round;          // device round counter (incremented)
  int64_t pstride;         // P_pad
  int64_t count;           // elements to process (P_pad)
  int32_t n;
};
hipError_t launch_commit(const CommitArgs& a, hipStream_t s);

struct TensorDesc {  // one parameter tensor: rows x cols, padded row stride ld
  int64_t packed_off, padded_off, ld;
  int32_t rows, cols;
};
struct PackArgs {
  TensorDesc t[2 * 16];
  int32_t ntensors;
  int64_t P;
};
hipError_t launch_pack(const PackArgs& pa, const float* padded, float* packed, hipStream_t s);
hipError_t launch_unpack(const PackArgs& pa, const float* packed, float* padded,
                         uint16_t* padded16, int32_t copies, int64_t pstride, hipStream_t s);
hipError_t launch_loss_reduce(const float* loss, int32_t n, int64_t per_worker, float* out,
                              hipStream_t s);
// writes the round's commit order and, when dev_scale is not null, the
// commits' scale factors (host_scale) to the device
hipError_t launch_set_order(const int32_t* host_order, const float* host_scale, int32_t n,
                            int32_t* dev_order, float* dev_scale,
                            hipStream_t s);
hipError_t launch_batch_indices(int32_t worker, int64_t t, int32_t mb, int64_t S, int64_t* out,
                                hipStream_t s);
hipError_t launch_copy_bf16(const float* src, uint16_t* dst, int64_t count, hipStream_t s);

// Evaluation rows: per-row softmax cross-entropy and argmax of the logits,
// with per-block partial sums for a fixed-order total.
struct EvalArgs {
  const float* z;      // logits [rows][ldz]
  int64_t ldz;
  const int32_t* y;    // labels of these rows
  int64_t rows;
  int32_t C;
  float* row_loss;     // [rows] or null
  int32_t* row_pred;   // [rows] or null
  double* part;        // [2 * blocks]: loss sum, correct count of each block
};
int64_t eval_blocks(int64_t rows);
hipError_t launch_eval_rows(const EvalArgs& a, hipStream_t s);
// acc[0..1] (= or +=) the sums of part[0..2*blocks) in a fixed order
hipError_t launch_eval_reduce(const double* part, int64_t blocks, double* acc, int32_t first,
                              hipStream_t s);

// host-side He-normal initial parameters (packed layout)
void he_normal_init(const int32_t* dims, int32_t L, uint64_t seed, float* packed);

}  // namespace agn
