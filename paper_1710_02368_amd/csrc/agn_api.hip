// C ABI of libagn: context management, argument validation, the device
// memory plan and the launch sequence of one AGN round.
//
// Device state of a context (float32 unless noted; P_pad = padded
// parameter count, every tensor 256-byte aligned, weight rows padded to a
// multiple of 8 elements):
//   central   [P_pad]           the central variable (Eq. 2)
//   snap      [n][P_pad]        each worker's last pulled copy (start of its round)
//   buf[0,1]  [n][P_pad]        ping-pong parameters of the local steps; on the
//                               last step the normalized delta (theta_lambda -
//                               theta_0) / lambda is stored in place of theta
//   *16       bf16 shadows of snap/buf (bf16 mode: the matrix-product operands)
//   H[l]      [n][m][ld_l]      hidden activations after ReLU, l = 1..L-1
//   Z         [n][m][ld_L]      logits
//   dZ[l]     [n][m][ld_l]      gradients of the batch loss w.r.t. layer inputs, l = 1..L
//   loss      [n][lambda][m]    per-row cross-entropy of the last round
// Step i of a round reads its weights from src = (i == 0 ? snap : buf[(i-1)%2])
// and writes dst = buf[i%2]; reading and writing different buffers lets the
// input-gradient and weight-gradient products of one layer run in either
// order.  Nothing is allocated after agn_create.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "agn_internal.h"
#include "../../include/agn.h"

using namespace agn;

// Workspace of agn_evaluate_noalloc: one array per device, held until the
// process ends.  In host code its name stands for a host-side shadow, not a
// device address: every host use goes through the address that
// hipGetSymbolAddress returns for the current device (scratch_address).
static __device__ __align__(256) unsigned char scratch[AGN_NOALLOC_SCRATCH_BYTES];

struct TimingSlot {
  int enabled = 0;
  std::vector<hipEvent_t> ev;  // start/end pairs
  size_t used = 0;             // pairs recorded
  int64_t dropped = 0;
};

struct agn_ctx {
  int L = 0, m = 0, dtype = 0, n = 0, lam = 0;
  int dims[AGN_MAX_LAYERS + 1] = {};
  float eta = 0.f;
  int64_t P = 0, P_pad = 0;
  int64_t woff[AGN_MAX_LAYERS] = {}, boff[AGN_MAX_LAYERS] = {}, ldw[AGN_MAX_LAYERS] = {};
  int64_t lda[AGN_MAX_LAYERS + 1] = {};  // row stride of activations of width d_l
  float* central = nullptr;
  float* snap = nullptr;
  float* buf[2] = {nullptr, nullptr};
  uint16_t* snap16 = nullptr;
  uint16_t* buf16[2] = {nullptr, nullptr};
  void* H[AGN_MAX_LAYERS + 1] = {};
  void* dZ[AGN_MAX_LAYERS + 1] = {};
  float* Z = nullptr;
  float* loss = nullptr;
  int32_t* order = nullptr;
  int64_t* round_dev = nullptr;
  float* zero = nullptr;  // 4 KB of zeros
  float* sink = nullptr;  // 4 KB that absorbs stores past a matrix edge (never read)
  int64_t rounds = 0;
  int64_t N_fixed = -1;
  hipStream_t stream = nullptr;       // caller's stream (all work is ordered on it)
  hipStream_t cap_stream = nullptr;   // private stream used only to capture the round graph
  hipGraph_t graph = nullptr;
  hipGraphExec_t graph_exec = nullptr;
  const void* graph_x = nullptr;      // data the captured graph was recorded with
  const void* graph_y = nullptr;
  int64_t graph_n = -1;
  int device = 0;
  int use_head = 0;  // fused output-layer kernels (few classes)
  int head_dw_folded = 0;  // local steps of the last round that folded the output layer's update into the first layer's launch
  int normalize = 1; // commit a / lambda (AGN) or a (DOWNPOUR with local exploration)
  int staleness_scaling = 0;           // scale each commit by 1 / (tau + 1)
  float* commit_scale = nullptr;       // device, n factors of the current round
  std::vector<int64_t> pulled_version; // per worker: commits applied when it last pulled
  std::vector<int64_t> last_staleness; // per commit position of the last round
  int64_t version = 0;                 // commits applied so far
  int optimizer = AGN_OPT_SGD;
  float beta1 = 0.f, beta2 = 0.f, adam_eps = 0.f;
  float* mom_m = nullptr;  // Adam moment estimates [n][P_pad] (allocated on selection)
  float* mom_v = nullptr;
  // evaluation workspace (allocated by the first agn_evaluate call)
  void* ev_h[2] = {nullptr, nullptr};  // activations of EVAL_CHUNK rows, ping-pong
  float* ev_z = nullptr;               // logits of EVAL_CHUNK rows (unfused output layer)
  uint16_t* ev_w16 = nullptr;          // bf16 copy of the central variable
  double* ev_part = nullptr;           // per-block partial sums of one chunk
  double* ev_acc = nullptr;            // loss sum and correct count over all rows
  int64_t eval_N = 0;                  // rows of the last agn_evaluate call
  unsigned char* scratch = nullptr;    // this device's scratch array (agn_evaluate_noalloc)
  int last_committer = 0;              // worker that committed last (its pulled copy is the central variable)
  int have_deltas = 0;                 // the delta buffers hold the last round's deltas (not after agn_set_state)
  int capturing = 0;
  int untimed = 0;                     // launch without timing events (agn_evaluate_noalloc)
  hipStream_t ls = nullptr;           // stream the launch sequence is enqueued on
  int poisoned = 0;
  std::string err;
  PackArgs pack{};
  TimingSlot timing[AGN_K_NUM];
  std::vector<void*> allocs;
};

static std::string g_create_err;

namespace agn {
thread_local LaunchEvents g_launch_events{nullptr, nullptr};
}

namespace {

inline int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

int fail(agn_ctx* c, int code, const std::string& msg) {
  if (c) {
    c->err = msg;
    if (code == AGN_EHIP) c->poisoned = 1;
  } else {
    g_create_err = msg;
  }
  return code;
}

#define HIP_CHECK(ctx, expr)                                                                \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return fail((ctx), AGN_EHIP, std::string(#expr) + ": " + hipGetErrorString(e_));      \
  } while (0)

void drop_graph(agn_ctx* c) {
  if (c->graph_exec) (void)hipGraphExecDestroy(c->graph_exec);
  if (c->graph) (void)hipGraphDestroy(c->graph);
  c->graph_exec = nullptr;
  c->graph = nullptr;
  c->graph_x = c->graph_y = nullptr;
  c->graph_n = -1;
}

void free_all(agn_ctx* c) {
  drop_graph(c);
  if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
  c->cap_stream = nullptr;
  for (void* p : c->allocs) (void)hipFree(p);
  c->allocs.clear();
  for (auto& t : c->timing)
    for (hipEvent_t e : t.ev) (void)hipEventDestroy(e);
}

template <class T>
hipError_t dalloc(agn_ctx* c, T** p, int64_t count) {
  void* q = nullptr;
  hipError_t e = hipMalloc(&q, (size_t)std::max<int64_t>(count, 1) * sizeof(T));
  if (e != hipSuccess) return e;
  c->allocs.push_back(q);
  *p = reinterpret_cast<T*>(q);
  return hipSuccess;
}

// Bracket a launch of class `cls` with events when timing is enabled.
template <class F>
hipError_t timed(agn_ctx* c, int cls, F&& launch) {
  TimingSlot& t = c->timing[cls];
  if (!t.enabled || c->capturing || c->untimed) return launch();
  if (t.used >= (1u << 15)) {
    ++t.dropped;
    return launch();
  }
  if (2 * t.used + 2 > t.ev.size()) {
    for (int i = 0; i < 2; ++i) {
      hipEvent_t e;
      hipError_t r = hipEventCreate(&e);
      if (r != hipSuccess) return r;
      t.ev.push_back(e);
    }
  }
  // the class's one kernel records the events at its own start and end
  g_launch_events = LaunchEvents{t.ev[2 * t.used], t.ev[2 * t.used + 1]};
  hipError_t r = launch();
  const bool taken = g_launch_events.start == nullptr;
  g_launch_events = LaunchEvents{nullptr, nullptr};
  if (r != hipSuccess) return r;
  if (!taken) return hipErrorInvalidValue;  // (every timed class launches a kernel)
  ++t.used;
  return hipSuccess;
}

int check_ctx(agn_ctx* c) {
  if (!c) return fail(nullptr, AGN_EINVAL, "null context");
  if (c->poisoned) return fail(c, AGN_ESTATE, "context poisoned by an earlier HIP error: " + c->err);
  return AGN_OK;
}

int set_device(agn_ctx* c) {
  HIP_CHECK(c, hipSetDevice(c->device));
  return AGN_OK;
}

// The device address of `scratch` on device `dev` (current), looked up once
// per device: each device holds its own copy of the array.
std::mutex g_scratch_mu;
std::vector<std::pair<int, unsigned char*>> g_scratch_addr;

hipError_t scratch_address(int dev, unsigned char** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  for (const auto& e : g_scratch_addr)
    if (e.first == dev) {
      *out = e.second;
      return hipSuccess;
    }
  void* ptr = nullptr;
  const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  g_scratch_addr.emplace_back(dev, static_cast<unsigned char*>(ptr));
  *out = static_cast<unsigned char*>(ptr);
  return hipSuccess;
}

// One local step of every worker: forward, softmax cross-entropy, backward
// with the SGD update fused into the weight-gradient products.
// Adam arguments of layer l's weight-gradient epilogue (off when SGD)
AdamArgs adam_args(const agn_ctx* c, int l) {
  AdamArgs a{};
  if (c->optimizer != AGN_OPT_ADAM) return a;
  a.mw = c->mom_m + c->woff[l];
  a.vw = c->mom_v + c->woff[l];
  a.mb = c->mom_m + c->boff[l];
  a.vb = c->mom_v + c->boff[l];
  a.beta1 = c->beta1;
  a.beta2 = c->beta2;
  a.eps = c->adam_eps;
  a.on = 1;
  return a;
}

int enqueue_step(agn_ctx* c, const agn_data* d, int64_t S, int step) {
  const int L = c->L, m = c->m, n = c->n;
  const bool bf = c->dtype == AGN_BF16;
  const bool last = step == c->lam - 1;
  const float* src = step == 0 ? c->snap : c->buf[(step - 1) & 1];
  float* dst = c->buf[step & 1];
  const uint16_t* src16 = bf ? (step == 0 ? c->snap16 : c->buf16[(step - 1) & 1]) : nullptr;
  uint16_t* dst16 = bf ? c->buf16[step & 1] : nullptr;
  const int64_t ps = c->P_pad;

  Gather gath{c->round_dev, c->lam, step, m, S};
  const int64_t d0 = c->dims[0];
  const int x_vec = (d0 % (bf ? 8 : 4) == 0) && ((uintptr_t)d->x % 16 == 0);
  Operand xop{d->x, d0, 0, 1, x_vec};
  auto gemm = [&](int a_kc, int b_kc, const GemmArgs& g) {
    return bf ? launch_gemm_bf16(a_kc, b_kc, g, c->ls) : launch_gemm_f32(a_kc, b_kc, g, c->ls);
  };

  // dW_l = dZ_{l+1}^T H_l fused with the update of W_l and b_l
  auto dw_args = [&](int l) {
    const int64_t dz_ld = c->lda[l + 1], dz_st = (int64_t)m * c->lda[l + 1];
    GemmArgs w{};
    w.M = c->dims[l + 1];
    w.N = c->dims[l];
    w.K = m;
    w.batch = n;
    w.a = Operand{c->dZ[l + 1], dz_ld, dz_st, 0, 1};
    w.b = l == 0 ? xop : Operand{c->H[l], c->lda[l], (int64_t)m * c->lda[l], 0, 1};
    w.g = gath;
    w.epi = EPI_DW_UPDATE;
    w.w_src = src + c->woff[l];
    w.w_dst = dst + c->woff[l];
    w.w_snap = c->snap + c->woff[l];
    w.b_src = src + c->boff[l];
    w.b_dst = dst + c->boff[l];
    w.b_snap = c->snap + c->boff[l];
    w.w_dst16 = (bf && !last) ? dst16 + c->woff[l] : nullptr;
    w.ldw = c->ldw[l];
    w.pstride = ps;
    w.eta = c->eta;
    w.lam = c->normalize ? (float)c->lam : 1.f;  // divisor of the committed delta
    w.last = last;
    w.zero = c->zero;
    w.sink = c->sink;
    w.adam = adam_args(c, l);
    return w;
  };
  HeadDwArgs hdw{};
  bool fold_head_dw = false;
  // the first layer's weight gradient as 64-row strips of W_0
  const bool strip_dw = !bf && gemm_f32_strip_dw_ok(dw_args(0));

  // forward: hidden layers with bias + ReLU, then the logits (unless the
  // fused output-layer kernel computes them)
  const int fwd_layers = c->use_head ? L - 1 : L;
  for (int l = 0; l < fwd_layers; ++l) {
    GemmArgs g{};
    g.M = m;
    g.N = c->dims[l + 1];
    g.K = c->dims[l];
    g.batch = n;
    g.a = l == 0 ? xop : Operand{c->H[l], c->lda[l], (int64_t)m * c->lda[l], 0, 1};
    g.b = bf ? Operand{src16 + c->woff[l], c->ldw[l], ps, 0, 1} : Operand{src + c->woff[l], c->ldw[l], ps, 0, 1};
    g.g = gath;
    g.epi = l < L - 1 ? EPI_FWD_RELU : EPI_FWD_LINEAR;
    g.out = l < L - 1 ? c->H[l + 1] : (void*)c->Z;
    g.ldo = c->lda[l + 1];
    g.ostride = (int64_t)m * c->lda[l + 1];
    g.bias = src + c->boff[l];
    g.bstride = ps;
    g.zero = c->zero;
    HIP_CHECK(c, timed(c, AGN_K_FWD, [&] { return gemm(1, 1, g); }));
  }

  if (c->use_head) {
    // logits + softmax cross-entropy + dZ_L + dZ_{L-1}, then dW_{L-1} + update
    const bool first = L == 1;
    const float* hin = first ? (const float*)d->x : (const float*)c->H[L - 1];
    const int64_t ldh = first ? d0 : c->lda[L - 1];
    const int64_t hst = first ? 0 : (int64_t)m * c->lda[L - 1];
    HeadArgs h{};
    h.h = hin;
    h.ldh = ldh;
    h.hstride = hst;
    h.gather = first;
    h.w = src + c->woff[L - 1];
    h.b = src + c->boff[L - 1];
    h.ldw = c->ldw[L - 1];
    h.pstride = ps;
    h.y = d->y;
    h.g = gath;
    h.n = n;
    h.m = m;
    h.d = c->dims[L - 1];
    h.C = c->dims[L];
    h.dz = (float*)c->dZ[L];
    h.lddz = c->lda[L];
    h.dzstride = (int64_t)m * c->lda[L];
    h.dprev = first ? nullptr : (float*)c->dZ[L - 1];
    h.loss = c->loss;
    h.lam = c->lam;
    h.step = step;
    HIP_CHECK(c, timed(c, AGN_K_OUTPUT, [&] { return launch_head(h, c->ls); }));
    HeadDwArgs& w = hdw;
    w.h = hin;
    w.ldh = ldh;
    w.hstride = hst;
    w.gather = first;
    w.g = gath;
    w.dz = (const float*)c->dZ[L];
    w.lddz = c->lda[L];
    w.dzstride = (int64_t)m * c->lda[L];
    w.n = n;
    w.m = m;
    w.d = c->dims[L - 1];
    w.C = c->dims[L];
    w.w_src = src + c->woff[L - 1];
    w.w_dst = dst + c->woff[L - 1];
    w.w_snap = c->snap + c->woff[L - 1];
    w.b_src = src + c->boff[L - 1];
    w.b_dst = dst + c->boff[L - 1];
    w.b_snap = c->snap + c->boff[L - 1];
    w.ldw = c->ldw[L - 1];
    w.pstride = ps;
    w.eta = c->eta;
    w.lam = c->normalize ? (float)c->lam : 1.f;  // divisor of the committed delta
    w.last = last;
    w.adam = adam_args(c, L - 1);
    // with a first-layer weight gradient on the persistent direct-load path,
    // the output layer's update rides in that launch (it touches nothing the
    // layers in between read or write).  The strip schedule of the first
    // layer leaves it a launch of its own: inside the strips each unit's
    // chain of dependent loads ran ahead of the strip's work in every
    // workgroup (0.8 ms per round at 40 workers against 0.4 for the launch)
    fold_head_dw = !bf && !strip_dw && L >= 2 && gemm_f32_dl_dw_head_ok(dw_args(0), w);
    if (!fold_head_dw) HIP_CHECK(c, timed(c, AGN_K_OUTPUT_DW, [&] { return launch_head_dw(w, c->ls); }));
  } else {
    // softmax cross-entropy: per-row loss and the output gradient dZ_L
    SoftmaxArgs s{};
    s.z = c->Z;
    s.ldz = c->lda[L];
    s.zstride = (int64_t)m * c->lda[L];
    s.y = d->y;
    s.g = gath;
    s.n = n;
    s.m = m;
    s.C = c->dims[L];
    s.dz = c->dZ[L];
    s.ldd = c->lda[L];
    s.dstride = (int64_t)m * c->lda[L];
    s.dz_bf16 = bf;
    s.loss = c->loss;
    s.lam = c->lam;
    s.step = step;
    HIP_CHECK(c, timed(c, AGN_K_OUTPUT, [&] { return launch_softmax_ce(s, c->ls); }));
  }

  // backward, last layer first (the fused output layer already did layer L-1):
  // per layer one launch with the input-gradient product (l >= 1) and the
  // weight-gradient product fused with the update
  for (int l = c->use_head ? L - 2 : L - 1; l >= 0; --l) {
    const int64_t dz_ld = c->lda[l + 1], dz_st = (int64_t)m * c->lda[l + 1];
    const GemmArgs w = dw_args(l);
    if (l >= 1) {  // dZ_l = (dZ_{l+1} W_l) * [H_l > 0]
      GemmArgs x{};
      x.M = m;
      x.N = c->dims[l];
      x.K = c->dims[l + 1];
      x.batch = n;
      x.a = Operand{c->dZ[l + 1], dz_ld, dz_st, 0, 1, 1};  // (gradient rows: zero padding, never written)
      x.b = bf ? Operand{src16 + c->woff[l], c->ldw[l], ps, 0, 1} : Operand{src + c->woff[l], c->ldw[l], ps, 0, 1};
      x.g = gath;
      x.epi = EPI_DX_MASK;
      x.out = c->dZ[l];
      x.ldo = c->lda[l];
      x.ostride = (int64_t)m * c->lda[l];
      x.mask = c->H[l];
      x.ldm = c->lda[l];
      x.mstride = (int64_t)m * c->lda[l];
      x.zero = c->zero;
      HIP_CHECK(c, timed(c, AGN_K_BWD, [&] {
        return bf ? launch_gemm_bf16_bwd(x, w, c->ls) : launch_gemm_f32_bwd(x, w, c->ls);
      }));
    } else if (strip_dw) {
      HIP_CHECK(c, timed(c, AGN_K_DW_FIRST, [&] { return launch_gemm_f32_strip_dw(w, c->ls); }));
    } else if (fold_head_dw) {
      HIP_CHECK(c, timed(c, AGN_K_DW_FIRST, [&] { return launch_gemm_f32_dl_dw_head(w, hdw, c->ls); }));
    } else {
      HIP_CHECK(c, timed(c, AGN_K_DW_FIRST, [&] { return gemm(0, 0, w); }));
    }
  }
  if (step == 0) c->head_dw_folded = 0;
  c->head_dw_folded += fold_head_dw ? 1 : 0;
  (void)dst16;
  return AGN_OK;
}

// lambda local steps of every worker, then normalize + commit + pull
int enqueue_round(agn_ctx* c, const agn_data* d) {
  const int64_t S = d->num_samples / c->n;
  for (int i = 0; i < c->lam; ++i)
    if (int r = enqueue_step(c, d, S, i)) return r;
  CommitArgs ca{};
  ca.central = c->central;
  ca.snap = c->snap;
  ca.delta = c->buf[(c->lam - 1) & 1];
  ca.snap16 = c->snap16;
  ca.order = c->order;
  ca.scale = c->staleness_scaling ? c->commit_scale : nullptr;
  ca.round = c->round_dev;
  ca.pstride = c->P_pad;
  ca.count = c->P_pad;
  ca.n = c->n;
  HIP_CHECK(c, timed(c, AGN_K_COMMIT, [&] { return launch_commit(ca, c->ls); }));
  return AGN_OK;
}

// Rows the evaluation takes through its forward pass at a time: large
// enough that each product of a 1000-wide layer spreads over several
// workgroups per compute unit.
constexpr int64_t EVAL_CHUNK = 8192;

// The evaluation's own buffers (nothing a round uses), allocated once.
int eval_alloc(agn_ctx* c) {
  if (c->ev_acc) return AGN_OK;
  const bool bf = c->dtype == AGN_BF16;
  int64_t wmax = 0;
  for (int l = 1; l < c->L; ++l) wmax = std::max(wmax, c->lda[l]);
  const int64_t act = bf ? 2 : 4;
  const int64_t blocks = std::max(eval_blocks(EVAL_CHUNK), head_eval_blocks(EVAL_CHUNK));
  // (a failed call keeps what it got; the next call allocates the rest)
  bool ok = true;
  for (int i = 0; ok && i < 2 && wmax > 0; ++i) {
    char* p = nullptr;
    if (!c->ev_h[i]) ok = dalloc(c, &p, EVAL_CHUNK * wmax * act) == hipSuccess, c->ev_h[i] = p;
  }
  if (ok && !c->use_head && !c->ev_z) ok = dalloc(c, &c->ev_z, EVAL_CHUNK * c->lda[c->L]) == hipSuccess;
  if (ok && bf && !c->ev_w16) ok = dalloc(c, &c->ev_w16, c->P_pad) == hipSuccess;
  if (ok && !c->ev_part) ok = dalloc(c, &c->ev_part, 2 * blocks) == hipSuccess;
  double* acc = nullptr;
  if (ok) ok = dalloc(c, &acc, 2) == hipSuccess;
  if (!ok) return fail(c, AGN_ENOMEM, "cannot allocate the evaluation workspace");
  c->ev_acc = acc;  // (set last: marks the workspace complete)
  return AGN_OK;
}

// Buffers of one evaluation: activations of `chunk` rows (ping-pong, the
// widest hidden layer), their logits (unfused output layer), the bf16
// operands of the central variable (bf16 contexts), per-block partial sums
// of one chunk and the float64 totals.
struct EvalSpace {
  void* h[2];
  float* z;
  const uint16_t* w16;
  double* part;
  double* acc;
  int64_t chunk;
};

// Bytes of an EvalSpace for `rows` rows (each buffer 256-byte aligned), and
// the buffers when base != nullptr.
int64_t eval_space_bytes(const agn_ctx* c, int64_t rows, unsigned char* base, EvalSpace* ws) {
  const bool bf = c->dtype == AGN_BF16;
  int64_t wmax = 0;
  for (int l = 1; l < c->L; ++l) wmax = std::max(wmax, c->lda[l]);
  const int64_t act = bf ? 2 : 4;
  const int64_t blocks = std::max(eval_blocks(rows), head_eval_blocks(rows));
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    const int64_t at = off;
    off += round_up(std::max<int64_t>(bytes, 1), 256);
    return base ? base + at : nullptr;
  };
  unsigned char* acc = take(2 * sizeof(double));
  unsigned char* part = take(2 * blocks * sizeof(double));
  unsigned char* h0 = wmax > 0 ? take(rows * wmax * act) : nullptr;
  unsigned char* h1 = wmax > 0 ? take(rows * wmax * act) : nullptr;
  unsigned char* z = c->use_head ? nullptr : take(rows * c->lda[c->L] * 4);
  if (ws) {
    ws->h[0] = h0;
    ws->h[1] = h1;
    ws->z = reinterpret_cast<float*>(z);
    ws->part = reinterpret_cast<double*>(part);
    ws->acc = reinterpret_cast<double*>(acc);
    ws->chunk = rows;
    ws->w16 = nullptr;
  }
  return off;
}

// The central variable's forward pass over data->x, ws.chunk rows at a
// time: the hidden layers' products (bias + ReLU), then either the fused
// output-layer kernel (logits, loss, prediction) or the logits product and
// the per-row kernel; per-chunk partial sums are folded into ws.acc in row
// order.
int enqueue_eval(agn_ctx* c, const agn_data* d, float* row_loss, int32_t* row_pred, const EvalSpace& ws) {
  const int L = c->L;
  const bool bf = c->dtype == AGN_BF16;
  const int64_t N = d->num_samples, d0 = c->dims[0];
  const int64_t xes = bf ? 2 : 4;
  const Gather rows_as_stored{c->round_dev, c->lam, 0, c->m, 1};  // (no gathered operand)
  const int products = c->use_head ? L - 1 : L;
  for (int64_t r0 = 0; r0 < N; r0 += ws.chunk) {
    const int32_t rows = (int32_t)std::min(ws.chunk, N - r0);
    const void* x = static_cast<const char*>(d->x) + r0 * d0 * xes;
    const int x_vec = (d0 % (bf ? 8 : 4) == 0) && ((uintptr_t)x % 16 == 0);
    for (int l = 0; l < products; ++l) {
      GemmArgs g{};
      g.M = rows;
      g.N = c->dims[l + 1];
      g.K = c->dims[l];
      g.batch = 1;
      g.a = l == 0 ? Operand{x, d0, 0, 0, x_vec} : Operand{ws.h[(l - 1) & 1], c->lda[l], 0, 0, 1};
      g.b = bf ? Operand{ws.w16 + c->woff[l], c->ldw[l], 0, 0, 1}
               : Operand{c->central + c->woff[l], c->ldw[l], 0, 0, 1};
      g.g = rows_as_stored;
      g.epi = l < L - 1 ? EPI_FWD_RELU : EPI_FWD_LINEAR;
      g.out = l < L - 1 ? ws.h[l & 1] : (void*)ws.z;
      g.ldo = c->lda[l + 1];
      g.ostride = 0;
      g.bias = c->central + c->boff[l];
      g.bstride = 0;
      g.zero = c->zero;
      HIP_CHECK(c, timed(c, AGN_K_EVAL, [&] {
        return bf ? launch_gemm_bf16(1, 1, g, c->ls) : launch_gemm_f32(1, 1, g, c->ls);
      }));
    }
    int64_t blocks = 0;
    if (c->use_head) {  // fused output layer (float32, few classes)
      HeadArgs h{};
      h.h = L == 1 ? static_cast<const float*>(x) : static_cast<const float*>(ws.h[(L - 2) & 1]);
      h.ldh = L == 1 ? d0 : c->lda[L - 1];
      h.hstride = 0;
      h.gather = 0;
      h.w = c->central + c->woff[L - 1];
      h.b = c->central + c->boff[L - 1];
      h.ldw = c->ldw[L - 1];
      h.pstride = 0;
      h.y = d->y + r0;
      h.g = rows_as_stored;
      h.n = 1;
      h.m = rows;
      h.d = c->dims[L - 1];
      h.C = c->dims[L];
      h.row_loss = row_loss ? row_loss + r0 : nullptr;
      h.row_pred = row_pred ? row_pred + r0 : nullptr;
      h.part = ws.part;
      HIP_CHECK(c, timed(c, AGN_K_EVAL, [&] { return launch_head_eval(h, c->ls); }));
      blocks = head_eval_blocks(rows);
    } else {
      EvalArgs e{};
      e.z = ws.z;
      e.ldz = c->lda[L];
      e.y = d->y + r0;
      e.rows = rows;
      e.C = c->dims[L];
      e.row_loss = row_loss ? row_loss + r0 : nullptr;
      e.row_pred = row_pred ? row_pred + r0 : nullptr;
      e.part = ws.part;
      HIP_CHECK(c, launch_eval_rows(e, c->ls));
      blocks = eval_blocks(rows);
    }
    HIP_CHECK(c, launch_eval_reduce(ws.part, blocks, ws.acc, r0 == 0, c->ls));
  }
  return AGN_OK;
}

// Eq. 4 helpers: a curve is valid when it has >= 2 finite samples starting
// at time 0 with increasing times; its area over [0, tm] follows the
// straight lines between samples, the segment around tm cut on its line.
bool te_curve_ok(const double* t, const double* f, int64_t n) {
  if (!t || !f || n < 2 || t[0] != 0.0) return false;
  for (int64_t i = 0; i < n; ++i)
    if (!std::isfinite(t[i]) || !std::isfinite(f[i]) || (i > 0 && !(t[i] > t[i - 1]))) return false;
  return true;
}

// Copy an evaluation's totals to the host (when out is not NULL).
int eval_result(agn_ctx* c, const EvalSpace& ws, int64_t N, agn_eval_result* out) {
  if (!out) return AGN_OK;
  double acc[2] = {0.0, 0.0};
  HIP_CHECK(c, hipMemcpyAsync(acc, ws.acc, sizeof acc, hipMemcpyDeviceToHost, c->stream));
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  out->mean_loss = acc[0] / (double)N;
  out->correct = (int64_t)acc[1];
  out->accuracy = (double)out->correct / (double)N;
  return AGN_OK;
}

// agn_evaluate_noalloc evaluates at least this many rows per forward pass
constexpr int64_t NOALLOC_MIN_ROWS = 64;

double te_area(const double* t, const double* f, int64_t n, double tm) {
  double area = 0.0;
  for (int64_t i = 1; i < n && t[i - 1] < tm; ++i) {
    double t1 = t[i], f1 = f[i];
    if (t1 > tm) {
      f1 = f[i - 1] + (f[i] - f[i - 1]) * (tm - t[i - 1]) / (t[i] - t[i - 1]);
      t1 = tm;
    }
    area += 0.5 * (f[i - 1] + f1) * (t1 - t[i - 1]);
  }
  return area;
}

}  // namespace

extern "C" {

int agn_create(const agn_shapes* shapes, int32_t n, int32_t lambda, float eta, uint64_t seed,
               agn_ctx** out) {
  if (out) *out = nullptr;
  if (!out) return fail(nullptr, AGN_EINVAL, "out is NULL");
  if (!shapes) return fail(nullptr, AGN_EINVAL, "shapes is NULL");
  const int L = shapes->num_layers;
  if (L < 1 || L > AGN_MAX_LAYERS) return fail(nullptr, AGN_EINVAL, "num_layers must be in [1, 16]");
  if (!shapes->dims) return fail(nullptr, AGN_EINVAL, "dims is NULL");
  for (int l = 0; l <= L; ++l)
    if (shapes->dims[l] < 1 || shapes->dims[l] > (1 << 20))
      return fail(nullptr, AGN_EINVAL, "every width must be in [1, 2^20]");
  if (shapes->dims[L] < 2) return fail(nullptr, AGN_EINVAL, "need at least 2 classes");
  if (shapes->batch < 1 || shapes->batch > (1 << 20))
    return fail(nullptr, AGN_EINVAL, "batch must be in [1, 2^20]");
  if (shapes->dtype != AGN_FP32 && shapes->dtype != AGN_BF16)
    return fail(nullptr, AGN_EINVAL, "dtype must be AGN_FP32 or AGN_BF16");
  if (n < 1 || n > AGN_MAX_WORKERS) return fail(nullptr, AGN_EINVAL, "n must be in [1, 256]");
  if (lambda < 1) return fail(nullptr, AGN_EINVAL, "lambda must be >= 1");
  if (!std::isfinite(eta)) return fail(nullptr, AGN_EINVAL, "eta must be finite");

  agn_ctx* c = new (std::nothrow) agn_ctx();
  if (!c) return fail(nullptr, AGN_ENOMEM, "host allocation failed");
  c->L = L;
  c->m = shapes->batch;
  c->dtype = shapes->dtype;
  c->n = n;
  c->lam = lambda;
  c->eta = eta;
  c->pulled_version.assign(n, 0);
  c->last_staleness.assign(n, 0);
  for (int l = 0; l <= L; ++l) c->dims[l] = shapes->dims[l];

  // parameter layout: W_l rows padded to 8 elements, tensors 64-element aligned
  int64_t off = 0, P = 0;
  c->pack.ntensors = 2 * L;
  for (int l = 0; l < L; ++l) {
    const int64_t din = c->dims[l], dout = c->dims[l + 1];
    c->ldw[l] = round_up(din, 8);
    c->woff[l] = off;
    c->pack.t[2 * l] = TensorDesc{P, off, c->ldw[l], (int32_t)dout, (int32_t)din};
    off = round_up(off + dout * c->ldw[l], 64);
    P += din * dout;
    c->boff[l] = off;
    c->pack.t[2 * l + 1] = TensorDesc{P, off, dout, 1, (int32_t)dout};
    off = round_up(off + dout, 64);
    P += dout;
  }
  c->P = P;
  c->P_pad = off;
  c->pack.P = P;
  for (int l = 0; l <= L; ++l) c->lda[l] = round_up(c->dims[l], 8);

  auto bail = [&](int code, const std::string& msg) {
    free_all(c);
    delete c;
    return fail(nullptr, code, msg);
  };
  if (hipGetDevice(&c->device) != hipSuccess) return bail(AGN_EHIP, "no HIP device");
  {
    const hipError_t e = scratch_address(c->device, &c->scratch);
    if (e != hipSuccess)
      return bail(AGN_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
  }
  c->use_head = c->dtype == AGN_FP32 && head_prepare(c->dims[L], c->dims[L - 1]);
  if (hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking) != hipSuccess)
    return bail(AGN_EHIP, "hipStreamCreate failed");

  const bool bf = c->dtype == AGN_BF16;
  const int64_t nps = (int64_t)n * c->P_pad;
  const size_t act = bf ? 2 : 4;
  bool ok = dalloc(c, &c->central, c->P_pad) == hipSuccess && dalloc(c, &c->snap, nps) == hipSuccess &&
            dalloc(c, &c->buf[0], nps) == hipSuccess && dalloc(c, &c->buf[1], nps) == hipSuccess &&
            dalloc(c, &c->Z, (int64_t)n * c->m * c->lda[L]) == hipSuccess &&
            dalloc(c, &c->loss, (int64_t)n * lambda * c->m) == hipSuccess &&
            dalloc(c, &c->order, n) == hipSuccess && dalloc(c, &c->round_dev, 1) == hipSuccess &&
            dalloc(c, &c->commit_scale, n) == hipSuccess &&
            dalloc(c, &c->zero, 1024) == hipSuccess && dalloc(c, &c->sink, 1024) == hipSuccess;
  if (ok && bf)
    ok = dalloc(c, &c->snap16, nps) == hipSuccess && dalloc(c, &c->buf16[0], nps) == hipSuccess &&
         dalloc(c, &c->buf16[1], nps) == hipSuccess;
  for (int l = 1; ok && l <= L; ++l) {
    char* p = nullptr;
    const int64_t bytes = (int64_t)n * c->m * c->lda[l] * act;
    if (l < L) ok = dalloc(c, &p, bytes) == hipSuccess, c->H[l] = p;
    if (ok) ok = dalloc(c, &p, bytes) == hipSuccess, c->dZ[l] = p;
  }
  if (!ok) return bail(AGN_ENOMEM, "device allocation failed");

  // zero everything (padding stays zero forever), then the initial parameters
  hipError_t e = hipSuccess;
  e = hipMemset(c->central, 0, c->P_pad * 4);
  if (e == hipSuccess) e = hipMemset(c->snap, 0, nps * 4);
  if (e == hipSuccess) e = hipMemset(c->buf[0], 0, nps * 4);
  if (e == hipSuccess) e = hipMemset(c->buf[1], 0, nps * 4);
  if (e == hipSuccess && bf) e = hipMemset(c->snap16, 0, nps * 2);
  if (e == hipSuccess && bf) e = hipMemset(c->buf16[0], 0, nps * 2);
  if (e == hipSuccess && bf) e = hipMemset(c->buf16[1], 0, nps * 2);
  if (e == hipSuccess) e = hipMemset(c->round_dev, 0, 8);
  if (e == hipSuccess) e = hipMemset(c->zero, 0, 1024 * sizeof(float));
  if (e == hipSuccess) e = hipMemset(c->loss, 0, (size_t)n * lambda * c->m * 4);
  // activations and gradients: their row padding stays zero (no kernel
  // writes it; the bf16 products read it as a zero K tail)
  for (int l = 1; e == hipSuccess && l <= L; ++l) {
    const size_t bytes = (size_t)n * c->m * c->lda[l] * act;
    if (l < L) e = hipMemset(c->H[l], 0, bytes);
    if (e == hipSuccess) e = hipMemset(c->dZ[l], 0, bytes);
  }
  if (e != hipSuccess) return bail(AGN_EHIP, std::string("hipMemset: ") + hipGetErrorString(e));

  std::vector<float> init(P);
  he_normal_init(c->dims, L, seed, init.data());
  float* tmp = nullptr;
  e = hipMalloc(&tmp, P * sizeof(float));
  if (e != hipSuccess) return bail(AGN_ENOMEM, "device allocation failed");
  e = hipMemcpy(tmp, init.data(), P * sizeof(float), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = launch_unpack(c->pack, tmp, c->central, nullptr, 1, 0, nullptr);
  if (e == hipSuccess) e = launch_unpack(c->pack, tmp, c->snap, c->snap16, n, c->P_pad, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  (void)hipFree(tmp);
  if (e != hipSuccess) return bail(AGN_EHIP, std::string("init: ") + hipGetErrorString(e));
  *out = c;
  return AGN_OK;
}

int agn_set_stream(agn_ctx* c, void* s) {
  if (int r = check_ctx(c)) return r;
  c->stream = reinterpret_cast<hipStream_t>(s);
  return AGN_OK;
}

int agn_set_normalization(agn_ctx* c, int32_t normalize) {
  if (int r = check_ctx(c)) return r;
  if (normalize != 0 && normalize != 1) return fail(c, AGN_EINVAL, "normalize must be 0 or 1");
  if (c->rounds != 0) return fail(c, AGN_ESTATE, "agn_set_normalization is allowed only before the first round");
  c->normalize = normalize;
  return AGN_OK;
}

int agn_set_staleness_scaling(agn_ctx* c, int32_t enable) {
  if (int r = check_ctx(c)) return r;
  if (enable != 0 && enable != 1) return fail(c, AGN_EINVAL, "enable must be 0 or 1");
  if (c->rounds != 0) return fail(c, AGN_ESTATE, "agn_set_staleness_scaling is allowed only before the first round");
  c->staleness_scaling = enable;
  drop_graph(c);
  return AGN_OK;
}

int agn_staleness(agn_ctx* c, int64_t* out) {
  if (int r = check_ctx(c)) return r;
  if (!out) return fail(c, AGN_EINVAL, "out is NULL");
  if (c->rounds == 0) return fail(c, AGN_ESTATE, "no round has run yet");
  for (int j = 0; j < c->n; ++j) out[j] = c->last_staleness[j];
  return AGN_OK;
}

int agn_set_optimizer(agn_ctx* c, int32_t optimizer, float beta1, float beta2, float eps) {
  if (int r = check_ctx(c)) return r;
  if (optimizer != AGN_OPT_SGD && optimizer != AGN_OPT_ADAM) return fail(c, AGN_EINVAL, "unknown optimizer");
  if (optimizer == AGN_OPT_ADAM) {
    if (!(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f))
      return fail(c, AGN_EINVAL, "Adam betas must lie in [0, 1)");
    if (!(eps > 0.f) || !std::isfinite(eps)) return fail(c, AGN_EINVAL, "Adam eps must be positive and finite");
  }
  if (c->rounds != 0) return fail(c, AGN_ESTATE, "agn_set_optimizer is allowed only before the first round");
  if (int r = set_device(c)) return r;
  if (optimizer == AGN_OPT_ADAM && !c->mom_m) {
    const int64_t cnt = (int64_t)c->n * c->P_pad;
    if (dalloc(c, &c->mom_m, cnt) != hipSuccess || dalloc(c, &c->mom_v, cnt) != hipSuccess)
      return fail(c, AGN_ENOMEM, "cannot allocate the Adam moment buffers");
  }
  if (optimizer == AGN_OPT_ADAM) {  // moments start at zero
    HIP_CHECK(c, hipMemsetAsync(c->mom_m, 0, (size_t)c->n * c->P_pad * sizeof(float), c->stream));
    HIP_CHECK(c, hipMemsetAsync(c->mom_v, 0, (size_t)c->n * c->P_pad * sizeof(float), c->stream));
    HIP_CHECK(c, hipStreamSynchronize(c->stream));
  }
  c->optimizer = optimizer;
  c->beta1 = beta1;
  c->beta2 = beta2;
  c->adam_eps = eps;
  drop_graph(c);
  return AGN_OK;
}

int agn_round(agn_ctx* c, const agn_data* d, const int32_t* order) {
  if (int r = check_ctx(c)) return r;
  if (!d || !d->x || !d->y) return fail(c, AGN_EINVAL, "data, data->x and data->y must be non-NULL");
  if (d->x_dtype != (c->dtype == AGN_BF16 ? 1 : 0))
    return fail(c, AGN_EINVAL, "x_dtype must be 1 for AGN_BF16 contexts and 0 otherwise");
  if (d->num_samples < c->n) return fail(c, AGN_EINVAL, "num_samples must be >= n");
  if (c->N_fixed >= 0 && d->num_samples != c->N_fixed)
    return fail(c, AGN_EINVAL, "num_samples changed between rounds");
  if (!order) return fail(c, AGN_EINVAL, "commit_order is NULL");
  {
    std::vector<char> seen(c->n, 0);
    for (int j = 0; j < c->n; ++j) {
      const int k = order[j];
      if (k < 0 || k >= c->n || seen[k]) return fail(c, AGN_EINVAL, "commit_order is not a permutation of 0..n-1");
      seen[k] = 1;
    }
  }
  if (int r = set_device(c)) return r;
  // staleness of each commit (commits applied since the worker's last pull;
  // it pulls right after its own commit) and, when enabled, its scale
  std::vector<int64_t> tau(c->n);
  std::vector<float> scale(c->n);
  for (int j = 0; j < c->n; ++j) {
    tau[j] = c->version + j - c->pulled_version[order[j]];
    scale[j] = (float)(1.0 / (double)(tau[j] + 1));
  }
  // the commit order of this round (read by the commit kernel)
  HIP_CHECK(c, launch_set_order(order, c->staleness_scaling ? scale.data() : nullptr, c->n, c->order,
                                c->commit_scale, c->stream));
  bool timing = false;
  for (int k = 0; k < AGN_K_EVAL; ++k) timing = timing || c->timing[k].enabled;
  if (timing) {  // eager launches, each timed class bracketed by events
    c->ls = c->stream;
    if (int r = enqueue_round(c, d)) return r;
  } else {       // replay the captured round
    if (!c->graph_exec || c->graph_x != d->x || c->graph_y != d->y || c->graph_n != d->num_samples) {
      drop_graph(c);
      c->ls = c->cap_stream;
      c->capturing = 1;
      hipError_t e = hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeRelaxed);
      int r = e == hipSuccess ? enqueue_round(c, d) : AGN_OK;
      hipGraph_t gr = nullptr;
      hipError_t e2 = hipStreamEndCapture(c->cap_stream, &gr);
      c->capturing = 0;
      if (r) {
        if (gr) (void)hipGraphDestroy(gr);
        return r;
      }
      HIP_CHECK(c, e);
      HIP_CHECK(c, e2);
      c->graph = gr;
      HIP_CHECK(c, hipGraphInstantiate(&c->graph_exec, c->graph, nullptr, nullptr, 0));
      c->graph_x = d->x;
      c->graph_y = d->y;
      c->graph_n = d->num_samples;
    }
    HIP_CHECK(c, hipGraphLaunch(c->graph_exec, c->stream));
  }
  c->N_fixed = d->num_samples;
  c->last_committer = order[c->n - 1];
  c->have_deltas = 1;
  ++c->rounds;
  for (int j = 0; j < c->n; ++j) c->pulled_version[order[j]] = c->version + j + 1;
  c->version += c->n;
  c->last_staleness = tau;
  return AGN_OK;
}

int agn_central(agn_ctx* c, float* out) {
  if (int r = check_ctx(c)) return r;
  if (!out) return fail(c, AGN_EINVAL, "out is NULL");
  if (int r = set_device(c)) return r;
  HIP_CHECK(c, launch_pack(c->pack, c->central, out, c->stream));
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  return AGN_OK;
}

int agn_loss(agn_ctx* c, float* out) {
  if (int r = check_ctx(c)) return r;
  if (!out) return fail(c, AGN_EINVAL, "out is NULL");
  if (c->rounds == 0) return fail(c, AGN_ESTATE, "no round has run yet");
  if (int r = set_device(c)) return r;
  HIP_CHECK(c, launch_loss_reduce(c->loss, c->n, (int64_t)c->lam * c->m, out, c->stream));
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  return AGN_OK;
}

int agn_evaluate(agn_ctx* c, const agn_data* d, float* row_loss, int32_t* row_pred,
                 agn_eval_result* out) {
  if (int r = check_ctx(c)) return r;
  if (!d || !d->x || !d->y) return fail(c, AGN_EINVAL, "data, data->x and data->y must be non-NULL");
  if (d->x_dtype != (c->dtype == AGN_BF16 ? 1 : 0))
    return fail(c, AGN_EINVAL, "x_dtype must be 1 for AGN_BF16 contexts and 0 otherwise");
  if (d->num_samples < 1) return fail(c, AGN_EINVAL, "num_samples must be >= 1");
  if (int r = set_device(c)) return r;
  if (int r = eval_alloc(c)) return r;
  c->ls = c->stream;
  const EvalSpace ws{{c->ev_h[0], c->ev_h[1]}, c->ev_z, c->ev_w16, c->ev_part, c->ev_acc, EVAL_CHUNK};
  if (c->dtype == AGN_BF16) HIP_CHECK(c, launch_copy_bf16(c->central, c->ev_w16, c->P_pad, c->ls));
  if (int r = enqueue_eval(c, d, row_loss, row_pred, ws)) return r;
  c->eval_N = d->num_samples;
  return eval_result(c, ws, d->num_samples, out);
}

int agn_evaluate_noalloc(agn_ctx* c, const agn_data* d, float* row_loss, int32_t* row_pred,
                         agn_eval_result* out) {
  if (int r = check_ctx(c)) return r;
  if (!d || !d->x || !d->y) return fail(c, AGN_EINVAL, "data, data->x and data->y must be non-NULL");
  if (d->x_dtype != (c->dtype == AGN_BF16 ? 1 : 0))
    return fail(c, AGN_EINVAL, "x_dtype must be 1 for AGN_BF16 contexts and 0 otherwise");
  if (d->num_samples < 1) return fail(c, AGN_EINVAL, "num_samples must be >= 1");
  // the most rows per forward pass (a multiple of 64, at most the
  // allocating path's 8192) whose buffers fit in the scratch array
  int64_t rows = EVAL_CHUNK;
  while (rows >= NOALLOC_MIN_ROWS && eval_space_bytes(c, rows, nullptr, nullptr) > (int64_t)AGN_NOALLOC_SCRATCH_BYTES)
    rows -= NOALLOC_MIN_ROWS;
  if (rows < NOALLOC_MIN_ROWS)
    return fail(c, AGN_EINVAL, "the evaluation buffers of 64 rows of this model exceed the " +
                                   std::to_string(AGN_NOALLOC_SCRATCH_BYTES) +
                                   "-byte scratch array of agn_evaluate_noalloc (use agn_evaluate)");
  if (int r = set_device(c)) return r;
  EvalSpace ws{};
  eval_space_bytes(c, rows, c->scratch, &ws);
  // bf16 operands of the central variable: the bf16 copy that the last
  // commit wrote for the last committer's pull (before the first round,
  // and after agn_set_central, every worker's copy is the central one)
  if (c->dtype == AGN_BF16) ws.w16 = c->snap16 + (int64_t)c->last_committer * c->P_pad;
  c->ls = c->stream;
  c->untimed = 1;
  const int r = enqueue_eval(c, d, row_loss, row_pred, ws);
  c->untimed = 0;
  if (r) return r;
  c->eval_N = d->num_samples;
  return eval_result(c, ws, d->num_samples, out);
}

int agn_temporal_efficiency(const double* t_a, const double* f_a, int64_t n_a, const double* t_b,
                            const double* f_b, int64_t n_b, double* out) {
  if (!out) return fail(nullptr, AGN_EINVAL, "out is NULL");
  if (!te_curve_ok(t_a, f_a, n_a) || !te_curve_ok(t_b, f_b, n_b))
    return fail(nullptr, AGN_EINVAL,
                "a curve needs >= 2 finite samples, times starting at 0 and increasing");
  const double tm = std::min(t_a[n_a - 1], t_b[n_b - 1]);
  const double den = te_area(t_b, f_b, n_b, tm);
  if (den == 0.0) return fail(nullptr, AGN_EINVAL, "the area under curve b is zero");
  *out = te_area(t_a, f_a, n_a, tm) / den;
  return AGN_OK;
}

int64_t agn_num_params(const agn_ctx* c) { return c ? c->P : -1; }

const char* agn_last_error(const agn_ctx* c) { return c ? c->err.c_str() : g_create_err.c_str(); }

void agn_destroy(agn_ctx* c) {
  if (!c) return;
  (void)hipSetDevice(c->device);
  (void)hipStreamSynchronize(c->stream);
  free_all(c);
  delete c;
}

// ---- checkpoint / resume ---------------------------------------------------

namespace {

constexpr char kStateMagic[8] = {'A', 'G', 'N', 'S', 'T', 'A', 'T', 'E'};
constexpr int32_t kStateVersion = 1;

struct StateHeader {
  char magic[8];
  int32_t version, L, m, n, lam, dtype, optimizer, normalize, staleness_scaling;
  int32_t dims[AGN_MAX_LAYERS + 1];
  float eta, beta1, beta2, adam_eps;
  int64_t P, rounds, commits, num_samples, last_committer;
};

StateHeader state_header(const agn_ctx* c) {
  StateHeader h;
  std::memset(&h, 0, sizeof(h));
  std::memcpy(h.magic, kStateMagic, sizeof(h.magic));
  h.version = kStateVersion;
  h.L = c->L;
  h.m = c->m;
  h.n = c->n;
  h.lam = c->lam;
  h.dtype = c->dtype;
  h.optimizer = c->optimizer;
  h.normalize = c->normalize;
  h.staleness_scaling = c->staleness_scaling;
  for (int l = 0; l <= c->L; ++l) h.dims[l] = c->dims[l];
  h.eta = c->eta;
  h.beta1 = c->optimizer == AGN_OPT_ADAM ? c->beta1 : 0.f;
  h.beta2 = c->optimizer == AGN_OPT_ADAM ? c->beta2 : 0.f;
  h.adam_eps = c->optimizer == AGN_OPT_ADAM ? c->adam_eps : 0.f;
  h.P = c->P;
  h.rounds = c->rounds;
  h.commits = c->version;
  h.num_samples = c->N_fixed;
  h.last_committer = c->last_committer;
  return h;
}

// float32 vectors of P parameters in the state: central, n pulled copies,
// and with Adam 2n moment vectors
int64_t state_vectors(const agn_ctx* c) { return 1 + (int64_t)c->n * (c->optimizer == AGN_OPT_ADAM ? 3 : 1); }
int64_t state_loss_floats(const agn_ctx* c) { return (int64_t)c->n * c->lam * c->m; }
int64_t state_size(const agn_ctx* c) {
  return (int64_t)sizeof(StateHeader) + 2 * (int64_t)c->n * (int64_t)sizeof(int64_t) +
         (state_loss_floats(c) + state_vectors(c) * c->P) * (int64_t)sizeof(float);
}

// device vector v of the state (padded layout, P_pad floats)
float* state_vector(agn_ctx* c, int64_t v) {
  if (v == 0) return c->central;
  --v;
  if (v < c->n) return c->snap + v * c->P_pad;
  v -= c->n;
  if (v < c->n) return c->mom_m + v * c->P_pad;
  return c->mom_v + (v - c->n) * c->P_pad;
}

// padded <-> packed on the host (the layout of agn_central)
void pack_host(const PackArgs& pa, const float* padded, float* packed) {
  for (int t = 0; t < pa.ntensors; ++t) {
    const TensorDesc& d = pa.t[t];
    for (int r = 0; r < d.rows; ++r)
      std::memcpy(packed + d.packed_off + (int64_t)r * d.cols, padded + d.padded_off + (int64_t)r * d.ld,
                  (size_t)d.cols * sizeof(float));
  }
}
void unpack_host(const PackArgs& pa, const float* packed, float* padded) {
  for (int t = 0; t < pa.ntensors; ++t) {
    const TensorDesc& d = pa.t[t];
    for (int r = 0; r < d.rows; ++r)
      std::memcpy(padded + d.padded_off + (int64_t)r * d.ld, packed + d.packed_off + (int64_t)r * d.cols,
                  (size_t)d.cols * sizeof(float));
  }
}

// the first field of h that differs from the configuration of c, or nullptr
const char* state_mismatch(const agn_ctx* c, const StateHeader& h) {
  const StateHeader o = state_header(c);
  if (std::memcmp(h.magic, kStateMagic, sizeof(h.magic)) != 0) return "magic (not an AGN state)";
  if (h.version != kStateVersion) return "format version";
  if (h.L != o.L) return "number of layers";
  for (int l = 0; l <= AGN_MAX_LAYERS; ++l)
    if (h.dims[l] != o.dims[l]) return "layer widths";
  if (h.m != o.m) return "mini-batch size m";
  if (h.n != o.n) return "number of workers n";
  if (h.lam != o.lam) return "lambda";
  if (h.dtype != o.dtype) return "dtype";
  if (h.optimizer != o.optimizer) return "local rule (select Adam with agn_set_optimizer before restoring an Adam state)";
  if (h.normalize != o.normalize) return "commit rule (agn_set_normalization)";
  if (h.staleness_scaling != o.staleness_scaling) return "staleness scaling (agn_set_staleness_scaling)";
  if (std::memcmp(&h.eta, &o.eta, sizeof(float)) != 0) return "eta";
  if (std::memcmp(&h.beta1, &o.beta1, 3 * sizeof(float)) != 0) return "Adam's beta1, beta2 or eps";
  if (h.P != o.P) return "number of parameters";
  return nullptr;
}

}  // namespace

int64_t agn_state_bytes(const agn_ctx* c) { return c ? state_size(c) : -1; }

int agn_get_state(agn_ctx* c, void* out, int64_t bytes) {
  if (int r = check_ctx(c)) return r;
  if (!out) return fail(c, AGN_EINVAL, "out is NULL");
  if (bytes != state_size(c))
    return fail(c, AGN_EINVAL, "the state needs exactly " + std::to_string(state_size(c)) + " bytes");
  if (int r = set_device(c)) return r;
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  char* p = static_cast<char*>(out);
  const StateHeader h = state_header(c);
  std::memcpy(p, &h, sizeof(h));
  p += sizeof(h);
  for (int k = 0; k < c->n; ++k) {
    const int64_t pv = c->pulled_version[k];
    std::memcpy(p + k * sizeof(int64_t), &pv, sizeof(pv));
    const int64_t st = k < (int)c->last_staleness.size() ? c->last_staleness[k] : 0;
    std::memcpy(p + (c->n + k) * sizeof(int64_t), &st, sizeof(st));
  }
  p += 2 * c->n * sizeof(int64_t);
  const int64_t nl = state_loss_floats(c);
  HIP_CHECK(c, hipMemcpyAsync(p, c->loss, nl * sizeof(float), hipMemcpyDeviceToHost, c->stream));
  p += nl * sizeof(float);
  std::vector<float> tmp((size_t)c->P_pad);
  for (int64_t v = 0; v < state_vectors(c); ++v) {
    HIP_CHECK(c, hipMemcpyAsync(tmp.data(), state_vector(c, v), c->P_pad * sizeof(float), hipMemcpyDeviceToHost,
                                c->stream));
    HIP_CHECK(c, hipStreamSynchronize(c->stream));
    pack_host(c->pack, tmp.data(), reinterpret_cast<float*>(p));
    p += c->P * sizeof(float);
  }
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  return AGN_OK;
}

int agn_set_state(agn_ctx* c, const void* in, int64_t bytes) {
  if (int r = check_ctx(c)) return r;
  if (!in) return fail(c, AGN_EINVAL, "in is NULL");
  if (bytes != state_size(c))
    return fail(c, AGN_EINVAL, "a state of this context has exactly " + std::to_string(state_size(c)) + " bytes");
  const char* p = static_cast<const char*>(in);
  StateHeader h;
  std::memcpy(&h, p, sizeof(h));
  if (const char* what = state_mismatch(c, h))
    return fail(c, AGN_EINVAL, std::string("the state was taken from another configuration: ") + what);
  // the counters must be consistent: rounds * n commits, pull counters in
  // [0, commits], a worker that committed last
  if (h.rounds < 0 || h.commits != h.rounds * h.n || h.last_committer < 0 || h.last_committer >= h.n ||
      (h.rounds > 0 && h.num_samples < h.n) || (h.rounds == 0 && h.num_samples != -1))
    return fail(c, AGN_EINVAL, "inconsistent round counters in the state");
  std::vector<int64_t> pv(c->n), st(c->n);
  std::memcpy(pv.data(), p + sizeof(h), c->n * sizeof(int64_t));
  std::memcpy(st.data(), p + sizeof(h) + c->n * sizeof(int64_t), c->n * sizeof(int64_t));
  for (int k = 0; k < c->n; ++k)
    if (pv[k] < 0 || pv[k] > h.commits) return fail(c, AGN_EINVAL, "inconsistent pull counters in the state");
  if (int r = set_device(c)) return r;
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  p += sizeof(h) + 2 * c->n * sizeof(int64_t);
  const int64_t nl = state_loss_floats(c);
  HIP_CHECK(c, hipMemcpyAsync(c->loss, p, nl * sizeof(float), hipMemcpyHostToDevice, c->stream));
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  p += nl * sizeof(float);
  std::vector<float> tmp((size_t)c->P_pad, 0.f);  // padding stays zero
  for (int64_t v = 0; v < state_vectors(c); ++v) {
    unpack_host(c->pack, reinterpret_cast<const float*>(p), tmp.data());
    HIP_CHECK(c, hipMemcpyAsync(state_vector(c, v), tmp.data(), c->P_pad * sizeof(float), hipMemcpyHostToDevice,
                                c->stream));
    HIP_CHECK(c, hipStreamSynchronize(c->stream));
    p += c->P * sizeof(float);
  }
  if (c->dtype == AGN_BF16)  // the bf16 copies of the pulls, as the commit writes them
    HIP_CHECK(c, launch_copy_bf16(c->snap, c->snap16, (int64_t)c->n * c->P_pad, c->stream));
  const int64_t rounds = h.rounds;
  HIP_CHECK(c, hipMemcpyAsync(c->round_dev, &rounds, sizeof(rounds), hipMemcpyHostToDevice, c->stream));
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  c->rounds = h.rounds;
  c->version = h.commits;
  c->N_fixed = h.num_samples;
  c->last_committer = (int)h.last_committer;
  c->pulled_version = pv;
  c->last_staleness = h.rounds > 0 ? st : std::vector<int64_t>();
  c->have_deltas = 0;
  return AGN_OK;
}

int agn_set_central(agn_ctx* c, const float* in) {
  if (int r = check_ctx(c)) return r;
  if (!in) return fail(c, AGN_EINVAL, "in is NULL");
  if (c->rounds != 0) return fail(c, AGN_ESTATE, "agn_set_central is allowed only before the first round");
  if (int r = set_device(c)) return r;
  HIP_CHECK(c, launch_unpack(c->pack, in, c->central, nullptr, 1, 0, c->stream));
  HIP_CHECK(c, launch_unpack(c->pack, in, c->snap, c->snap16, c->n, c->P_pad, c->stream));
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  return AGN_OK;
}

int agn_worker_params(agn_ctx* c, int32_t worker, float* out) {
  if (int r = check_ctx(c)) return r;
  if (!out) return fail(c, AGN_EINVAL, "out is NULL");
  if (worker < 0 || worker >= c->n) return fail(c, AGN_EINVAL, "worker out of range");
  if (int r = set_device(c)) return r;
  HIP_CHECK(c, launch_pack(c->pack, c->snap + (int64_t)worker * c->P_pad, out, c->stream));
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  return AGN_OK;
}

int agn_debug_delta(agn_ctx* c, int32_t worker, float* out) {
  if (int r = check_ctx(c)) return r;
  if (!out) return fail(c, AGN_EINVAL, "out is NULL");
  if (worker < 0 || worker >= c->n) return fail(c, AGN_EINVAL, "worker out of range");
  if (!c->have_deltas) return fail(c, AGN_ESTATE, "no round has run since the context was created or restored");
  if (int r = set_device(c)) return r;
  const float* delta = c->buf[(c->lam - 1) & 1] + (int64_t)worker * c->P_pad;
  HIP_CHECK(c, launch_pack(c->pack, delta, out, c->stream));
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  return AGN_OK;
}

int agn_debug_batch_indices(agn_ctx* c, int32_t worker, int64_t step_t, int64_t num_samples, int64_t* out) {
  if (int r = check_ctx(c)) return r;
  if (!out) return fail(c, AGN_EINVAL, "out is NULL");
  if (worker < 0 || worker >= c->n) return fail(c, AGN_EINVAL, "worker out of range");
  if (step_t < 0) return fail(c, AGN_EINVAL, "step_t must be >= 0");
  if (num_samples < c->n) return fail(c, AGN_EINVAL, "num_samples must be >= n");
  if (int r = set_device(c)) return r;
  HIP_CHECK(c, launch_batch_indices(worker, step_t, c->m, num_samples / c->n, out, c->stream));
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  return AGN_OK;
}

int agn_kernel_class_work(agn_ctx* c, int32_t cls, double* flops, double* bytes) {
  if (int r = check_ctx(c)) return r;
  if (cls < 0 || cls >= AGN_K_NUM) return fail(c, AGN_EINVAL, "kernel class out of range");
  if (!flops || !bytes) return fail(c, AGN_EINVAL, "null output pointer");
  const int L = c->L;
  const double rows = (double)c->n * c->lam * c->m;  // worker-samples per round
  auto mac = [&](int l) { return (double)c->dims[l] * c->dims[l + 1]; };
  const double C = c->dims[L];
  const double xb = c->dtype == AGN_BF16 ? 2.0 : 4.0;
  // updated parameters: read + write per local step (+ bf16 shadow write,
  // + Adam's two moment estimates read and written)
  const double upd = ((c->dtype == AGN_BF16 ? 10.0 : 8.0) + (c->optimizer == AGN_OPT_ADAM ? 16.0 : 0.0)) *
                     (double)c->n * c->lam;
  double f = 0.0, b = 0.0;
  switch (cls) {
    case AGN_K_FWD:
      for (int l = 0; l < (c->use_head ? L - 1 : L); ++l) f += 2.0 * mac(l) * rows;
      break;
    case AGN_K_OUTPUT:
      if (c->use_head) {
        f = 2.0 * mac(L - 1) * rows * (L >= 2 ? 2.0 : 1.0);
        b = rows * (4.0 * c->dims[L - 1] * (L >= 2 ? 2.0 : 1.0) + 4.0 * C + 8.0);
      } else {
        b = rows * (4.0 * C + xb * C + 4.0);
      }
      break;
    case AGN_K_OUTPUT_DW:
      if (c->use_head) {  // (steps that folded it into the first layer's launch count there)
        const double own = 1.0 - (double)c->head_dw_folded / c->lam;
        f = 2.0 * mac(L - 1) * rows * own;
        b = upd * (mac(L - 1) + C) * own;
      }
      break;
    case AGN_K_BWD:  // hidden layers not done in the output kernels
      for (int l = 1; l < (c->use_head ? L - 1 : L); ++l) {
        f += 4.0 * mac(l) * rows;
        b += upd * (mac(l) + c->dims[l + 1]);
        // bf16: the input gradient reads the weights' bf16 shadow, a stream of
        // its own (in float32 it shares the update's read of the weights)
        if (c->dtype == AGN_BF16) b += 2.0 * (double)c->n * c->lam * mac(l);
      }
      break;
    case AGN_K_DW_FIRST:
      if (!(c->use_head && L == 1)) {
        f = 2.0 * mac(0) * rows;
        b = upd * (mac(0) + c->dims[1]);
      }
      if (c->use_head && c->head_dw_folded) {  // steps where the output layer's update rides in this launch
        const double folded = (double)c->head_dw_folded / c->lam;
        f += 2.0 * mac(L - 1) * rows * folded;
        b += upd * (mac(L - 1) + C) * folded;
      }
      break;
    case AGN_K_COMMIT:
      // central + n deltas in, n pulls + central out (+ the bf16 copies of
      // the pulls, the operands of each worker's next round)
      b = (8.0 * (double)(c->n + 1) + (c->dtype == AGN_BF16 ? 2.0 * c->n : 0.0)) * c->P;
      break;
    case AGN_K_EVAL: {  // the last evaluation: inputs and weights read, logits written
      const double N = (double)c->eval_N;
      for (int l = 0; l < L; ++l) f += 2.0 * mac(l) * N;
      b = c->eval_N > 0 ? N * (xb * c->dims[0] + 4.0 * C) + xb * (double)c->P : 0.0;
      break;
    }
  }
  *flops = f;
  *bytes = b;
  return AGN_OK;
}

int agn_set_kernel_timing(agn_ctx* c, int32_t cls, int32_t enable) {
  if (int r = check_ctx(c)) return r;
  if (cls < 0 || cls >= AGN_K_NUM) return fail(c, AGN_EINVAL, "kernel class out of range");
  c->timing[cls].enabled = enable != 0;
  c->timing[cls].used = 0;
  c->timing[cls].dropped = 0;
  return AGN_OK;
}

int agn_kernel_timing(agn_ctx* c, int32_t cls, double* total_ms, int64_t* launches) {
  if (int r = check_ctx(c)) return r;
  if (cls < 0 || cls >= AGN_K_NUM) return fail(c, AGN_EINVAL, "kernel class out of range");
  if (!total_ms || !launches) return fail(c, AGN_EINVAL, "null output pointer");
  if (int r = set_device(c)) return r;
  HIP_CHECK(c, hipStreamSynchronize(c->stream));
  const TimingSlot& t = c->timing[cls];
  double tot = 0.0;
  for (size_t i = 0; i < t.used; ++i) {
    float ms = 0.f;
    HIP_CHECK(c, hipEventElapsedTime(&ms, t.ev[2 * i], t.ev[2 * i + 1]));
    tot += ms;
  }
  *total_ms = tot;
  *launches = (int64_t)t.used;
  return AGN_OK;
}

}  // extern "C"
