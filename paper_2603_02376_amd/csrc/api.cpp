// C ABI of the MoE-layer library: argument validation, workspace layout and
// the orchestration of the kernels (route, dispatch, expert FFN, shared
// expert, combine). Every step of the layer runs in the library's own HIP
// kernels; this file only checks arguments and enqueues launches.
#include "moe.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <map>
#include <mutex>
#include <string>

#include "moe_internal.h"

namespace {

thread_local std::string g_last_error;

int fail(int status, const std::string& msg) {
  g_last_error = msg;
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(MOE_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Every launch helper reports hipGetLastError() after its launch. An error
// left pending by earlier, unrelated work on this thread would otherwise be
// reported as this call's failure, so each entry point clears it once its
// arguments are validated, right before its first HIP call.
void clear_pending_error() { (void)hipGetLastError(); }

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

size_t esize(const moe_config_t& c) { return c.dtype == MOE_BF16 ? 2 : 4; }

// Row tile of the router GEMM: 64 rows from 2048 tokens up (half the
// re-reads of the router weights of 32-row tiles, and one round of
// workgroups), 32 below.
constexpr int kGateM64Tokens = 2048;
bool gate_m64(int32_t T) { return T >= kGateM64Tokens; }

// K-split of the router GEMM (bf16 only): enough row tiles x splits to
// occupy ~256 workgroups with 64-row tiles (~512 with 32-row tiles), at
// least 4 k-steps of 64 per split. A function of (T, d) only, so the
// workspace size does not depend on the device.
int gate_splits(const moe_config_t& c, int32_t T) {
  if (c.dtype != MOE_BF16 || T <= 0) return 1;
  const bool m64 = gate_m64(T);
  const int mtiles = m64 ? (T + 63) / 64 : (T + 31) / 32;
  const int target = m64 ? 256 : 512;
  const int nkt = c.d / 64;
  int s = std::max(1, std::min(nkt / 4, (target + mtiles - 1) / mtiles));
  const int q = (nkt + s - 1) / s;
  return (nkt + q - 1) / q;  // no empty split
}

// Tile-queue heads of the weight-streaming GEMMs (8 per GEMM) and the
// per-group counters of the one-launch FFN, all zeroed before use: the
// routed FFN's GEMM1 and GEMM2 heads [0, 16) and counters [16, kRoutedInts),
// then the heads of the shared expert's own FFN from kSharedQueue (that FFN
// may run on another stream at the same time, so it has its own).
constexpr int kRoutedInts = 16 + moe::kFfnDepsInts;
constexpr int kSharedQueue = 288;
constexpr int kQueueInts = kSharedQueue + 16;
static_assert(kRoutedInts <= kSharedQueue, "queue regions overlap");

// Byte offsets of every scratch region inside the caller's workspace.
struct Layout {
  size_t gate_partials, logits, topk_idx, topk_w, masks, bases, counts, offsets, sorted_token, sorted_assign,
      inv_perm, h, y_perm, shared_h, shared_out, queues, qcodes, qscales, dense_part, dense_part_bytes, total;
};

Layout make_layout(const moe_config_t& c, int32_t T) {
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  const size_t t = (size_t)T, tk = (size_t)T * c.k, es = esize(c);
  const size_t nch = (t + moe::kDispatchChunk - 1) / moe::kDispatchChunk;
  const int gs = gate_splits(c, T);
  L.gate_partials = take(gs > 1 ? (size_t)gs * t * c.E * 4 : 0);
  L.logits = take(t * c.E * 4);
  L.topk_idx = take(tk * 4);
  L.topk_w = take(tk * 4);
  L.masks = take(nch * c.E * 8);
  L.bases = take(nch * c.E * 4);
  L.counts = take((size_t)c.E * 4);
  L.offsets = take((size_t)(c.E + 1) * 4);
  L.sorted_token = take(tk * 4);
  L.sorted_assign = take(tk * 4);
  L.inv_perm = take(tk * 4);
  L.h = take(tk * c.I * es);
  L.y_perm = take(tk * c.d * es);
  L.shared_h = take(c.n_shared ? t * c.I_shared * es : 0);
  L.shared_out = take(c.n_shared ? t * c.d * es : 0);
  L.queues = take(kQueueInts * 4);
  const bool q8 = c.token_quant != MOE_QUANT_NONE;
  L.qcodes = take(q8 ? t * c.d : 0);  // moe_layer's quantized tokens
  L.qscales = take(q8 ? t * 4 : 0);
  L.dense_part_bytes = c.weight_layout == MOE_LAYOUT_PACKED ? moe::dense_part_bytes((int64_t)tk, c.E, c.d, c.I) : 0;
  L.dense_part = take(L.dense_part_bytes);
  L.total = off;
  return L;
}

int validate(const moe_config_t* c, int32_t T) {
  if (!c) return fail(MOE_ERR_INVALID_ARG, "config is NULL");
  if (T < 0) return fail(MOE_ERR_INVALID_ARG, "T < 0");
  if (c->d <= 0 || c->E <= 0 || c->k <= 0 || c->I <= 0)
    return fail(MOE_ERR_INVALID_ARG, "d, E, k and I must be positive");
  if (c->k > c->E) return fail(MOE_ERR_INVALID_ARG, "k > E");
  if (c->n_groups < 1 || c->E % c->n_groups != 0)
    return fail(MOE_ERR_INVALID_ARG, "E must be a positive multiple of n_groups");
  if (c->topk_groups < 1 || c->topk_groups > c->n_groups)
    return fail(MOE_ERR_INVALID_ARG, "need 1 <= topk_groups <= n_groups");
  if (c->n_groups > 1 && (int64_t)c->k > (int64_t)c->topk_groups * (c->E / c->n_groups))
    return fail(MOE_ERR_INVALID_ARG, "k exceeds the experts left by the group limit");
  if (c->score != MOE_SCORE_SOFTMAX && c->score != MOE_SCORE_SIGMOID)
    return fail(MOE_ERR_INVALID_ARG, "unknown score function");
  if (c->n_shared < 0) return fail(MOE_ERR_INVALID_ARG, "n_shared < 0");
  if (c->n_shared > 0 && c->I_shared <= 0) return fail(MOE_ERR_INVALID_ARG, "I_shared must be positive");
  if (!std::isfinite(c->route_scale)) return fail(MOE_ERR_INVALID_ARG, "route_scale is not finite");
  if (c->dtype != MOE_F32 && c->dtype != MOE_BF16) return fail(MOE_ERR_UNSUPPORTED, "unknown dtype");
  if (c->E > 256) return fail(MOE_ERR_UNSUPPORTED, "E > 256");
  if (c->k > 16) return fail(MOE_ERR_UNSUPPORTED, "k > 16");
  if (c->n_groups > 64) return fail(MOE_ERR_UNSUPPORTED, "n_groups > 64");
  if (c->n_shared > 1) return fail(MOE_ERR_UNSUPPORTED, "n_shared > 1");
  if (c->d % 64 != 0 || c->I % 64 != 0 || (c->n_shared && c->I_shared % 64 != 0))
    return fail(MOE_ERR_UNSUPPORTED, "d, I and I_shared must be multiples of 64");
  if ((int64_t)T * c->k >= (int64_t)1 << 31) return fail(MOE_ERR_UNSUPPORTED, "T*k >= 2^31");
  if (c->weight_layout != MOE_LAYOUT_ROWMAJOR && c->weight_layout != MOE_LAYOUT_PACKED)
    return fail(MOE_ERR_INVALID_ARG, "unknown weight layout");
  if (c->token_quant != MOE_QUANT_NONE && c->token_quant != MOE_QUANT_INT8 && c->token_quant != MOE_QUANT_FP8)
    return fail(MOE_ERR_INVALID_ARG, "unknown token quantization");
  if (c->token_quant != MOE_QUANT_NONE && (c->dtype != MOE_BF16 || c->weight_layout != MOE_LAYOUT_PACKED))
    return fail(MOE_ERR_UNSUPPORTED, "quantized tokens need bf16 and packed weights");
  if (c->weight_layout == MOE_LAYOUT_PACKED &&
      (c->dtype != MOE_BF16 || c->I % 128 != 0 || c->d % 256 != 0 || (c->n_shared && c->I_shared % 128 != 0)))
    return fail(MOE_ERR_UNSUPPORTED, "packed weights need bf16, I and I_shared % 128 == 0 and d % 256 == 0");
  // The weight-streaming GEMMs address their row operand (x, then the
  // intermediate h) with 32-bit byte offsets.
  if (c->weight_layout == MOE_LAYOUT_PACKED &&
      ((int64_t)T * c->d * 2 > (int64_t)UINT32_MAX || (int64_t)T * c->k * c->I * 2 > (int64_t)UINT32_MAX ||
       (int64_t)T * c->n_shared * c->I_shared * 2 > (int64_t)UINT32_MAX))
    return fail(MOE_ERR_UNSUPPORTED, "packed weights need T*d and T*k*I below 2^31 elements");
  return MOE_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int need(const void* p, const char* name) {
  if (!p) return fail(MOE_ERR_INVALID_ARG, std::string(name) + " is NULL");
  if (!aligned16(p)) return fail(MOE_ERR_INVALID_ARG, std::string(name) + " is not 16-byte aligned");
  return MOE_OK;
}

// int32 index arrays of the expert-parallel calls: non-null and 4-byte
// aligned (they may start inside another array, e.g. offsets + 1).
int need_i32(const void* p, const char* name) {
  if (!p) return fail(MOE_ERR_INVALID_ARG, std::string(name) + " is NULL");
  if (reinterpret_cast<uintptr_t>(p) & 3u) return fail(MOE_ERR_INVALID_ARG, std::string(name) + " is not 4-byte aligned");
  return MOE_OK;
}

#define MOE_CHECK(expr)            \
  do {                             \
    const int _s = (expr);         \
    if (_s != MOE_OK) return _s;   \
  } while (0)

int check_ws(const moe_config_t* c, int32_t T, void* ws, size_t ws_bytes) {
  if (!ws) return fail(MOE_ERR_INVALID_ARG, "ws is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign) return fail(MOE_ERR_INVALID_ARG, "ws is not 256-byte aligned");
  const size_t want = make_layout(*c, T).total;
  if (ws_bytes < want)
    return fail(MOE_ERR_WORKSPACE, "workspace too small: need " + std::to_string(want) + " bytes, got " +
                                       std::to_string(ws_bytes));
  return MOE_OK;
}

// ---- internal launch helpers (arguments already validated) -----------------

hipError_t run_gemm(const moe_config_t& c, const moe::GemmProblem& p, int epi, bool out_f32, hipStream_t s) {
  if (c.dtype == MOE_BF16) return moe::launch_gemm_bf16(p, epi, out_f32, s);
  return moe::launch_gemm_f32(p, epi, s);
}

// Router GEMM then routing. With a K split the GEMM writes fp32 partial
// logits to `partials` and the route kernel sums them (in a fixed order) into
// `logits`; without one the GEMM writes `logits` directly. x == nullptr: the
// logits are an input.
hipError_t run_gate_route(const moe_config_t& c, int32_t T, const void* x, const void* w_router,
                          const float* bias, float* logits, float* partials, int32_t* idx, float* w,
                          hipStream_t s) {
  const int splits = x ? gate_splits(c, T) : 1;
  if (x) {
    moe::GemmProblem g{};
    g.A = x;
    g.a_rows = T;
    g.groups = 1;
    g.M = T;
    g.B0 = w_router;
    g.N = c.E;
    g.K = c.d;
    g.C = splits > 1 ? partials : logits;
    g.ldc = c.E;
    g.ksplit = splits;
    g.c_split_stride = (int64_t)T * c.E;
    g.tile = gate_m64(T) ? moe::GEMM_TILE_M64 : moe::GEMM_TILE_SKINNY;
    const hipError_t e = run_gemm(c, g, moe::EPI_STORE, true, s);
    if (e != hipSuccess) return e;
  }
  moe::RouteParams r{};
  r.logits_in = splits > 1 ? partials : logits;
  r.nsplit = splits;
  r.split_stride = (int64_t)T * c.E;
  r.logits_out = splits > 1 ? logits : nullptr;
  r.bias = (c.score == MOE_SCORE_SIGMOID) ? bias : nullptr;
  r.T = T;
  r.E = c.E;
  r.k = c.k;
  r.n_groups = c.n_groups;
  r.topk_groups = c.topk_groups;
  r.score = c.score;
  r.renorm = c.renorm;
  r.scale = c.route_scale;
  r.topk_idx = idx;
  r.topk_w = w;
  return moe::launch_route(r, s);
}

hipError_t run_dispatch(const moe_config_t& c, int32_t T, const int32_t* idx, char* ws, const Layout& L,
                        int32_t* counts, int32_t* offsets, int32_t* st, int32_t* sa, int32_t* inv, hipStream_t s,
                        int32_t* zero = nullptr, int32_t n_zero = 0) {
  moe::DispatchParams d{};
  d.topk_idx = idx;
  d.T = T;
  d.E = c.E;
  d.k = c.k;
  d.masks = reinterpret_cast<uint64_t*>(ws + L.masks);
  d.bases = reinterpret_cast<int32_t*>(ws + L.bases);
  d.counts = counts;
  d.offsets = offsets;
  d.sorted_token = st;
  d.sorted_assign = sa;
  d.inv_perm = inv;
  d.zero = zero;
  d.n_zero = n_zero;
  return moe::launch_dispatch(d, s);
}

// The shared expert fused into the routed weight-streaming launches as one
// extra group: its packed weights, its intermediate and output buffers
// (w_gate_up == nullptr: its GEMM1 has run on its own and only GEMM2 takes
// it along).
struct FusedShared {
  const void* w_gate_up = nullptr;
  const void* w_down = nullptr;
  void* h = nullptr;
  void* out = nullptr;
};

// How run_ffn runs the two GEMMs.
struct FfnOptions {
  bool packed = false;                // weights from moe_pack_weights (wu unused): the packed-weight kernels
  const FusedShared* fused = nullptr;  // packed, same intermediate size: the shared expert over all a_rows
                                       // tokens rides along as an extra group
  // 16 tile-queue heads (GEMM1, GEMM2) for the packed path, then (with
  // one_launch) the one-launch FFN's counters; zeroed here unless
  // queues_zeroed (moe_layer zeroes them in its dispatch)
  int32_t* queues = nullptr;
  bool queues_zeroed = false;
  const float* x_scales = nullptr;  // x holds int8 codes of rows with these fp32 scales (packed only)
  bool x_fp8 = false;               // with x_scales: the codes are FP8 (E4M3)
  // packed only: group g owns rows [offsets[g], seg_end[g]); at most max_wg
  // workgroups per GEMM (0: one per compute unit)
  const int32_t* seg_end = nullptr;
  int32_t max_wg = 0;
  // the groups hold exactly `rows` rows between them (false for a range of
  // groups or row segments: the GEMMs then keep the weight-streaming kernel,
  // whose choice does not depend on the groups' sizes)
  bool rows_exact = true;
  // workspace in which the compute-bound GEMM2 may split the K range of
  // short remainder blocks (nullptr: never)
  void* dense_part = nullptr;
  size_t dense_part_bytes = 0;
  // both weight-streaming GEMMs as one launch when the problem allows it
  // (bf16 tokens over whole groups, every compute unit), so the end of GEMM1
  // overlaps the start of GEMM2
  bool one_launch = false;
};

// Dense or grouped SwiGLU FFN: h = silu(X Wgᵀ) * (X Wuᵀ) into `h`, then
// y = h Wdᵀ into `y`.
hipError_t run_ffn(const moe_config_t& c, int32_t a_rows, int32_t rows, int32_t groups, int32_t inter, const void* x,
                   const int32_t* gather, const int32_t* offsets, const void* wg, const void* wu, const void* wd,
                   void* h, void* y, hipStream_t s, const FfnOptions& o = {}) {
  const bool packed = o.packed;
  int32_t* const queues = o.queues;
  const int32_t* const seg_end = o.seg_end;
  const bool one_launch = o.one_launch && packed && queues && !o.x_scales && !seg_end && o.max_wg == 0;
  if (packed && queues && !o.queues_zeroed) {
    const hipError_t e = moe::launch_queue_reset(queues, one_launch ? kRoutedInts : 16, s);
    if (e != hipSuccess) return e;
  }
  moe::GemmProblem up{};
  up.A = x;
  up.a_rows = a_rows;
  up.gather = gather;
  up.offsets = offsets;
  up.groups = groups;
  up.M = rows;
  up.B0 = wg;
  up.B1 = wu;
  up.N = inter;
  up.K = c.d;
  up.C = h;
  up.ldc = inter;
  if (o.fused && o.fused->w_gate_up) {
    up.xA = x;
    up.xB = o.fused->w_gate_up;
    up.xC = o.fused->h;
    up.x_rows = a_rows;
  }
  up.tile_queue = queues;
  up.a_scale = o.x_scales;
  up.a_fp8 = o.x_fp8 ? 1 : 0;
  up.seg_end = seg_end;
  up.max_wg = o.max_wg;
  up.rows_exact = o.rows_exact && !seg_end ? 1 : 0;
  moe::GemmProblem down{};
  down.A = h;
  down.a_rows = rows;
  down.offsets = offsets;
  down.groups = groups;
  down.M = rows;
  down.B0 = wd;
  down.N = c.d;
  down.K = inter;
  down.C = y;
  down.ldc = c.d;
  if (o.fused) {
    down.xA = o.fused->h;
    down.xB = o.fused->w_down;
    down.xC = o.fused->out;
    down.x_rows = a_rows;
  }
  down.tile_queue = queues ? queues + 8 : nullptr;
  down.seg_end = seg_end;
  down.max_wg = o.max_wg;
  down.rows_exact = up.rows_exact;
  down.dense_part = o.dense_part;
  down.dense_part_bytes = (int64_t)o.dense_part_bytes;
  if (one_launch) {
    up.deps = down.deps = queues + 16;
    const hipError_t e = moe::launch_ffn_stream(up, down, s);
    if (e != hipErrorNotSupported) return e;  // otherwise nothing was launched
  }
  hipError_t e = packed ? moe::launch_gemm_stream(up, moe::EPI_SWIGLU, s) : run_gemm(c, up, moe::EPI_SWIGLU, false, s);
  if (e != hipSuccess) return e;
  return packed ? moe::launch_gemm_stream(down, moe::EPI_STORE, s) : run_gemm(c, down, moe::EPI_STORE, false, s);
}

hipError_t run_combine(const moe_config_t& c, int32_t T, const void* y, const int32_t* inv, const float* w,
                       const void* shared, void* out, hipStream_t s) {
  moe::CombineParams p{};
  p.y_perm = y;
  p.inv_perm = inv;
  p.topk_w = w;
  p.shared_out = shared;
  p.out = out;
  p.T = T;
  p.k = c.k;
  p.d = c.d;
  return moe::launch_combine(p, c.dtype == MOE_BF16, s);
}

// Two events per (thread, device) for the fork/join of moe_layer's streams,
// created on first use and destroyed when the thread ends.
struct StreamEvents {
  hipEvent_t fork = nullptr, join = nullptr;
  StreamEvents() = default;
  StreamEvents(const StreamEvents&) = delete;
  StreamEvents& operator=(const StreamEvents&) = delete;
  ~StreamEvents() {
    if (fork) (void)hipEventDestroy(fork);
    if (join) (void)hipEventDestroy(join);
  }
};

hipError_t layer_events(StreamEvents** out) {
  thread_local StreamEvents ev[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  StreamEvents& se = ev[dev];
  if (!se.join) {
    if (!se.fork && (e = hipEventCreateWithFlags(&se.fork, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&se.join, hipEventDisableTiming)) != hipSuccess) return e;
  }
  *out = &se;
  return hipSuccess;
}

// Events per (thread, device) of moe_ep_expert_ffn: the fork and one per
// transferred expert range.
constexpr int kEpMaxChunks = 16;
struct EpEvents {
  hipEvent_t fork = nullptr;
  hipEvent_t chunk[kEpMaxChunks] = {};
  EpEvents() = default;
  EpEvents(const EpEvents&) = delete;
  EpEvents& operator=(const EpEvents&) = delete;
  ~EpEvents() {
    for (hipEvent_t c : chunk)
      if (c) (void)hipEventDestroy(c);
    if (fork) (void)hipEventDestroy(fork);
  }
};

hipError_t ep_events(EpEvents** out) {
  thread_local EpEvents ev[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  EpEvents& se = ev[dev];
  if (!se.fork) {  // the fork last: set once every event exists
    for (int i = 0; i < kEpMaxChunks; ++i)
      if (!se.chunk[i] && (e = hipEventCreateWithFlags(&se.chunk[i], hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&se.fork, hipEventDisableTiming)) != hipSuccess) return e;
  }
  *out = &se;
  return hipSuccess;
}

// The receive buffer's checks shared by the expert-parallel entry points:
// a packed bf16 config, and n_rows rows whose workspace is that of
// ceil(n_rows / k) tokens.
int validate_ep(const moe_config_t* c, int32_t n_rows, int32_t* tokens_out) {
  if (!c) return fail(MOE_ERR_INVALID_ARG, "config is NULL");
  if (n_rows < 0) return fail(MOE_ERR_INVALID_ARG, "n_rows < 0");
  if (c->k <= 0) return fail(MOE_ERR_INVALID_ARG, "k must be positive");
  const int32_t T = (int32_t)(((int64_t)n_rows + c->k - 1) / c->k);
  MOE_CHECK(validate(c, T));
  if (c->weight_layout != MOE_LAYOUT_PACKED || c->token_quant != MOE_QUANT_NONE)
    return fail(MOE_ERR_UNSUPPORTED, "the expert-parallel calls need packed bf16 weights and unquantized tokens");
  if ((int64_t)n_rows * c->d * 2 > (int64_t)UINT32_MAX)
    return fail(MOE_ERR_UNSUPPORTED, "n_rows*d must be below 2^31 elements");
  *tokens_out = T;
  return MOE_OK;
}

// FFN of experts [e0, e1) over row segments of x (no gather).
hipError_t run_ffn_segments(const moe_config_t& c, int32_t n_rows, const void* x, const int32_t* seg_begin,
                            const int32_t* seg_end, int32_t e0, int32_t e1, const void* w_gate_up, const void* w_down,
                            void* y, int32_t max_wg, char* ws, const Layout& L, hipStream_t s) {
  if (e1 <= e0 || n_rows == 0) return hipSuccess;
  // packed bf16: an expert's gate+up block is 2*I*d elements, its down block d*I
  const char* wgu = static_cast<const char*>(w_gate_up) + (size_t)e0 * 2 * c.I * c.d * 2;
  const char* wd = static_cast<const char*>(w_down) + (size_t)e0 * c.d * c.I * 2;
  FfnOptions o;
  o.packed = true;
  o.queues = reinterpret_cast<int32_t*>(ws + L.queues);
  o.seg_end = seg_end ? seg_end + e0 : nullptr;
  o.max_wg = max_wg;
  o.rows_exact = false;
  return run_ffn(c, n_rows, n_rows, e1 - e0, c.I, x, nullptr, seg_begin + e0, wgu, nullptr, wd, ws + L.h, y, s, o);
}

hipError_t run_ep_copy(const moe_config_t& c, int32_t mode, int32_t n_rows, const void* src, int32_t src_tokens,
                       const int32_t* row_token, const int32_t* offsets, const int32_t* self_end, int32_t e0,
                       int32_t e1, void* recv, int32_t max_wg, hipStream_t s) {
  moe::EpCopyParams p{};
  p.src = src;
  p.src_rows = src_tokens;
  p.row_token = row_token;
  p.offsets = offsets;
  p.self_end = self_end;
  p.e0 = e0;
  p.e1 = e1;
  p.mode = mode;
  p.n_rows = n_rows;
  p.row_bytes = c.d * (int32_t)esize(c);
  p.dst = recv;
  return moe::launch_ep_copy(p, max_wg, s);
}

}  // namespace

namespace moe {

int device_cu_count() {
  static std::mutex mu;
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lock(mu);
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

hipError_t set_dynamic_lds(const void* kern, int bytes) {
  static std::mutex mu;
  static std::map<std::pair<const void*, int>, hipError_t> done;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  const auto key = std::make_pair(kern, dev);
  const auto it = done.find(key);
  if (it != done.end()) return it->second;
  e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  done.emplace(key, e);
  return e;
}

}  // namespace moe

extern "C" {

size_t moe_workspace_size(const moe_config_t* cfg, int32_t T) {
  const std::string saved = g_last_error;
  if (validate(cfg, T) != MOE_OK) return 0;
  g_last_error = saved;
  return make_layout(*cfg, T).total;
}

int moe_route(const moe_config_t* cfg, int32_t T, const void* x, const void* w_router, const float* bias,
              float* logits, int32_t* topk_idx, float* topk_w, void* ws, size_t ws_bytes, hipStream_t stream) {
  MOE_CHECK(validate(cfg, T));
  if (cfg->score == MOE_SCORE_SOFTMAX && bias) return fail(MOE_ERR_INVALID_ARG, "bias given for softmax routing");
  MOE_CHECK(need(logits, "logits"));
  MOE_CHECK(need(topk_idx, "topk_idx"));
  MOE_CHECK(need(topk_w, "topk_w"));
  if (x) {
    MOE_CHECK(need(x, "x"));
    MOE_CHECK(need(w_router, "w_router"));
    MOE_CHECK(check_ws(cfg, T, ws, ws_bytes));
  }
  if (T == 0) return MOE_OK;
  clear_pending_error();
  float* partials = x ? reinterpret_cast<float*>(static_cast<char*>(ws) + make_layout(*cfg, T).gate_partials) : nullptr;
  const hipError_t e = run_gate_route(*cfg, T, x, w_router, bias, logits, partials, topk_idx, topk_w, stream);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "route");
}

int moe_dispatch(const moe_config_t* cfg, int32_t T, const int32_t* topk_idx, int32_t* counts, int32_t* offsets,
                 int32_t* sorted_token, int32_t* sorted_assign, int32_t* inv_perm, void* ws, size_t ws_bytes,
                 hipStream_t stream) {
  MOE_CHECK(validate(cfg, T));
  MOE_CHECK(need(topk_idx, "topk_idx"));
  MOE_CHECK(need(counts, "counts"));
  MOE_CHECK(need(offsets, "offsets"));
  MOE_CHECK(need(sorted_token, "sorted_token"));
  MOE_CHECK(need(inv_perm, "inv_perm"));
  if (sorted_assign && !aligned16(sorted_assign)) return fail(MOE_ERR_INVALID_ARG, "sorted_assign is not 16-byte aligned");
  MOE_CHECK(check_ws(cfg, T, ws, ws_bytes));
  if (T == 0) return MOE_OK;
  clear_pending_error();
  const Layout L = make_layout(*cfg, T);
  const hipError_t e = run_dispatch(*cfg, T, topk_idx, static_cast<char*>(ws), L, counts, offsets, sorted_token,
                                    sorted_assign, inv_perm, stream);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "dispatch");
}

int moe_dispatch_noalloc(const moe_config_t* cfg, int32_t T, const int32_t* topk_idx, int32_t* counts,
                         int32_t* offsets, int32_t* sorted_token, int32_t* sorted_assign, int32_t* inv_perm,
                         hipStream_t stream) {
  MOE_CHECK(validate(cfg, T));
  MOE_CHECK(need(topk_idx, "topk_idx"));
  MOE_CHECK(need(counts, "counts"));
  MOE_CHECK(need(offsets, "offsets"));
  MOE_CHECK(need(sorted_token, "sorted_token"));
  MOE_CHECK(need(inv_perm, "inv_perm"));
  if (sorted_assign && !aligned16(sorted_assign)) return fail(MOE_ERR_INVALID_ARG, "sorted_assign is not 16-byte aligned");
  const size_t items = (size_t)((T + moe::kDispatchChunk - 1) / moe::kDispatchChunk) * (size_t)cfg->E;
  if (items > moe::kDispatchNoAllocItems)
    return fail(MOE_ERR_UNSUPPORTED, "moe_dispatch_noalloc: ceil(T/64)*E = " + std::to_string(items) +
                                         " exceeds its scratch limit of " + std::to_string(moe::kDispatchNoAllocItems));
  if (T == 0) return MOE_OK;
  clear_pending_error();
  void* scr = nullptr;
  hipError_t e = moe::dispatch_noalloc_scratch(&scr);
  if (e != hipSuccess) return hip_fail(e, "dispatch scratch address");
  moe::DispatchParams d{};
  d.topk_idx = topk_idx;
  d.T = T;
  d.E = cfg->E;
  d.k = cfg->k;
  d.masks = static_cast<uint64_t*>(scr);
  d.bases = reinterpret_cast<int32_t*>(static_cast<char*>(scr) + moe::kDispatchNoAllocItems * 8);
  d.counts = counts;
  d.offsets = offsets;
  d.sorted_token = sorted_token;
  d.sorted_assign = sorted_assign;
  d.inv_perm = inv_perm;
  e = moe::launch_dispatch(d, stream);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "dispatch");
}

int moe_expert_ffn(const moe_config_t* cfg, int32_t T, const void* x, const int32_t* sorted_token,
                   const int32_t* offsets, const void* w_gate, const void* w_up, const void* w_down, void* y_perm,
                   void* ws, size_t ws_bytes, hipStream_t stream) {
  MOE_CHECK(validate(cfg, T));
  MOE_CHECK(need(x, "x"));
  MOE_CHECK(need(sorted_token, "sorted_token"));
  MOE_CHECK(need(offsets, "offsets"));
  const bool packed = cfg->weight_layout == MOE_LAYOUT_PACKED;
  MOE_CHECK(need(w_gate, "w_gate"));
  if (!packed) MOE_CHECK(need(w_up, "w_up"));
  MOE_CHECK(need(w_down, "w_down"));
  MOE_CHECK(need(y_perm, "y_perm"));
  MOE_CHECK(check_ws(cfg, T, ws, ws_bytes));
  if (T == 0) return MOE_OK;
  clear_pending_error();
  const Layout L = make_layout(*cfg, T);
  FfnOptions o;
  o.packed = packed;
  o.queues = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + L.queues);
  o.dense_part = static_cast<char*>(ws) + L.dense_part;
  o.dense_part_bytes = L.dense_part_bytes;
  o.one_launch = true;
  const hipError_t e = run_ffn(*cfg, T, T * cfg->k, cfg->E, cfg->I, x, sorted_token, offsets, w_gate, w_up, w_down,
                               static_cast<char*>(ws) + L.h, y_perm, stream, o);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "expert FFN");
}

int moe_quantize(const moe_config_t* cfg, int32_t T, const void* x, int8_t* codes, float* scales,
                 hipStream_t stream) {
  if (!cfg) return fail(MOE_ERR_INVALID_ARG, "config is NULL");
  if (cfg->token_quant != MOE_QUANT_NONE && cfg->token_quant != MOE_QUANT_INT8 && cfg->token_quant != MOE_QUANT_FP8)
    return fail(MOE_ERR_INVALID_ARG, "unknown token quantization");
  // the quantization needs only the token shape: the weight rules do not apply
  moe_config_t c = *cfg;
  c.token_quant = MOE_QUANT_NONE;
  c.weight_layout = MOE_LAYOUT_ROWMAJOR;
  MOE_CHECK(validate(&c, T));
  if (cfg->dtype != MOE_BF16) return fail(MOE_ERR_UNSUPPORTED, "moe_quantize needs bf16 tokens");
  MOE_CHECK(need(x, "x"));
  MOE_CHECK(need(codes, "codes"));
  MOE_CHECK(need(scales, "scales"));
  if (T == 0) return MOE_OK;
  clear_pending_error();
  const hipError_t e =
      moe::launch_quantize(x, codes, scales, T, cfg->d, cfg->token_quant == MOE_QUANT_FP8, stream);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "quantize");
}

int moe_expert_ffn_q8(const moe_config_t* cfg, int32_t T, const int8_t* codes, const float* scales,
                      const int32_t* sorted_token, const int32_t* offsets, const void* w_gate_up,
                      const void* w_down, void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream) {
  MOE_CHECK(validate(cfg, T));
  if (cfg->dtype != MOE_BF16 || cfg->weight_layout != MOE_LAYOUT_PACKED)
    return fail(MOE_ERR_UNSUPPORTED, "moe_expert_ffn_q8 needs bf16 and packed weights");
  MOE_CHECK(need(codes, "codes"));
  MOE_CHECK(need(scales, "scales"));
  MOE_CHECK(need(sorted_token, "sorted_token"));
  MOE_CHECK(need(offsets, "offsets"));
  MOE_CHECK(need(w_gate_up, "w_gate_up"));
  MOE_CHECK(need(w_down, "w_down"));
  MOE_CHECK(need(y_perm, "y_perm"));
  MOE_CHECK(check_ws(cfg, T, ws, ws_bytes));
  if (T == 0) return MOE_OK;
  clear_pending_error();
  const Layout L = make_layout(*cfg, T);
  FfnOptions o;
  o.packed = true;
  o.queues = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + L.queues);
  o.x_scales = scales;
  o.x_fp8 = cfg->token_quant == MOE_QUANT_FP8;
  const hipError_t e = run_ffn(*cfg, T, T * cfg->k, cfg->E, cfg->I, codes, sorted_token, offsets, w_gate_up, nullptr,
                               w_down, static_cast<char*>(ws) + L.h, y_perm, stream, o);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "expert FFN (quantized tokens)");
}

int moe_shared_ffn(const moe_config_t* cfg, int32_t T, const void* x, const void* ws_gate, const void* ws_up,
                   const void* ws_down, void* out, void* ws, size_t ws_bytes, hipStream_t stream) {
  MOE_CHECK(validate(cfg, T));
  if (cfg->n_shared != 1) return fail(MOE_ERR_INVALID_ARG, "config has no shared expert");
  const bool packed = cfg->weight_layout == MOE_LAYOUT_PACKED;
  MOE_CHECK(need(x, "x"));
  MOE_CHECK(need(ws_gate, "ws_gate"));
  if (!packed) MOE_CHECK(need(ws_up, "ws_up"));
  MOE_CHECK(need(ws_down, "ws_down"));
  MOE_CHECK(need(out, "out"));
  MOE_CHECK(check_ws(cfg, T, ws, ws_bytes));
  if (T == 0) return MOE_OK;
  clear_pending_error();
  const Layout L = make_layout(*cfg, T);
  FfnOptions o;
  o.packed = packed;
  o.queues = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + L.queues) + kSharedQueue;
  const hipError_t e = run_ffn(*cfg, T, T, 1, cfg->I_shared, x, nullptr, nullptr, ws_gate, ws_up, ws_down,
                               static_cast<char*>(ws) + L.shared_h, out, stream, o);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "shared FFN");
}

int moe_combine(const moe_config_t* cfg, int32_t T, const void* y_perm, const int32_t* inv_perm,
                const float* topk_w, const void* shared_out, void* out, hipStream_t stream) {
  MOE_CHECK(validate(cfg, T));
  MOE_CHECK(need(y_perm, "y_perm"));
  MOE_CHECK(need(inv_perm, "inv_perm"));
  MOE_CHECK(need(topk_w, "topk_w"));
  MOE_CHECK(need(out, "out"));
  if (shared_out && !aligned16(shared_out)) return fail(MOE_ERR_INVALID_ARG, "shared_out is not 16-byte aligned");
  if (T == 0) return MOE_OK;
  clear_pending_error();
  const hipError_t e = run_combine(*cfg, T, y_perm, inv_perm, topk_w, shared_out, out, stream);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "combine");
}

int moe_layer(const moe_config_t* cfg, int32_t T, const void* x, const void* w_router, const float* bias,
              const void* w_gate, const void* w_up, const void* w_down, const void* ws_gate, const void* ws_up,
              const void* ws_down, void* out, void* ws, size_t ws_bytes, hipStream_t s_main, hipStream_t s_aux,
              moe_layer_debug_t* dbg) {
  MOE_CHECK(validate(cfg, T));
  const moe_config_t& c = *cfg;
  if (c.score == MOE_SCORE_SOFTMAX && bias) return fail(MOE_ERR_INVALID_ARG, "bias given for softmax routing");
  const bool packed = c.weight_layout == MOE_LAYOUT_PACKED;
  MOE_CHECK(need(x, "x"));
  MOE_CHECK(need(w_router, "w_router"));
  MOE_CHECK(need(w_gate, "w_gate"));
  if (!packed) MOE_CHECK(need(w_up, "w_up"));
  MOE_CHECK(need(w_down, "w_down"));
  MOE_CHECK(need(out, "out"));
  if (c.n_shared) {
    MOE_CHECK(need(ws_gate, "ws_gate"));
    if (!packed) MOE_CHECK(need(ws_up, "ws_up"));
    MOE_CHECK(need(ws_down, "ws_down"));
  }
  MOE_CHECK(check_ws(cfg, T, ws, ws_bytes));
  moe_layer_debug_t none{};
  const moe_layer_debug_t& d = dbg ? *dbg : none;
  const void* dptrs[] = {d.logits, d.topk_idx, d.topk_w, d.counts, d.offsets, d.sorted_token,
                         d.sorted_assign, d.inv_perm, d.y_perm, d.shared_out};
  for (const void* p : dptrs)
    if (p && !aligned16(p)) return fail(MOE_ERR_INVALID_ARG, "debug buffer is not 16-byte aligned");
  if (d.shared_out && !c.n_shared) return fail(MOE_ERR_INVALID_ARG, "debug shared_out without a shared expert");
  if (T == 0) return MOE_OK;
  clear_pending_error();

  const Layout L = make_layout(c, T);
  char* w = static_cast<char*>(ws);
  float* logits = d.logits ? d.logits : reinterpret_cast<float*>(w + L.logits);
  int32_t* idx = d.topk_idx ? d.topk_idx : reinterpret_cast<int32_t*>(w + L.topk_idx);
  float* tw = d.topk_w ? d.topk_w : reinterpret_cast<float*>(w + L.topk_w);
  int32_t* counts = d.counts ? d.counts : reinterpret_cast<int32_t*>(w + L.counts);
  int32_t* offsets = d.offsets ? d.offsets : reinterpret_cast<int32_t*>(w + L.offsets);
  int32_t* st = d.sorted_token ? d.sorted_token : reinterpret_cast<int32_t*>(w + L.sorted_token);
  int32_t* inv = d.inv_perm ? d.inv_perm : reinterpret_cast<int32_t*>(w + L.inv_perm);
  void* y = d.y_perm ? d.y_perm : w + L.y_perm;
  void* shared = c.n_shared ? (d.shared_out ? d.shared_out : w + L.shared_out) : nullptr;
  int32_t* const queues = reinterpret_cast<int32_t*>(w + L.queues);  // routed FFN from 0, shared FFN from kSharedQueue

  hipError_t e;
  // Packed weights with equal intermediate sizes: the shared expert runs
  // inside the routed expert GEMMs as one more group, so its compute fills
  // the matrix cores of the memory-bound routed work. Otherwise it runs on
  // its own, on s_aux when given (overlapping gate, routing and dispatch).
  const bool q8 = c.token_quant != MOE_QUANT_NONE;  // int8 or FP8 codes
  const bool f8 = c.token_quant == MOE_QUANT_FP8;
  const bool fuse = packed && c.n_shared && c.I_shared == c.I && !q8;
  // With quantized tokens the shared expert's GEMM1 (bf16 input) runs on its
  // own before the routed GEMM1, and its GEMM2 rides along in the routed one.
  const bool fuse_down = packed && c.n_shared && c.I_shared == c.I && q8;
  const bool own = c.n_shared && !fuse && !fuse_down;  // the shared expert as a separate FFN
  const bool two = own && s_aux && s_aux != s_main;
  FfnOptions shared_opts;  // the shared expert as its own FFN
  shared_opts.packed = packed;
  shared_opts.queues = queues + kSharedQueue;
  StreamEvents* ev = nullptr;
  if (two) {
    // fork: the shared expert on s_aux may start once x is ready on s_main
    if ((e = layer_events(&ev)) != hipSuccess) return hip_fail(e, "event create");
    if ((e = hipEventRecord(ev->fork, s_main)) != hipSuccess) return hip_fail(e, "event record");
    if ((e = hipStreamWaitEvent(s_aux, ev->fork, 0)) != hipSuccess) return hip_fail(e, "stream wait");
    if ((e = run_ffn(c, T, T, 1, c.I_shared, x, nullptr, nullptr, ws_gate, ws_up, ws_down, w + L.shared_h, shared,
                     s_aux, shared_opts)) != hipSuccess)
      return hip_fail(e, "shared FFN");
    if ((e = hipEventRecord(ev->join, s_aux)) != hipSuccess) return hip_fail(e, "event record");
  }
  if ((e = run_gate_route(c, T, x, w_router, bias, logits, reinterpret_cast<float*>(w + L.gate_partials), idx, tw,
                          s_main)) != hipSuccess)
    return hip_fail(e, "route");
  // the dispatch also zeroes the routed FFN's tile-queue heads and counters
  // (packed weights; with quantized tokens also the shared GEMM1's heads)
  if ((e = run_dispatch(c, T, idx, w, L, counts, offsets, st, d.sorted_assign, inv, s_main, packed ? queues : nullptr,
                        packed ? (fuse_down ? kSharedQueue + 8 : kRoutedInts) : 0)) != hipSuccess)
    return hip_fail(e, "dispatch");
  int8_t* const qcodes = reinterpret_cast<int8_t*>(w + L.qcodes);
  float* const qscales = reinterpret_cast<float*>(w + L.qscales);
  if (q8 && (e = moe::launch_quantize(x, qcodes, qscales, T, c.d, f8, s_main)) != hipSuccess)
    return hip_fail(e, "quantize");
  FusedShared fs;
  if (fuse || fuse_down) {
    fs.w_gate_up = fuse ? ws_gate : nullptr;
    fs.w_down = ws_down;
    fs.h = w + L.shared_h;
    fs.out = shared;
  }
  if (fuse_down) {  // the shared expert's GEMM1 on its own (queue heads from kSharedQueue, zeroed by the dispatch)
    moe::GemmProblem g{};
    g.A = x;
    g.a_rows = T;
    g.groups = 1;
    g.M = T;
    g.B0 = ws_gate;
    g.N = c.I_shared;
    g.K = c.d;
    g.C = fs.h;
    g.ldc = c.I_shared;
    g.tile_queue = queues + kSharedQueue;
    if ((e = moe::launch_gemm_stream(g, moe::EPI_SWIGLU, s_main)) != hipSuccess) return hip_fail(e, "shared GEMM1");
  }
  FfnOptions routed;
  routed.packed = packed;
  routed.fused = (fuse || fuse_down) ? &fs : nullptr;
  routed.queues = queues;
  routed.queues_zeroed = true;  // by the dispatch
  routed.x_scales = q8 ? qscales : nullptr;
  routed.x_fp8 = f8;
  routed.dense_part = w + L.dense_part;
  routed.dense_part_bytes = L.dense_part_bytes;
  routed.one_launch = true;
  if ((e = run_ffn(c, T, T * c.k, c.E, c.I, q8 ? static_cast<const void*>(qcodes) : x, st, offsets, w_gate, w_up,
                   w_down, w + L.h, y, s_main, routed)) != hipSuccess)
    return hip_fail(e, "expert FFN");
  if (own) {
    if (two) {
      if ((e = hipStreamWaitEvent(s_main, ev->join, 0)) != hipSuccess) return hip_fail(e, "stream wait");
    } else if ((e = run_ffn(c, T, T, 1, c.I_shared, x, nullptr, nullptr, ws_gate, ws_up, ws_down, w + L.shared_h,
                            shared, s_main, shared_opts)) != hipSuccess) {
      return hip_fail(e, "shared FFN");
    }
  }
  if ((e = run_combine(c, T, y, inv, tw, shared, out, s_main)) != hipSuccess) return hip_fail(e, "combine");
  return MOE_OK;
}

int moe_ep_plan(const moe_config_t* cfg, int32_t e_first, const int32_t* self_offsets, const int32_t* self_sorted_token,
                int32_t self_assignments, const int32_t* peer_offsets, const int32_t* peer_sorted_token,
                int32_t peer_assignments, int32_t* row_token, int32_t capacity, int32_t* offsets, int32_t* self_end,
                hipStream_t stream) {
  if (!cfg) return fail(MOE_ERR_INVALID_ARG, "config is NULL");
  if (cfg->E <= 0 || cfg->E > 256) return fail(MOE_ERR_INVALID_ARG, "local experts must be in [1, 256]");
  if (e_first < 0) return fail(MOE_ERR_INVALID_ARG, "e_first < 0");
  if (self_assignments < 0 || peer_assignments < 0 || capacity < 0)
    return fail(MOE_ERR_INVALID_ARG, "negative size");
  MOE_CHECK(need_i32(self_offsets, "self_offsets"));
  MOE_CHECK(need_i32(peer_offsets, "peer_offsets"));
  if (self_assignments > 0) MOE_CHECK(need_i32(self_sorted_token, "self_sorted_token"));
  if (peer_assignments > 0) MOE_CHECK(need_i32(peer_sorted_token, "peer_sorted_token"));
  if (capacity > 0) MOE_CHECK(need_i32(row_token, "row_token"));
  MOE_CHECK(need_i32(offsets, "offsets"));
  MOE_CHECK(need_i32(self_end, "self_end"));
  moe::EpPlanParams p{};
  p.self_offsets = self_offsets;
  p.self_sorted = self_sorted_token;
  p.self_total = self_assignments;
  p.peer_offsets = peer_offsets;
  p.peer_sorted = peer_sorted_token;
  p.peer_total = peer_assignments;
  p.e_first = e_first;
  p.e_count = cfg->E;
  p.capacity = capacity;
  p.row_token = row_token;
  p.offsets = offsets;
  p.self_end = self_end;
  clear_pending_error();
  const hipError_t e = moe::launch_ep_plan(p, stream);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "receive plan");
}

int moe_ep_copy_rows(const moe_config_t* cfg, int32_t source, int32_t n_rows, const void* x_src, int32_t src_tokens,
                     const int32_t* row_token, const int32_t* offsets, const int32_t* self_end, int32_t e_begin,
                     int32_t e_end, void* recv, int32_t max_workgroups, hipStream_t stream) {
  int32_t T = 0;
  MOE_CHECK(validate_ep(cfg, n_rows, &T));
  if (source != MOE_EP_SELF && source != MOE_EP_REMOTE) return fail(MOE_ERR_INVALID_ARG, "unknown row source");
  if (e_begin < 0 || e_end > cfg->E || e_begin > e_end) return fail(MOE_ERR_INVALID_ARG, "bad expert range");
  MOE_CHECK(need_i32(row_token, "row_token"));
  MOE_CHECK(need_i32(offsets, "offsets"));
  MOE_CHECK(need_i32(self_end, "self_end"));
  MOE_CHECK(need(recv, "recv"));
  if (src_tokens < 0) return fail(MOE_ERR_INVALID_ARG, "src_tokens < 0");
  if (src_tokens > 0) MOE_CHECK(need(x_src, "x_src"));
  if (n_rows == 0 || e_begin == e_end || src_tokens == 0) return MOE_OK;
  clear_pending_error();
  const hipError_t e = run_ep_copy(*cfg, source, n_rows, x_src, src_tokens, row_token, offsets, self_end, e_begin,
                                   e_end, recv, max_workgroups, stream);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "row copy");
}

int moe_expert_ffn_segments(const moe_config_t* cfg, int32_t n_rows, const void* x, const int32_t* seg_begin,
                            const int32_t* seg_end, int32_t e_begin, int32_t e_end, const void* w_gate_up,
                            const void* w_down, void* y, int32_t max_workgroups, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
  int32_t T = 0;
  MOE_CHECK(validate_ep(cfg, n_rows, &T));
  if (e_begin < 0 || e_end > cfg->E || e_begin > e_end) return fail(MOE_ERR_INVALID_ARG, "bad expert range");
  MOE_CHECK(need(x, "x"));
  MOE_CHECK(need_i32(seg_begin, "seg_begin"));
  if (seg_end) MOE_CHECK(need_i32(seg_end, "seg_end"));
  MOE_CHECK(need(w_gate_up, "w_gate_up"));
  MOE_CHECK(need(w_down, "w_down"));
  MOE_CHECK(need(y, "y"));
  MOE_CHECK(check_ws(cfg, T, ws, ws_bytes));
  if (n_rows == 0 || e_begin == e_end) return MOE_OK;
  clear_pending_error();
  const hipError_t e = run_ffn_segments(*cfg, n_rows, x, seg_begin, seg_end, e_begin, e_end, w_gate_up, w_down, y,
                                        max_workgroups, static_cast<char*>(ws), make_layout(*cfg, T), stream);
  return e == hipSuccess ? MOE_OK : hip_fail(e, "expert FFN");
}

int moe_ep_expert_ffn(const moe_config_t* cfg, const moe_ep_options_t* opt, int32_t n_rows, const void* x_self,
                      int32_t self_tokens, const void* x_peer, int32_t peer_tokens, const int32_t* row_token,
                      const int32_t* offsets, const int32_t* self_end, const void* w_gate_up, const void* w_down,
                      void* recv, void* y, void* ws, size_t ws_bytes, hipStream_t s_compute, hipStream_t s_link) {
  int32_t T = 0;
  MOE_CHECK(validate_ep(cfg, n_rows, &T));
  if (!opt) return fail(MOE_ERR_INVALID_ARG, "options are NULL");
  const moe_ep_options_t o = *opt;
  if (o.schedule != MOE_EP_SEQUENTIAL && o.schedule != MOE_EP_SELF_REMOTE && o.schedule != MOE_EP_EXPERT_CHUNKS)
    return fail(MOE_ERR_INVALID_ARG, "unknown schedule");
  if (o.schedule == MOE_EP_EXPERT_CHUNKS && (o.chunks < 1 || o.chunks > kEpMaxChunks || o.chunks > cfg->E))
    return fail(MOE_ERR_INVALID_ARG, "chunks must be in [1, min(16, E)]");
  if (o.link_workgroups < 0 || o.gemm_workgroups < 0) return fail(MOE_ERR_INVALID_ARG, "negative workgroup cap");
  if (self_tokens < 0 || peer_tokens < 0) return fail(MOE_ERR_INVALID_ARG, "token counts < 0");
  if (self_tokens > 0) MOE_CHECK(need(x_self, "x_self"));
  if (peer_tokens > 0) MOE_CHECK(need(x_peer, "x_peer"));
  MOE_CHECK(need_i32(row_token, "row_token"));
  MOE_CHECK(need_i32(offsets, "offsets"));
  MOE_CHECK(need_i32(self_end, "self_end"));
  MOE_CHECK(need(w_gate_up, "w_gate_up"));
  MOE_CHECK(need(w_down, "w_down"));
  MOE_CHECK(need(recv, "recv"));
  MOE_CHECK(need(y, "y"));
  MOE_CHECK(check_ws(cfg, T, ws, ws_bytes));
  if (n_rows == 0) return MOE_OK;
  clear_pending_error();

  const moe_config_t& c = *cfg;
  const Layout L = make_layout(c, T);
  char* const w = static_cast<char*>(ws);
  const bool two = s_link && s_link != s_compute;
  hipStream_t const sl = two ? s_link : s_compute;
  EpEvents* ev = nullptr;
  hipError_t e;
  if ((e = ep_events(&ev)) != hipSuccess) return hip_fail(e, "event create");
  if (two) {  // the transfer may start once the caller's inputs are ready on s_compute
    if ((e = hipEventRecord(ev->fork, s_compute)) != hipSuccess) return hip_fail(e, "event record");
    if ((e = hipStreamWaitEvent(sl, ev->fork, 0)) != hipSuccess) return hip_fail(e, "stream wait");
  }
  auto copy = [&](int mode, int e0, int e1, int max_wg, hipStream_t s) {
    const void* src = mode == MOE_EP_SELF ? x_self : x_peer;
    const int32_t nsrc = mode == MOE_EP_SELF ? self_tokens : peer_tokens;
    if (nsrc == 0) return hipSuccess;
    return run_ep_copy(c, mode, n_rows, src, nsrc, row_token, offsets, self_end, e0, e1, recv, max_wg, s);
  };
  auto ffn = [&](const int32_t* b, const int32_t* en, int e0, int e1, int max_wg) {
    return run_ffn_segments(c, n_rows, recv, b, en, e0, e1, w_gate_up, w_down, y, max_wg, w, L, s_compute);
  };
  auto join = [&](hipEvent_t done) -> hipError_t {  // s_compute waits for the transfer up to here
    if (!two) return hipSuccess;
    hipError_t r = hipEventRecord(done, sl);
    return r != hipSuccess ? r : hipStreamWaitEvent(s_compute, done, 0);
  };
  const int E = c.E;
  switch (o.schedule) {
    case MOE_EP_SEQUENTIAL:
      // every row in, then one FFN over all of them
      if ((e = copy(MOE_EP_REMOTE, 0, E, o.link_workgroups, sl)) != hipSuccess) return hip_fail(e, "transfer");
      if ((e = copy(MOE_EP_SELF, 0, E, 0, s_compute)) != hipSuccess) return hip_fail(e, "self copy");
      if ((e = join(ev->chunk[0])) != hipSuccess) return hip_fail(e, "stream join");
      if ((e = ffn(offsets, nullptr, 0, E, 0)) != hipSuccess) return hip_fail(e, "expert FFN");
      break;
    case MOE_EP_SELF_REMOTE:
      // the self rows' FFN runs while the remote rows arrive; the remote
      // rows' FFN starts when all of them are in
      if ((e = copy(MOE_EP_REMOTE, 0, E, o.link_workgroups, sl)) != hipSuccess) return hip_fail(e, "transfer");
      if ((e = copy(MOE_EP_SELF, 0, E, 0, s_compute)) != hipSuccess) return hip_fail(e, "self copy");
      if ((e = ffn(offsets, self_end, 0, E, o.gemm_workgroups)) != hipSuccess) return hip_fail(e, "self FFN");
      if ((e = join(ev->chunk[0])) != hipSuccess) return hip_fail(e, "stream join");
      if ((e = ffn(self_end, offsets + 1, 0, E, 0)) != hipSuccess) return hip_fail(e, "remote FFN");
      break;
    default: {
      // the remote rows arrive by expert range; each range's FFN (its self
      // and remote rows in one pass over its weights) starts when its rows
      // are in
      const int C = o.chunks;
      if ((e = copy(MOE_EP_SELF, 0, E, 0, s_compute)) != hipSuccess) return hip_fail(e, "self copy");
      for (int i = 0; i < C; ++i) {
        const int e0 = (int)((int64_t)E * i / C), e1 = (int)((int64_t)E * (i + 1) / C);
        if ((e = copy(MOE_EP_REMOTE, e0, e1, o.link_workgroups, sl)) != hipSuccess) return hip_fail(e, "transfer");
        if ((e = join(ev->chunk[i])) != hipSuccess) return hip_fail(e, "stream join");
        if ((e = ffn(offsets, nullptr, e0, e1, i + 1 < C ? o.gemm_workgroups : 0)) != hipSuccess)
          return hip_fail(e, "expert FFN");
      }
    }
  }
  return MOE_OK;
}

int moe_pack_weights(const moe_config_t* cfg, const void* w_gate, const void* w_up, const void* w_down,
                     void* gate_up_packed, void* down_packed, hipStream_t stream) {
  if (!cfg) return fail(MOE_ERR_INVALID_ARG, "config is NULL");
  moe_config_t c = *cfg;
  c.weight_layout = MOE_LAYOUT_PACKED;
  MOE_CHECK(validate(&c, 0));
  if (gate_up_packed) {
    MOE_CHECK(need(w_gate, "w_gate"));
    MOE_CHECK(need(w_up, "w_up"));
    MOE_CHECK(need(gate_up_packed, "gate_up_packed"));
  }
  if (down_packed) {
    MOE_CHECK(need(w_down, "w_down"));
    MOE_CHECK(need(down_packed, "down_packed"));
  }
  if (!gate_up_packed && !down_packed) return MOE_OK;
  clear_pending_error();
  hipError_t e;
  if (gate_up_packed && (e = moe::launch_pack(w_gate, w_up, gate_up_packed, c.E, c.I, c.d, true, stream)) != hipSuccess)
    return hip_fail(e, "pack gate/up");
  if (down_packed && (e = moe::launch_pack(w_down, nullptr, down_packed, c.E, c.d, c.I, false, stream)) != hipSuccess)
    return hip_fail(e, "pack down");
  return MOE_OK;
}

const char* moe_status_string(int status) {
  switch (status) {
    case MOE_OK: return "ok";
    case MOE_ERR_INVALID_ARG: return "invalid argument";
    case MOE_ERR_UNSUPPORTED: return "unsupported configuration";
    case MOE_ERR_WORKSPACE: return "workspace too small";
    case MOE_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* moe_last_error(void) { return g_last_error.c_str(); }

const char* moe_version(void) { return "moe-mi355x 0.1.0 (gfx950)"; }

}  // extern "C"
