// C ABI entry points: argument validation, workspace carving and launch order of
// the region-sparse DiT step.  Nothing here allocates device memory.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "fd_common.h"

namespace {

thread_local char g_err[512] = "";

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

int score_rows_per_chunk(int C) {
  const int r = 2048 / C;
  return r < 1 ? 1 : r;
}

struct BlockWs {
  float* mod;
  uint16_t* a;
  uint16_t* q;
  uint16_t* o;
  uint16_t* g;
  float* partial;      // split-K partial tiles
  float* lse;          // [N][H] base-2 log-sum-exp of each active query's scaled scores
  size_t bytes;
};

BlockWs carve_block_ws(const fd_plan* p, const fd_dims* d, void* base) {
  const size_t n = static_cast<size_t>(p->n_tokens);
  size_t off = 0;
  BlockWs w;
  const uintptr_t b0 = reinterpret_cast<uintptr_t>(base);
  auto take = [&](size_t bytes) {
    const uintptr_t ptr = b0 + off;
    off += align_up(bytes);
    return reinterpret_cast<void*>(ptr);
  };
  w.mod = static_cast<float*>(take(static_cast<size_t>(p->n_requests) * 6 * d->D * sizeof(float)));
  w.a = static_cast<uint16_t*>(take(n * d->D * 2));
  w.q = static_cast<uint16_t*>(take(n * d->D * 2));
  w.o = static_cast<uint16_t*>(take(n * d->D * 2));
  w.g = static_cast<uint16_t*>(take(n * d->F * 2));
  const size_t gemm_part = fdh::gemm_scratch_bytes();
  const size_t attn_part = fdh::attn_scratch_bytes(d->dh);
  w.partial = static_cast<float*>(take(gemm_part > attn_part ? gemm_part : attn_part));
  w.lse = static_cast<float*>(take(n * d->H * sizeof(float)));
  w.bytes = off;
  return w;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

fd_status check_plan(const fd_plan* p) {
  if (!p) return fdh::set_error("plan is null"), FD_E_ARG;
  if (p->n_tokens < 1 || p->n_regions < 1 || p->n_requests < 1 || p->max_region_tokens < 1 ||
      p->max_request_tokens < 1)
    return fdh::set_error("plan sizes must be positive"), FD_E_ARG;
  if (!p->region_ptr || !p->region_tokens || !p->region_req || !p->token_region || !p->req_tok_off ||
      !p->req_reg_off)
    return fdh::set_error("plan has a null device array"), FD_E_ARG;
  return FD_OK;
}

fd_status check_dims(const fd_dims* d) {
  if (!d) return fdh::set_error("dims is null"), FD_E_ARG;
  if (d->C < 1 || d->D < 1 || d->H < 1 || d->dh < 1 || d->F < 1)
    return fdh::set_error("dims must be positive"), FD_E_ARG;
  if (d->D != d->H * d->dh) return fdh::set_error("D (%d) != H * dh (%d * %d)", d->D, d->H, d->dh), FD_E_SHAPE;
  if (d->dh != 16 && d->dh != 64 && d->dh != 128)
    return fdh::set_error("head dim %d not in {16, 64, 128}", d->dh), FD_E_UNSUPPORTED;
  if (d->D % 64 || d->F % 64) return fdh::set_error("D and F must be multiples of 64"), FD_E_UNSUPPORTED;
  if (d->D > 12288) return fdh::set_error("D > 12288 unsupported"), FD_E_UNSUPPORTED;
  if (d->C % 16 || d->C > 256) return fdh::set_error("C must be a multiple of 16, <= 256"), FD_E_UNSUPPORTED;
  return FD_OK;
}

fd_status check_C(int C) {
  if (C < 16 || C % 16 || C > 256) return fdh::set_error("C must be a multiple of 16 in [16, 256]"), FD_E_UNSUPPORTED;
  return FD_OK;
}

#define FD_REQUIRE(cond, ...)                  \
  do {                                         \
    if (!(cond)) {                             \
      fdh::set_error(__VA_ARGS__);             \
      return FD_E_ARG;                         \
    }                                          \
  } while (0)

#define FD_TRY(expr)                  \
  do {                                \
    fd_status st_ = (expr);           \
    if (st_ != FD_OK) return st_;     \
  } while (0)

#define FD_LAUNCH(kernel_id, stream, call)               \
  do {                                                   \
    fdh::timer_begin(kernel_id, stream);                 \
    hipError_t e_ = (call);                              \
    fdh::timer_end(kernel_id, stream);                   \
    if (e_ != hipSuccess) return fdh::hip_fail(e_, #call); \
  } while (0)

// ---------------------------------------------------------------- kernel timer
struct Timer {
  std::mutex mu;
  int kernel = 0;
  int capacity = 0;
  int count = 0;
  std::vector<hipEvent_t> ev;
} g_timer;

}  // namespace

namespace fdh {

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

fd_status hip_fail(hipError_t e, const char* what) {
  set_error("%s: %s", what, hipGetErrorString(e));
  return FD_E_HIP;
}

int num_cus() {
  static int cache[64];
  static std::once_flag once[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  std::call_once(once[dev], [&] {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) n = 256;
    cache[dev] = n;
  });
  return cache[dev];
}

void timer_begin(int kernel, hipStream_t s) {
  std::lock_guard<std::mutex> lk(g_timer.mu);
  if (g_timer.kernel != kernel || g_timer.count >= g_timer.capacity) return;
  (void)hipEventRecord(g_timer.ev[2 * g_timer.count], s);
}

void timer_end(int kernel, hipStream_t s) {
  std::lock_guard<std::mutex> lk(g_timer.mu);
  if (g_timer.kernel != kernel || g_timer.count >= g_timer.capacity) return;
  (void)hipEventRecord(g_timer.ev[2 * g_timer.count + 1], s);
  ++g_timer.count;
}

}  // namespace fdh

extern "C" {

const char* fd_last_error(void) { return g_err; }
const char* fd_version(void) { return "flashdiff-mi355x 0.1 (gfx950)"; }

fd_status fd_plan_build(int32_t n_tokens, int32_t n_regions, int32_t n_requests, const int32_t* token_region,
                        const int32_t* req_tok_off, int32_t* region_ptr, int32_t* region_tokens, int32_t* region_req,
                        int32_t* req_reg_off, int32_t* max_region_tokens, int32_t* max_request_tokens) {
  FD_REQUIRE(n_tokens >= 1 && n_regions >= 1 && n_requests >= 1, "sizes must be positive");
  FD_REQUIRE(n_regions <= n_tokens, "more regions (%d) than tokens (%d)", n_regions, n_tokens);
  FD_REQUIRE(token_region && req_tok_off && region_ptr && region_tokens && region_req && req_reg_off &&
                 max_region_tokens && max_request_tokens,
             "null pointer");
  FD_REQUIRE(req_tok_off[0] == 0 && req_tok_off[n_requests] == n_tokens, "req_tok_off must span [0, N]");
  int max_req = 0;
  for (int b = 0; b < n_requests; ++b) {
    const int nb = req_tok_off[b + 1] - req_tok_off[b];
    FD_REQUIRE(nb >= 1, "request %d has no tokens", b);
    if (nb > max_req) max_req = nb;
  }
  std::vector<int32_t> cnt(n_regions, 0);
  for (int u = 0; u < n_tokens; ++u) {
    const int r = token_region[u];
    FD_REQUIRE(r >= 0 && r < n_regions, "token %d has region %d outside [0, %d)", u, r, n_regions);
    ++cnt[r];
  }
  region_ptr[0] = 0;
  int max_reg = 0;
  for (int r = 0; r < n_regions; ++r) {
    FD_REQUIRE(cnt[r] >= 1, "region %d is empty", r);
    region_ptr[r + 1] = region_ptr[r] + cnt[r];
    if (cnt[r] > max_reg) max_reg = cnt[r];
    region_req[r] = -1;
  }
  std::vector<int32_t> fill(region_ptr, region_ptr + n_regions);
  int b = 0;
  for (int u = 0; u < n_tokens; ++u) {
    while (u >= req_tok_off[b + 1]) ++b;
    const int r = token_region[u];
    if (region_req[r] < 0) region_req[r] = b;
    FD_REQUIRE(region_req[r] == b, "region %d spans requests %d and %d", r, region_req[r], b);
    region_tokens[fill[r]++] = u;
  }
  for (int r = 1; r < n_regions; ++r)
    FD_REQUIRE(region_req[r] >= region_req[r - 1], "region ids are not request-major at region %d", r);
  int r = 0;
  for (int bb = 0; bb < n_requests; ++bb) {
    req_reg_off[bb] = r;
    while (r < n_regions && region_req[r] == bb) ++r;
  }
  req_reg_off[n_requests] = r;
  *max_region_tokens = max_reg;
  *max_request_tokens = max_req;
  return FD_OK;
}

size_t fd_region_score_ws_size(const fd_plan* plan, int32_t C) {
  if (!plan || C < 1) return 0;
  const int rows = score_rows_per_chunk(C);
  const int nchunk = (plan->max_region_tokens + rows - 1) / rows;
  return align_up(static_cast<size_t>(plan->n_regions) * nchunk * sizeof(double));
}

fd_status fd_region_score(const fd_plan* plan, int32_t C, const float* x_cur, const float* x_prev, double* score,
                          void* ws, size_t ws_bytes, fd_stream_t stream) {
  FD_TRY(check_plan(plan));
  FD_TRY(check_C(C));
  FD_REQUIRE(x_cur && x_prev && score && ws, "null pointer");
  FD_REQUIRE(aligned(x_cur, 16) && aligned(x_prev, 16) && aligned(ws, 8), "misaligned buffer");
  if (ws_bytes < fd_region_score_ws_size(plan, C)) return fdh::set_error("score workspace too small"), FD_E_SHAPE;
  // regions cut into chunks of `rows` tokens, unless there are enough regions to
  // fill the GPU one workgroup each (then one pass, no finalize)
  int rows = score_rows_per_chunk(C);
  if (plan->n_regions >= 2 * fdh::num_cus()) rows = plan->max_region_tokens > 0 ? plan->max_region_tokens : 1;
  const int nchunk = (plan->max_region_tokens + rows - 1) / rows;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FD_LAUNCH(FD_K_SCORE, s,
            fdh::launch_region_score(plan, C, x_cur, x_prev, score, static_cast<double*>(ws), nchunk, rows, s));
  return FD_OK;
}

// ---------------------------------------------------------------- region score without allocation
// The partial sums of fd_region_score_noalloc live in this file-scope device array
// (one copy per GPU, held until the process ends).  In host code its name is not a
// device address: every host use goes through the address hipGetSymbolAddress
// returns for the current device, taken once per device.
}  // extern "C"

namespace {

constexpr size_t kScoreScratchBytes = size_t(1) << 20;   // 131072 (region, chunk) partial sums
__device__ __align__(256) unsigned char scratch[kScoreScratchBytes];

constexpr int kMaxDevices = 64;
struct ScratchAddr {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t err = hipSuccess;
};
ScratchAddr g_scratch[kMaxDevices];

// Device address of `scratch` on the current device (looked up on the first call per device).
fd_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fdh::hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fdh::set_error("device %d beyond the scratch table", dev), FD_E_UNSUPPORTED;
  ScratchAddr& a = g_scratch[dev];
  std::call_once(a.once, [&] { a.err = hipGetSymbolAddress(&a.ptr, HIP_SYMBOL(scratch)); });
  if (a.err != hipSuccess || !a.ptr) return fdh::hip_fail(a.err, "hipGetSymbolAddress(scratch)");
  *out = a.ptr;
  return FD_OK;
}

}  // namespace

extern "C" {

fd_status fd_region_score_noalloc(const fd_plan* plan, int32_t C, const float* x_cur, const float* x_prev,
                                  double* score, fd_stream_t stream) {
  FD_TRY(check_plan(plan));
  FD_TRY(check_C(C));
  FD_REQUIRE(x_cur && x_prev && score, "null pointer");
  FD_REQUIRE(aligned(x_cur, 16) && aligned(x_prev, 16), "misaligned buffer");
  const size_t need = fd_region_score_ws_size(plan, C);
  if (need > kScoreScratchBytes)
    return fdh::set_error("score partials need %zu bytes, beyond the %zu-byte built-in scratch (use fd_region_score)",
                          need, kScoreScratchBytes),
           FD_E_UNSUPPORTED;
  void* ws = nullptr;
  FD_TRY(scratch_address(&ws));
  int rows = score_rows_per_chunk(C);
  if (plan->n_regions >= 2 * fdh::num_cus()) rows = plan->max_region_tokens > 0 ? plan->max_region_tokens : 1;
  const int nchunk = (plan->max_region_tokens + rows - 1) / rows;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FD_LAUNCH(FD_K_SCORE, s,
            fdh::launch_region_score(plan, C, x_cur, x_prev, score, static_cast<double*>(ws), nchunk, rows, s));
  return FD_OK;
}

fd_status fd_select(const fd_plan* plan, const double* score, const double* eps, fd_gate gate, double* s_tilde,
                    int32_t* skip_run, const uint8_t* prev_active, uint8_t* active, int32_t* idx, int32_t* cu_q,
                    int32_t* m, fd_stream_t stream) {
  FD_TRY(check_plan(plan));
  FD_REQUIRE(score && eps && s_tilde && skip_run && prev_active && active && idx && cu_q && m, "null pointer");
  if (plan->n_regions > 4096 || plan->n_requests > 1024)
    return fdh::set_error("select supports R <= 4096 and B <= 1024"), FD_E_UNSUPPORTED;
  FD_REQUIRE(gate.eta >= 0.0 && gate.max_skip >= 0, "eta and max_skip must be >= 0");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FD_LAUNCH(FD_K_SELECT, s,
            fdh::launch_select(plan, score, eps, gate, s_tilde, skip_run, prev_active, active, idx, cu_q, m, s));
  return FD_OK;
}

fd_status fd_gather(const fd_plan* plan, int32_t C, const float* x_cur, const int32_t* idx, const int32_t* m,
                    uint16_t* xa, fd_stream_t stream) {
  FD_TRY(check_plan(plan));
  FD_TRY(check_C(C));
  FD_REQUIRE(x_cur && idx && m && xa, "null pointer");
  FD_REQUIRE(aligned(x_cur, 16) && aligned(xa, 8), "misaligned buffer");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FD_LAUNCH(FD_K_GATHER, s, fdh::launch_gather(plan, C, x_cur, idx, m, xa, s));
  return FD_OK;
}

fd_status fd_embed(const fd_plan* plan, const fd_dims* dims, const uint16_t* xa, const uint16_t* w_e, const float* b_e,
                   const float* pos, const int32_t* idx, const int32_t* m, float* h, fd_stream_t stream) {
  FD_TRY(check_plan(plan));
  FD_TRY(check_dims(dims));
  FD_REQUIRE(xa && w_e && b_e && pos && idx && m && h, "null pointer");
  FD_REQUIRE(aligned(xa, 16) && aligned(w_e, 16), "misaligned buffer");
  fdh::GemmArgs g{};
  g.act = xa; g.wt = w_e; g.bias = b_e; g.n_max = plan->n_tokens; g.m = m; g.N = dims->D; g.K = dims->C;
  g.idx = idx; g.out_f32 = h; g.pos = pos;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FD_LAUNCH(FD_K_EMBED, s, fdh::launch_gemm(fdh::GEMM_EMBED, g, s));
  return FD_OK;
}

fd_status fd_adaln(const fd_dims* dims, int32_t n_blocks, int32_t n_out, int32_t n_requests, const uint16_t* w_ada,
                   const float* b_ada, const float* cond, float* mod, fd_stream_t stream) {
  FD_TRY(check_dims(dims));
  FD_REQUIRE(w_ada && b_ada && cond && mod, "null pointer");
  FD_REQUIRE(n_blocks >= 1 && n_out >= 1 && n_requests >= 1, "n_blocks, n_out and n_requests must be positive");
  FD_REQUIRE(static_cast<long long>(n_blocks) * n_out <= (1LL << 28), "too many modulation rows");
  FD_REQUIRE(aligned(w_ada, 16) && aligned(cond, 16), "misaligned buffer");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FD_LAUNCH(FD_K_ADALN, s,
            fdh::launch_adaln(w_ada, b_ada, cond, n_requests, dims->D, n_out, n_blocks, mod, s));
  return FD_OK;
}

size_t fd_block_ws_size(const fd_plan* plan, const fd_dims* dims) {
  if (!plan || !dims) return 0;
  return carve_block_ws(plan, dims, nullptr).bytes;
}

fd_status fd_block_forward(const fd_plan* plan, const fd_dims* dims, const fd_block_weights* w, const float* cond,
                           float* h, const int32_t* idx, const int32_t* cu_q, const int32_t* m, uint16_t* k_cache,
                           uint16_t* v_cache, void* ws, size_t ws_bytes, fd_stream_t stream) {
  FD_TRY(check_plan(plan));
  FD_TRY(check_dims(dims));
  FD_REQUIRE(w && h && idx && cu_q && m && k_cache && v_cache && ws, "null pointer");
  FD_REQUIRE(w->w_qkv && w->b_qkv && w->w_o && w->b_o && w->w_1 && w->b_1 && w->w_2 && w->b_2 &&
                 (w->mod || (w->w_ada && w->b_ada && cond)),
             "null weight pointer");
  FD_REQUIRE(aligned(w->w_qkv, 16) && aligned(w->w_o, 16) && aligned(w->w_1, 16) && aligned(w->w_2, 16) &&
                 (w->mod ? aligned(w->mod, 16) : aligned(w->w_ada, 16)) && aligned(h, 16) && aligned(k_cache, 16) &&
                 aligned(v_cache, 16) && aligned(ws, kAlign),
             "misaligned buffer");
  if (plan->n_requests > fdh::kMaxAttnRequests)
    return fdh::set_error("the block supports at most %d requests per call (%d given)", fdh::kMaxAttnRequests,
                          plan->n_requests),
           FD_E_UNSUPPORTED;
  const BlockWs bw = carve_block_ws(plan, dims, ws);
  if (ws_bytes < bw.bytes) return fdh::set_error("block workspace too small (%zu < %zu)", ws_bytes, bw.bytes), FD_E_SHAPE;
  const int D = dims->D, F = dims->F, B = plan->n_requests, N = plan->n_tokens;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);

  // modulation: precomputed by fd_adaln, else computed here
  const float* mod = w->mod ? w->mod : bw.mod;
  if (!w->mod)
    FD_LAUNCH(FD_K_ADALN, s,
              fdh::launch_adaln(w->w_ada, w->b_ada, cond, B, D, 6 * D, 1, bw.mod, s));
  FD_LAUNCH(FD_K_LN, s, fdh::launch_ln_modulate(h, cu_q, B, m, N, D, mod, 6 * D, 0, D, bw.a, idx, plan->token_region,
                                                        plan->region_req, s));
  fdh::GemmArgs g{};
  g.n_max = N; g.m = m; g.idx = idx; g.cu_q = cu_q; g.n_req = B; g.D = D;
  g.partial = bw.partial; g.max_units = fdh::gemm_max_tiles();
  g.act = bw.a; g.wt = w->w_qkv; g.bias = w->b_qkv; g.N = 3 * D; g.K = D;
  g.out_bf16 = bw.q; g.k_cache = k_cache; g.v_cache = v_cache;
  FD_LAUNCH(FD_K_GEMM_QKV, s, fdh::launch_gemm(fdh::GEMM_QKV, g, s));
  FD_LAUNCH(FD_K_ATTN, s,
            fdh::launch_attention(bw.q, k_cache, v_cache, bw.o, D, dims->H, dims->dh, cu_q, plan->req_tok_off, B, N,
                                  plan->max_request_tokens, bw.partial, bw.lse, s));
  g = fdh::GemmArgs{};
  g.n_max = N; g.m = m; g.idx = idx; g.cu_q = cu_q; g.n_req = B; g.D = D;
  g.partial = bw.partial; g.max_units = fdh::gemm_max_tiles();
  g.act = bw.o; g.wt = w->w_o; g.bias = w->b_o; g.N = D; g.K = D;
  g.out_f32 = h; g.gate = mod + 2 * D; g.gate_stride = 6 * D;
  FD_LAUNCH(FD_K_GEMM_O, s, fdh::launch_gemm(fdh::GEMM_RESID, g, s));
  FD_LAUNCH(FD_K_LN, s, fdh::launch_ln_modulate(h, cu_q, B, m, N, D, mod, 6 * D, 3 * D, 4 * D, bw.a, idx,
                                                        plan->token_region, plan->region_req, s));
  g = fdh::GemmArgs{};
  g.n_max = N; g.m = m; g.idx = idx; g.cu_q = cu_q; g.n_req = B; g.D = D;
  g.partial = bw.partial; g.max_units = fdh::gemm_max_tiles();
  g.act = bw.a; g.wt = w->w_1; g.bias = w->b_1; g.N = F; g.K = D; g.out_bf16 = bw.g;
  FD_LAUNCH(FD_K_GEMM_MLP1, s, fdh::launch_gemm(fdh::GEMM_GELU, g, s));
  g = fdh::GemmArgs{};
  g.n_max = N; g.m = m; g.idx = idx; g.cu_q = cu_q; g.n_req = B; g.D = D;
  g.partial = bw.partial; g.max_units = fdh::gemm_max_tiles();
  g.act = bw.g; g.wt = w->w_2; g.bias = w->b_2; g.N = D; g.K = F;
  g.out_f32 = h; g.gate = mod + 5 * D; g.gate_stride = 6 * D;
  FD_LAUNCH(FD_K_GEMM_MLP2, s, fdh::launch_gemm(fdh::GEMM_RESID, g, s));
  return FD_OK;
}

size_t fd_importance_ws_size(const fd_plan* plan, const fd_dims* dims) {
  if (!plan || !dims) return 0;
  return align_up(static_cast<size_t>(plan->n_tokens) * sizeof(int32_t)) +
         align_up(static_cast<size_t>(plan->n_regions) * dims->H * sizeof(float));
}

fd_status fd_region_importance(const fd_plan* plan, const fd_dims* dims, const void* block_ws, size_t block_ws_bytes,
                               const uint16_t* k_cache, const int32_t* idx, const int32_t* m, const uint8_t* active,
                               double* r_bar, double* delta, double* importance, void* ws, size_t ws_bytes,
                               fd_stream_t stream) {
  FD_TRY(check_plan(plan));
  FD_TRY(check_dims(dims));
  FD_REQUIRE(block_ws && k_cache && idx && m && active && r_bar && delta && ws, "null pointer");
  FD_REQUIRE(aligned(block_ws, kAlign) && aligned(ws, kAlign) && aligned(k_cache, 16), "misaligned buffer");
  const BlockWs bw = carve_block_ws(plan, dims, const_cast<void*>(block_ws));
  if (block_ws_bytes < bw.bytes)
    return fdh::set_error("block workspace too small (%zu < %zu)", block_ws_bytes, bw.bytes), FD_E_SHAPE;
  const size_t need = fd_importance_ws_size(plan, dims);
  if (ws_bytes < need) return fdh::set_error("importance workspace too small (%zu < %zu)", ws_bytes, need), FD_E_SHAPE;
  if (fdh::importance_lds_bytes(dims->dh, plan->max_region_tokens) > 156 * 1024)
    return fdh::set_error("regions of %d tokens exceed the importance kernel's LDS staging", plan->max_region_tokens),
           FD_E_UNSUPPORTED;
  const uintptr_t b0 = reinterpret_cast<uintptr_t>(ws);
  int32_t* pos = reinterpret_cast<int32_t*>(b0);
  float* part = reinterpret_cast<float*>(b0 + align_up(static_cast<size_t>(plan->n_tokens) * sizeof(int32_t)));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FD_LAUNCH(FD_K_IMPORTANCE, s,
            fdh::launch_importance(plan, dims->D, dims->H, dims->dh, idx, m, active, bw.q, k_cache, bw.lse, pos, part,
                                   r_bar, delta, importance, s));
  return FD_OK;
}

size_t fd_partition_ws_size(int32_t n_tokens, int32_t n_requests) {
  if (n_tokens < 0 || n_requests < 1) return 0;
  return fdh::partition_ws_bytes(n_tokens, n_requests);
}

fd_status fd_partition(int32_t n_requests, const int32_t* req_tok_off, const int32_t* req_reg_off,
                       const uint16_t* saliency, int32_t* token_region, void* ws, size_t ws_bytes,
                       fd_stream_t stream) {
  FD_REQUIRE(req_tok_off && req_reg_off && saliency && token_region && ws, "null pointer");
  FD_REQUIRE(n_requests >= 1, "n_requests = %d", n_requests);
  if (n_requests > fd::kMaxPartRequests)
    return fdh::set_error("%d requests exceed the partitioner's %d per call", n_requests, fd::kMaxPartRequests),
           FD_E_UNSUPPORTED;
  FD_REQUIRE(req_tok_off[0] == 0 && req_reg_off[0] == 0, "offsets must start at 0");
  for (int b = 0; b < n_requests; ++b) {
    const int n = req_tok_off[b + 1] - req_tok_off[b], r = req_reg_off[b + 1] - req_reg_off[b];
    FD_REQUIRE(r >= 1 && n >= r, "request %d: %d tokens cannot fill %d regions", b, n, r);
    if (n > fd::kMaxPartTokens || r > fd::kMaxPartRegions)
      return fdh::set_error("request %d: %d tokens / %d regions exceed the partitioner's %d / %d", b, n, r,
                            fd::kMaxPartTokens, fd::kMaxPartRegions),
             FD_E_UNSUPPORTED;
  }
  FD_REQUIRE(aligned(ws, kAlign), "misaligned buffer");
  const size_t need = fdh::partition_ws_bytes(req_tok_off[n_requests], n_requests);
  if (ws_bytes < need) return fdh::set_error("partition workspace too small (%zu < %zu)", ws_bytes, need), FD_E_SHAPE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FD_LAUNCH(FD_K_PARTITION, s,
            fdh::launch_partition(n_requests, req_tok_off, req_reg_off, saliency, token_region, ws, s));
  return FD_OK;
}

fd_status fd_final(const fd_plan* plan, const fd_dims* dims, const fd_final_weights* w, const float* cond,
                   const float* h, const int32_t* cu_q, const int32_t* m, float* v, void* ws, size_t ws_bytes,
                   fd_stream_t stream) {
  FD_TRY(check_plan(plan));
  FD_TRY(check_dims(dims));
  FD_REQUIRE(w && w->w_ada && w->b_ada && w->w_out && w->b_out && cond && h && cu_q && m && v && ws, "null pointer");
  FD_REQUIRE(aligned(w->w_ada, 16) && aligned(w->w_out, 16) && aligned(h, 16) && aligned(ws, kAlign),
             "misaligned buffer");
  const BlockWs bw = carve_block_ws(plan, dims, ws);
  if (ws_bytes < bw.bytes) return fdh::set_error("final workspace too small"), FD_E_SHAPE;
  const int D = dims->D, B = plan->n_requests, N = plan->n_tokens;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FD_LAUNCH(FD_K_ADALN, s,
            fdh::launch_adaln(w->w_ada, w->b_ada, cond, B, D, 2 * D, 1, bw.mod, s));
  FD_LAUNCH(FD_K_LN, s, fdh::launch_ln_modulate(h, cu_q, B, m, N, D, bw.mod, 2 * D, 0, D, bw.a, nullptr, nullptr, nullptr, s));
  fdh::GemmArgs g{};
  g.n_max = N; g.m = m; g.cu_q = cu_q; g.n_req = B;
  g.partial = bw.partial; g.max_units = fdh::gemm_max_tiles();
  g.act = bw.a; g.wt = w->w_out; g.bias = w->b_out; g.N = dims->C; g.K = D; g.out_f32 = v;
  FD_LAUNCH(FD_K_FINAL, s, fdh::launch_gemm(fdh::GEMM_OUT, g, s));
  return FD_OK;
}

fd_status fd_scatter_update(const fd_plan* plan, int32_t C, float* x, const float* v, const int32_t* idx,
                            const int32_t* m, const float* dt, float* vcache, const uint8_t* active, int32_t skip_mode,
                            fd_stream_t stream) {
  FD_TRY(check_plan(plan));
  FD_TRY(check_C(C));
  FD_REQUIRE(x && v && idx && m && dt && vcache && active, "null pointer");
  FD_REQUIRE(skip_mode == FD_SKIP_FREEZE || skip_mode == FD_SKIP_REUSE_DRIFT, "unknown skip mode %d", skip_mode);
  FD_REQUIRE(aligned(x, 16) && aligned(v, 16) && aligned(vcache, 16), "misaligned buffer");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FD_LAUNCH(FD_K_SCATTER, s, fdh::launch_scatter_update(plan, C, x, v, idx, m, dt, vcache, active, skip_mode, s));
  return FD_OK;
}

fd_status fd_timer_arm(int32_t kernel, int32_t capacity) {
  FD_REQUIRE(kernel >= FD_K_SCORE && kernel <= FD_K_PARTITION && capacity >= 1 && capacity <= (1 << 20),
             "bad timer arguments");
  std::lock_guard<std::mutex> lk(g_timer.mu);
  for (hipEvent_t e : g_timer.ev) (void)hipEventDestroy(e);
  g_timer.ev.assign(2 * static_cast<size_t>(capacity), nullptr);
  // timing-only events: no system-scope fence (cache write-back and invalidate) at
  // each record, which would stall the stream between the kernels around it
  for (auto& e : g_timer.ev) {
    hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
    if (r != hipSuccess) {
      g_timer.kernel = 0;
      g_timer.capacity = 0;
      return fdh::hip_fail(r, "hipEventCreateWithFlags");
    }
  }
  g_timer.kernel = kernel;
  g_timer.capacity = capacity;
  g_timer.count = 0;
  return FD_OK;
}

int32_t fd_timer_read(float* ms, int32_t capacity) {
  std::lock_guard<std::mutex> lk(g_timer.mu);
  const int n = g_timer.count < capacity ? g_timer.count : capacity;
  for (int i = 0; i < n; ++i) {
    if (hipEventSynchronize(g_timer.ev[2 * i + 1]) != hipSuccess ||
        hipEventElapsedTime(&ms[i], g_timer.ev[2 * i], g_timer.ev[2 * i + 1]) != hipSuccess)
      ms[i] = -1.f;
  }
  return n;
}

void fd_timer_disarm(void) {
  std::lock_guard<std::mutex> lk(g_timer.mu);
  for (hipEvent_t e : g_timer.ev) (void)hipEventDestroy(e);
  g_timer.ev.clear();
  g_timer.kernel = 0;
  g_timer.capacity = 0;
  g_timer.count = 0;
}

}  // extern "C"
