// Internal helpers shared by the HIP kernels of the region-sparse step (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "flashdiff.h"

#define FD_DEVICE __device__ __forceinline__

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

namespace fd {

constexpr int kWave = 64;

// Patch partitioner limits: requests per call, regions and tokens per request
// (per-request counts stay below 2^16 so that two value counts share a word).
constexpr int kMaxPartRequests = 64;
constexpr int kMaxPartRegions = 1024;
constexpr int kMaxPartTokens = 65535;

// fp32 -> bf16 bits, round to nearest even (hardware conversion on gfx950).
FD_DEVICE uint16_t f2bf(float x) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(x)); }
FD_DEVICE float bf2f(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
// two fp32 -> packed bf16 pair (lo in the low half), one v_cvt_pk_bf16_f32, round to nearest even
FD_DEVICE uint32_t pack_bf2(float lo, float hi) {
  const f32x2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

FD_DEVICE float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
FD_DEVICE double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
FD_DEVICE int wave_sum(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Request of active row i < cu_q[B]: the b with cu_q[b] <= i < cu_q[b+1], found as the
// largest b < B with cu_q[b] <= i (binary search over the ascending offsets; among
// empty requests sharing an offset the largest one is the row's).  O(log B) loads.
FD_DEVICE int row_request(const int32_t* __restrict__ cu_q, int B, int i) {
  int lo = 0, hi = B - 1;   // cu_q[lo] <= i always (cu_q[0] = 0)
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu_q[mid] <= i) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// GELU, tanh form: z/2 (1 + tanh(u)), u = sqrt(2/pi) (z + 0.044715 z^3).  Uses the
// identity (1 + tanh(u)) / 2 = 1 / (1 + exp(-2u)), i.e. one exponential and one division.
FD_DEVICE float gelu_tanh(float z) {
  const float k2 = 1.5957691216057308f;  // 2 sqrt(2/pi)
  const float t = k2 * (z + 0.044715f * z * z * z);
  return z / (1.0f + __expf(-t));
}
// The same GELU with hardware exp2 and reciprocal (about 2 ulp): used in the MLP
// epilogue, whose result is rounded to bf16 right after.
FD_DEVICE float gelu_tanh_fast(float z) {
  const float k2l = 2.302208198144325f;  // 2 sqrt(2/pi) log2(e)
  const float t = k2l * (z + 0.044715f * z * z * z);
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-t));
}

}  // namespace fd

// ------------------------------------------------------------------ host side

namespace fdh {

// Thread-local error message (set on failure, read by fd_last_error).
void set_error(const char* fmt, ...);
fd_status hip_fail(hipError_t e, const char* what);

// Timer hooks around a launch (no-ops unless the timer is armed for `kernel`).
void timer_begin(int kernel, hipStream_t s);
void timer_end(int kernel, hipStream_t s);

int num_cus();

// Launchers (defined in the kernel files; arguments already validated).
hipError_t launch_region_score(const fd_plan* p, int C, const float* xc, const float* xp, double* score,
                               double* partial, int nchunk, int rows_per_chunk, hipStream_t s);
hipError_t launch_select(const fd_plan* p, const double* score, const double* eps, fd_gate g,
                         double* s_tilde, int32_t* skip_run, const uint8_t* prev_active, uint8_t* active,
                         int32_t* idx, int32_t* cu_q, int32_t* m, hipStream_t s);
hipError_t launch_gather(const fd_plan* p, int C, const float* x, const int32_t* idx, const int32_t* m,
                         uint16_t* xa, hipStream_t s);
hipError_t launch_scatter_update(const fd_plan* p, int C, float* x, const float* v, const int32_t* idx,
                                 const int32_t* m, const float* dt, float* vcache, const uint8_t* active,
                                 int skip_mode, hipStream_t s);
hipError_t launch_adaln(const uint16_t* w, const float* b, const float* cond, int B, int D, int n_out, int n_blocks,
                        float* mod, hipStream_t s);
// The row's request: from idx and the plan's token -> region -> request tables
// when idx is given, else by binary search in cu_q.
hipError_t launch_ln_modulate(const float* h, const int32_t* cu_q, int B, const int32_t* m, int n_max, int D,
                              const float* mod, int mod_stride, int shift_off, int scale_off, uint16_t* a,
                              const int32_t* idx, const int32_t* token_region, const int32_t* region_req,
                              hipStream_t s);

// GEMM epilogue kinds.
enum GemmKind { GEMM_QKV = 0, GEMM_RESID = 1, GEMM_GELU = 2, GEMM_EMBED = 3, GEMM_OUT = 4 };

struct GemmArgs {
  const uint16_t* act;   // [M][K] bf16 activations
  const uint16_t* wt;    // [N][K] bf16 weights
  const float* bias;     // [N]
  int n_max;             // row capacity (upper bound of M)
  const int32_t* m;      // device active row count
  int N, K;
  // epilogue operands
  const int32_t* idx;    // token of each row (QKV cache scatter, EMBED position)
  const int32_t* cu_q; int n_req;
  uint16_t* out_bf16;    // QKV: q [M][D]; GELU: g [M][N]
  uint16_t* k_cache; uint16_t* v_cache; int D;  // QKV
  float* out_f32;        // RESID: h [M][N] (+=); EMBED: h [M][N]; OUT: v [M][N]
  const float* gate; int gate_stride;          // RESID: gate row per request
  const float* pos;      // EMBED: [N_tok][N]
  // split-K scratch (tiled kernel): fp32 partial tiles, summed by a second kernel
  float* partial; int max_units;
};
// Bytes of split-K scratch the tiled GEMM needs (fp32 partial tiles), for any shape.
size_t gemm_scratch_bytes();
int gemm_max_tiles();
hipError_t launch_gemm(GemmKind kind, const GemmArgs& a, hipStream_t s);

// Requests per attention launch (its schedule tables live in LDS).
constexpr int kMaxAttnRequests = 1024;
hipError_t launch_attention(const uint16_t* q, const uint16_t* kc, const uint16_t* vc, uint16_t* o, int D, int H,
                            int dh, const int32_t* cu_q, const int32_t* req_tok_off, int B, int n_max,
                            int max_req_tokens, float* partial, float* lse, hipStream_t s);
// Region importance (pos: active row of every token, part: [R][H] partial sums).
size_t importance_lds_bytes(int dh, int max_region_tokens);
hipError_t launch_importance(const fd_plan* p, int D, int H, int dh, const int32_t* idx, const int32_t* m,
                             const uint8_t* active, const uint16_t* q, const uint16_t* kc, const float* lse,
                             int32_t* pos, float* part, double* r_bar, double* delta, double* importance,
                             hipStream_t s);

// Patch partitioner: workspace bytes and the one-launch recursion (offsets are host arrays).
size_t partition_ws_bytes(int n_tokens, int n_requests);
hipError_t launch_partition(int n_requests, const int32_t* req_tok_off, const int32_t* req_reg_off,
                            const uint16_t* saliency, int32_t* region, void* ws, hipStream_t s);

// Bytes of KV-split scratch the attention kernel needs for head dim dh.
size_t attn_scratch_bytes(int dh);

}  // namespace fdh
