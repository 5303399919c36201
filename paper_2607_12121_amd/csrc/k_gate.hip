// Gate-side kernels of the region-sparse step: region activity score, Patch Gate
// selection with token compaction, bf16 gather of active latent rows, and the
// Euler scatter-update of the latent.  All are HBM- or latency-bound streams.
#include "fd_common.h"

namespace {

constexpr int kScoreThreads = 256;
constexpr int kUnroll = 4;   // independent rows / elements in flight per thread (score)
// float4 elements per thread (the loads of all of them in flight before the first
// store): measured at 256 requests, gather 63 -> 66% of HBM peak with 4 instead of
// 8, the update 65 -> 68% with 2 (1 was slower for both)
constexpr int kGatherUnroll = 4;
constexpr int kUpdateUnroll = 2;
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Partial activity of one chunk of one region: sum of d^2 over `rows_per_chunk`
// token rows, d = fl32(x_cur - x_prev), accumulated in fp64.  One workgroup per
// (chunk, region); float4 loads, consecutive lanes on consecutive channels, each
// thread's loads for kUnroll elements issued before any is used.  With a single
// chunk per region the workgroup writes the score itself (no finalize pass).
__global__ __launch_bounds__(kScoreThreads) void region_score_partial_kernel(
    const int32_t* __restrict__ region_ptr, const int32_t* __restrict__ region_tokens,
    const float* __restrict__ xc, const float* __restrict__ xp, int C, int rows_per_chunk,
    double* __restrict__ partial, double* __restrict__ score) {
  const int r = blockIdx.y;
  const int nchunk = gridDim.x;
  const int t0 = region_ptr[r], t1 = region_ptr[r + 1];
  const int row0 = t0 + blockIdx.x * rows_per_chunk;
  const int row1 = min(t1, row0 + rows_per_chunk);
  const int c4 = C >> 2;
  const int n_el = row1 > row0 ? (row1 - row0) * c4 : 0;
  double acc = 0.0;
  for (int e0 = threadIdx.x; e0 < n_el; e0 += kScoreThreads * kUnroll) {
    float4 a[kUnroll], b[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const int e = e0 + k * kScoreThreads;
      a[k] = make_float4(0.f, 0.f, 0.f, 0.f);
      b[k] = a[k];
      if (e < n_el) {
        const int row = row0 + e / c4;
        const int col = e - (e / c4) * c4;
        const size_t off = static_cast<size_t>(region_tokens[row]) * C;
        // streaming loads: 74 -> 84% of HBM peak at 256 requests
        const f32x4_t ta = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(xc + off) + col);
        const f32x4_t tb = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(xp + off) + col);
        a[k] = make_float4(ta.x, ta.y, ta.z, ta.w);
        b[k] = make_float4(tb.x, tb.y, tb.z, tb.w);
      }
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const double d0 = static_cast<double>(a[k].x - b[k].x);
      const double d1 = static_cast<double>(a[k].y - b[k].y);
      const double d2 = static_cast<double>(a[k].z - b[k].z);
      const double d3 = static_cast<double>(a[k].w - b[k].w);
      acc += (d0 * d0 + d1 * d1) + (d2 * d2 + d3 * d3);
    }
  }
  acc = fd::wave_sum(acc);
  __shared__ double wsum[kScoreThreads / fd::kWave];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wsum[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < kScoreThreads / fd::kWave; ++w) s += wsum[w];
    if (nchunk == 1)
      score[r] = (0.0 + s) / (static_cast<double>(t1 - t0) * static_cast<double>(C));   // as the finalize pass
    else
      partial[static_cast<size_t>(r) * nchunk + blockIdx.x] = s;
  }
}

// score[r] = (sum of the region's partials, in chunk order) / (|r| * C).
__global__ void region_score_finalize_kernel(const int32_t* __restrict__ region_ptr,
                                             const double* __restrict__ partial, int nchunk, int R, int C,
                                             double* __restrict__ score) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= R) return;
  double s = 0.0;
  for (int c = 0; c < nchunk; ++c) s += partial[static_cast<size_t>(r) * nchunk + c];
  const double n = static_cast<double>(region_ptr[r + 1] - region_ptr[r]) * static_cast<double>(C);
  score[r] = s / n;
}

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / fd::kWave;
constexpr int kMaxRegions = 4096;
constexpr int kMaxRequests = 1024;

// Patch Gate + compaction in one workgroup (R <= 4096, B <= 1024).
__global__ __launch_bounds__(kSelThreads) void gate_select_kernel(
    int R, int B, int N, const int32_t* __restrict__ region_req, const int32_t* __restrict__ req_reg_off,
    const int32_t* __restrict__ region_ptr, const int32_t* __restrict__ token_region,
    const double* __restrict__ score, const double* __restrict__ eps, double eta, int max_skip,
    double* __restrict__ s_tilde, int32_t* __restrict__ skip_run, const uint8_t* prev_active,
    uint8_t* active, int32_t* __restrict__ idx, int32_t* __restrict__ cu_q, int32_t* __restrict__ m_out) {
  __shared__ double st_s[kMaxRegions];
  __shared__ double d_s[kMaxRequests];
  __shared__ int cnt_s[kMaxRequests];
  __shared__ uint8_t act_s[kMaxRegions];
  __shared__ int wtot_s[kSelWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // 1. frozen change: refresh the score of regions executed at the previous step
  for (int r = tid; r < R; r += kSelThreads) {
    const double st = prev_active[r] ? score[r] : s_tilde[r];
    st_s[r] = st;
  }
  __syncthreads();
  for (int r = tid; r < R; r += kSelThreads) s_tilde[r] = st_s[r];

  // 2. D_b = sum over the request's regions of fl(s~ + eta), added one at a time in
  //    ascending region order: a fixed order, so that D_b rounds the same way in
  //    every evaluation of the gate and the decisions are reproducible bit for bit.
  for (int b = tid; b < B; b += kSelThreads) {
    const int lo = req_reg_off[b], hi = req_reg_off[b + 1];
    double s = 0.0;
    for (int r = lo; r < hi; ++r) s += st_s[r] + eta;
    d_s[b] = s;
  }
  __syncthreads();

  // 3-5. threshold, forced reactivation, skip counters
  for (int r = tid; r < R; r += kSelThreads) {
    const int b = region_req[r];
    const double e = eps[b];
    const int run = skip_run[r];
    const bool forced = max_skip > 0 && run >= max_skip;
    // below the threshold: fl(s~ + eta) < fl(eps D_b) (1 - 2^-40).  The band makes every
    // exact-arithmetic tie active (D_b's rounding error is below 2^-40 relative for
    // R <= 4096); NaN compares false (active).
    const bool below = (e == INFINITY) ? true : ((st_s[r] + eta) < (e * d_s[b]) * (1.0 - 0x1p-40));
    const bool act = forced || !below;
    act_s[r] = act ? 1 : 0;
    active[r] = act ? 1 : 0;
    skip_run[r] = act ? 0 : run + 1;
  }
  __syncthreads();

  // 6a. active tokens per request -> cu_q, m
  for (int b = wave; b < B; b += kSelWaves) {
    const int lo = req_reg_off[b], hi = req_reg_off[b + 1];
    int c = 0;
    for (int r = lo + lane; r < hi; r += fd::kWave) c += act_s[r] ? (region_ptr[r + 1] - region_ptr[r]) : 0;
    c = fd::wave_sum(c);
    if (lane == 0) cnt_s[b] = c;
  }
  __syncthreads();
  if (tid == 0) {
    int s = 0;
    cu_q[0] = 0;
    for (int b = 0; b < B; ++b) {
      s += cnt_s[b];
      cu_q[b + 1] = s;
    }
    *m_out = s;
  }

  // 6b. ascending compaction of active token ids: each thread owns a contiguous
  // token range; block-wide exclusive scan of the per-thread counts.
  const int per = (N + kSelThreads - 1) / kSelThreads;
  const int u0 = min(N, tid * per), u1 = min(N, u0 + per);
  int c = 0;
  for (int u = u0; u < u1; ++u) c += act_s[token_region[u]];
  int incl = c;
#pragma unroll
  for (int o = 1; o < fd::kWave; o <<= 1) {
    const int y = __shfl_up(incl, o, fd::kWave);
    if (lane >= o) incl += y;
  }
  if (lane == fd::kWave - 1) wtot_s[wave] = incl;
  __syncthreads();
  int base = 0;
  for (int w = 0; w < wave; ++w) base += wtot_s[w];
  int pos = base + incl - c;
  for (int u = u0; u < u1; ++u)
    if (act_s[token_region[u]]) idx[pos++] = u;
}

// xa[i] = bf16(x[idx[i]]) for i < M.  A workgroup covers kGatherUnroll * 256 consecutive
// float4 elements of the [M][C/4] grid; pass k of its threads covers 256 of them
// (whole rows, coalesced), and every thread issues its kGatherUnroll loads (addresses
// clamped into the grid) before any store, so each wave keeps 4 KB in flight.  SH >= 0:
// C = 4 << SH, so the row of a float4 element is a shift, not a division.
template <int SH>
__global__ __launch_bounds__(256) void gather_kernel(const float* __restrict__ x, const int32_t* __restrict__ idx,
                                                     const int32_t* __restrict__ m_dev, int C_,
                                                     uint16_t* __restrict__ xa) {
  const int C = SH >= 0 ? (4 << SH) : C_;
  const int c4 = C >> 2;
  const int total = (*m_dev) * c4;
  const int first = blockIdx.x * (256 * kGatherUnroll);
  if (first >= total) return;
  float4 v[kGatherUnroll];
#pragma unroll
  for (int k = 0; k < kGatherUnroll; ++k) {
    const int e = min(first + k * 256 + static_cast<int>(threadIdx.x), total - 1);
    const int row = e / c4, col = e - (e / c4) * c4;
    const f32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(x + static_cast<size_t>(idx[row]) * C) + col);
    v[k] = make_float4(t.x, t.y, t.z, t.w);
  }
#pragma unroll
  for (int k = 0; k < kGatherUnroll; ++k) {
    const int e = first + k * 256 + static_cast<int>(threadIdx.x);
    if (e < total) {
      const int row = e / c4, col = e - (e / c4) * c4;
      uint2 o;
      o.x = fd::pack_bf2(v[k].x, v[k].y);
      o.y = fd::pack_bf2(v[k].z, v[k].w);
      // streaming (non-temporal) store: the embedding GEMM reads the rows back once
      __builtin_nontemporal_store(__builtin_bit_cast(uint64_t, o),
                                  reinterpret_cast<uint64_t*>(xa + static_cast<size_t>(row) * C) + col);
    }
  }
}

// streaming (non-temporal) 16-byte load of data read once in the step
FD_DEVICE float4 ldnt4(const f32x4_t* p) {
  const f32x4_t t = __builtin_nontemporal_load(p);
  return make_float4(t.x, t.y, t.z, t.w);
}

FD_DEVICE float4 euler4(float4 x, float h, float4 f) {
  // x + fl32(h * f): two separately rounded fp32 operations (no contraction)
#pragma clang fp contract(off)
  const float px = h * f.x, py = h * f.y, pz = h * f.z, pw = h * f.w;
  return make_float4(x.x + px, x.y + py, x.z + pz, x.w + pw);
}

// Active rows: x[u] = x[u] + fl32(h_b * v[i]); vcache[u] = v[i], u = idx[i].  Same
// decomposition as the gather (kUpdateUnroll * 256 elements per workgroup, every
// load of a thread issued before its stores); both rows are read with streaming
// loads (measured 61 -> 65% of HBM peak at 256 requests), as are the gather's
// (66 -> 68%).  SH as for the gather.
template <int SH>
__global__ __launch_bounds__(256) void update_active_kernel(float* __restrict__ x, const float* __restrict__ v,
                                                            const int32_t* __restrict__ idx,
                                                            const int32_t* __restrict__ m_dev,
                                                            const int32_t* __restrict__ token_region,
                                                            const int32_t* __restrict__ region_req,
                                                            const float* __restrict__ dt, int n_req,
                                                            float* __restrict__ vcache, int C_) {
  const int C = SH >= 0 ? (4 << SH) : C_;
  const int c4 = C >> 2;
  const int total = (*m_dev) * c4;
  const int first = blockIdx.x * (256 * kUpdateUnroll);
  if (first >= total) return;
  // the rows of one workgroup almost always belong to one request: then h is
  // looked up once (uniform loads), else per row
  const int last = min(first + 256 * kUpdateUnroll, total) - 1;
  int b_lo = 0, b_hi = 0;
  if (n_req > 1) {
    b_lo = region_req[token_region[idx[first / c4]]];
    b_hi = region_req[token_region[idx[last / c4]]];
  }
  const float h_tile = dt[b_lo];
  int u[kUpdateUnroll];
  float h[kUpdateUnroll];
  float4 f[kUpdateUnroll], xv[kUpdateUnroll];
#pragma unroll
  for (int k = 0; k < kUpdateUnroll; ++k) {
    const int e = min(first + k * 256 + static_cast<int>(threadIdx.x), total - 1);
    u[k] = idx[e / c4];
  }
#pragma unroll
  for (int k = 0; k < kUpdateUnroll; ++k) {
    const int e = min(first + k * 256 + static_cast<int>(threadIdx.x), total - 1);
    const int row = e / c4, col = e - (e / c4) * c4;
    f[k] = ldnt4(reinterpret_cast<const f32x4_t*>(v + static_cast<size_t>(row) * C) + col);
    xv[k] = ldnt4(reinterpret_cast<const f32x4_t*>(x + static_cast<size_t>(u[k]) * C) + col);
    h[k] = b_lo == b_hi ? h_tile : dt[region_req[token_region[u[k]]]];
  }
#pragma unroll
  for (int k = 0; k < kUpdateUnroll; ++k) {
    const int e = first + k * 256 + static_cast<int>(threadIdx.x);
    if (e < total) {
      const int col = e - (e / c4) * c4;
      // streaming (non-temporal) stores: neither row is read again within the step
      __builtin_nontemporal_store(__builtin_bit_cast(f32x4_t, euler4(xv[k], h[k], f[k])),
                                  reinterpret_cast<f32x4_t*>(x + static_cast<size_t>(u[k]) * C) + col);
      __builtin_nontemporal_store(__builtin_bit_cast(f32x4_t, f[k]),
                                  reinterpret_cast<f32x4_t*>(vcache + static_cast<size_t>(u[k]) * C) + col);
    }
  }
}

// Skipped rows under the cached-drift rule: x[u] = x[u] + fl32(h_b * vcache[u]).
__global__ __launch_bounds__(256) void update_skipped_kernel(float* __restrict__ x, const float* __restrict__ vcache,
                                                             const uint8_t* __restrict__ active,
                                                             const int32_t* __restrict__ token_region,
                                                             const int32_t* __restrict__ region_req,
                                                             const float* __restrict__ dt, int N, int C) {
  const int c4 = C >> 2;
  const int total = N * c4;
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < total; e += gridDim.x * blockDim.x) {
    const int u = e / c4, col = e - (e / c4) * c4;
    const int r = token_region[u];
    if (active[r]) continue;
    const float h = dt[region_req[r]];
    const float4 f = reinterpret_cast<const float4*>(vcache + static_cast<size_t>(u) * C)[col];
    float4* xr = reinterpret_cast<float4*>(x + static_cast<size_t>(u) * C) + col;
    *xr = euler4(*xr, h, f);
  }
}

int stream_grid(long long elems) {
  const long long g = (elems + 255) / 256;
  const long long cap = 8LL * fdh::num_cus();
  return static_cast<int>(g < 1 ? 1 : (g > cap ? cap : g));
}

// `unroll` elements per thread, grid sized for M = N
int unrolled_grid(long long elems, int unroll) {
  const long long per = 256LL * unroll;
  return static_cast<int>(elems < 1 ? 1 : (elems + per - 1) / per);
}

}  // namespace

namespace fdh {

hipError_t launch_region_score(const fd_plan* p, int C, const float* xc, const float* xp, double* score,
                               double* partial, int nchunk, int rows_per_chunk, hipStream_t s) {
  dim3 grid(nchunk, p->n_regions);
  region_score_partial_kernel<<<grid, kScoreThreads, 0, s>>>(p->region_ptr, p->region_tokens, xc, xp, C,
                                                             rows_per_chunk, partial, score);
  if (nchunk > 1)
    region_score_finalize_kernel<<<(p->n_regions + 255) / 256, 256, 0, s>>>(p->region_ptr, partial, nchunk,
                                                                            p->n_regions, C, score);
  return hipGetLastError();
}

hipError_t launch_select(const fd_plan* p, const double* score, const double* eps, fd_gate g, double* s_tilde,
                         int32_t* skip_run, const uint8_t* prev_active, uint8_t* active, int32_t* idx,
                         int32_t* cu_q, int32_t* m, hipStream_t s) {
  gate_select_kernel<<<1, kSelThreads, 0, s>>>(p->n_regions, p->n_requests, p->n_tokens, p->region_req,
                                               p->req_reg_off, p->region_ptr, p->token_region, score, eps, g.eta,
                                               g.max_skip, s_tilde, skip_run, prev_active, active, idx, cu_q, m);
  return hipGetLastError();
}

hipError_t launch_gather(const fd_plan* p, int C, const float* x, const int32_t* idx, const int32_t* m,
                         uint16_t* xa, hipStream_t s) {
  const int grid = unrolled_grid(static_cast<long long>(p->n_tokens) * (C / 4), kGatherUnroll);
  if (C == 64)   // the paper's workloads: 16 channels x 2 x 2 patches
    gather_kernel<4><<<grid, 256, 0, s>>>(x, idx, m, C, xa);
  else
    gather_kernel<-1><<<grid, 256, 0, s>>>(x, idx, m, C, xa);
  return hipGetLastError();
}

hipError_t launch_scatter_update(const fd_plan* p, int C, float* x, const float* v, const int32_t* idx,
                                 const int32_t* m, const float* dt, float* vcache, const uint8_t* active,
                                 int skip_mode, hipStream_t s) {
  const long long el = static_cast<long long>(p->n_tokens) * (C / 4);
  if (skip_mode == FD_SKIP_REUSE_DRIFT)
    update_skipped_kernel<<<stream_grid(el), 256, 0, s>>>(x, vcache, active, p->token_region, p->region_req, dt,
                                                         p->n_tokens, C);
  if (C == 64)
    update_active_kernel<4><<<unrolled_grid(el, kUpdateUnroll), 256, 0, s>>>(x, v, idx, m, p->token_region, p->region_req,
                                                                           dt, p->n_requests, vcache, C);
  else
    update_active_kernel<-1><<<unrolled_grid(el, kUpdateUnroll), 256, 0, s>>>(x, v, idx, m, p->token_region, p->region_req,
                                                                            dt, p->n_requests, vcache, C);
  return hipGetLastError();
}

}  // namespace fdh
