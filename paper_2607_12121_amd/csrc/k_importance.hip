// Refinement importance of the active regions (the Patch Gate's own signal):
// R_i = |A_i|^-2 sum_{u,v in A_i} SA_uv with SA one block's self-attention
// averaged over its heads, recomputed for the pairs inside each active region
// from that block's queries, key cache and per-query softmax normalisers (base-2
// log-sum-exp of the scaled scores, written by the attention kernel); then
// Delta_i = |R_i - Rbar_i| and Rbar_i = R_i.  The full attention matrix is never
// formed: only |A_i|^2 scores per region and head.
#include "fd_common.h"

namespace {

constexpr int kImpThreads = 256;
constexpr int kImpWaves = kImpThreads / fd::kWave;

// pos[idx[i]] = i for i < M: the active row of every active token.
__global__ __launch_bounds__(256) void row_of_token_kernel(const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ m_dev,
                                                           int32_t* __restrict__ pos) {
  const int M = *m_dev;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < M; i += gridDim.x * blockDim.x) pos[idx[i]] = i;
}

// part[r][h] = sum_{u in A_r} sum_{v in A_r} exp2(scale_log2 * q_u,h . k_v,h - lse_u,h)
// for active regions r; one workgroup per (region, head).  The region's key rows
// of the head sit in LDS; lane l of every wave owns query row i0 + l (its q in
// registers) and wave w the keys of its quarter of the region, so all lanes of a
// wave read the same key element (an LDS broadcast).  bf16 products are summed
// in fp32 (v_dot2_f32_bf16); the workgroup sum runs in a fixed order.
template <int DH>
__global__ __launch_bounds__(kImpThreads) void importance_partial_kernel(
    const int32_t* __restrict__ region_ptr, const int32_t* __restrict__ region_tokens,
    const uint8_t* __restrict__ active, const int32_t* __restrict__ pos, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ kc, const float* __restrict__ lse, int D, int H, float scale_log2,
    float* __restrict__ part) {
  constexpr int W = DH / 2;   // bf16 pairs per row
  extern __shared__ uint32_t sk[];   // [n][W]
  __shared__ float wsum[kImpWaves];
  const int r = blockIdx.x, h = blockIdx.y;
  if (!active[r]) return;   // whole workgroup
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int t0 = region_ptr[r], n = region_ptr[r + 1] - t0;
  for (int e = threadIdx.x; e < n * W; e += kImpThreads) {
    const int j = e / W, c = e - (e / W) * W;
    sk[e] = reinterpret_cast<const uint32_t*>(kc + static_cast<size_t>(region_tokens[t0 + j]) * D + h * DH)[c];
  }
  __syncthreads();
  const int j0 = (wave * n) / kImpWaves, j1 = ((wave + 1) * n) / kImpWaves;
  float acc = 0.f;
  for (int i0 = 0; i0 < n; i0 += fd::kWave) {
    const int i = i0 + lane;
    if (i < n) {
      const int row = pos[region_tokens[t0 + i]];
      const uint32_t* qr = reinterpret_cast<const uint32_t*>(q + static_cast<size_t>(row) * D + h * DH);
      uint32_t qv[W];
#pragma unroll
      for (int c = 0; c < W; ++c) qv[c] = qr[c];
      const float li = lse[static_cast<size_t>(row) * H + h];
      for (int j = j0; j < j1; ++j) {
        const uint32_t* kr = sk + j * W;
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < W; ++c)
          s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(fd::bf16x2_t, qv[c]),
                                              __builtin_bit_cast(fd::bf16x2_t, kr[c]), s, false);
        acc += __builtin_amdgcn_exp2f(s * scale_log2 - li);
      }
    }
  }
  acc = fd::wave_sum(acc);
  if (lane == 0) wsum[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
    for (int w = 0; w < kImpWaves; ++w) t += wsum[w];
    part[static_cast<size_t>(r) * H + h] = t;
  }
}

// Active regions: R = (sum_h part[r][h]) / (H |A_r|^2), Delta = |R - Rbar|, Rbar = R;
// skipped regions keep both.  importance[r] = R (NaN for skipped ones) when given.
__global__ __launch_bounds__(256) void importance_update_kernel(const int32_t* __restrict__ region_ptr,
                                                                const uint8_t* __restrict__ active,
                                                                const float* __restrict__ part, int R, int H,
                                                                double* __restrict__ r_bar,
                                                                double* __restrict__ delta,
                                                                double* __restrict__ importance) {
  for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < R; r += gridDim.x * blockDim.x) {
    if (active[r]) {
      double sum = 0.0;
      for (int h = 0; h < H; ++h) sum += static_cast<double>(part[static_cast<size_t>(r) * H + h]);
      const double n = static_cast<double>(region_ptr[r + 1] - region_ptr[r]);
      const double imp = sum / (static_cast<double>(H) * n * n);
      delta[r] = fabs(imp - r_bar[r]);
      r_bar[r] = imp;
      if (importance) importance[r] = imp;
    } else if (importance) {
      importance[r] = __builtin_nan("");
    }
  }
}

}  // namespace

namespace fdh {

size_t importance_lds_bytes(int dh, int max_region_tokens) {
  return static_cast<size_t>(max_region_tokens) * (dh / 2) * sizeof(uint32_t);
}

hipError_t launch_importance(const fd_plan* p, int D, int H, int dh, const int32_t* idx, const int32_t* m,
                             const uint8_t* active, const uint16_t* q, const uint16_t* kc, const float* lse,
                             int32_t* pos, float* part, double* r_bar, double* delta, double* importance,
                             hipStream_t s) {
  const int rows_grid = (p->n_tokens + 255) / 256;
  row_of_token_kernel<<<rows_grid < 1024 ? rows_grid : 1024, 256, 0, s>>>(idx, m, pos);
  const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(dh));
  const size_t lds = importance_lds_bytes(dh, p->max_region_tokens);
  const dim3 grid(p->n_regions, H);
  switch (dh) {
    case 16:
      importance_partial_kernel<16><<<grid, kImpThreads, lds, s>>>(p->region_ptr, p->region_tokens, active, pos, q,
                                                                   kc, lse, D, H, scale_log2, part);
      break;
    case 64:
      importance_partial_kernel<64><<<grid, kImpThreads, lds, s>>>(p->region_ptr, p->region_tokens, active, pos, q,
                                                                   kc, lse, D, H, scale_log2, part);
      break;
    case 128:
      importance_partial_kernel<128><<<grid, kImpThreads, lds, s>>>(p->region_ptr, p->region_tokens, active, pos, q,
                                                                    kc, lse, D, H, scale_log2, part);
      break;
    default:
      return hipErrorInvalidValue;
  }
  const int ugrid = (p->n_regions + 255) / 256;
  importance_update_kernel<<<ugrid, 256, 0, s>>>(p->region_ptr, active, part, p->n_regions, H, r_bar, delta,
                                                 importance);
  return hipGetLastError();
}

}  // namespace fdh
