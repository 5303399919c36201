// adaLN modulation GEMV and LayerNorm + modulate of the active rows.
#include "fd_common.h"

namespace {

constexpr int kAdaThreads = 256;
constexpr int kAdaRowsPerWave = 4;
constexpr int kAdaRowsPerBlock = kAdaRowsPerWave * (kAdaThreads / fd::kWave);
constexpr int kAdaMaxB = 8;             // requests handled per pass over a weight row
constexpr int kAdaLdsFloats = 12288;    // 48 KB of SiLU(cond)

// mod[b][j] = sum_k W[j][k] * SiLU(cond[b][k]) + bias[j]   (W bf16 [n_out][D]).
// Each wave owns 4 output rows; lanes stream 16-byte pieces of those rows and
// dot them with SiLU(cond) staged in LDS for up to 8 requests at a time.
__global__ __launch_bounds__(kAdaThreads) void adaln_gemv_kernel(const uint16_t* __restrict__ W,
                                                                 const float* __restrict__ bias,
                                                                 const float* __restrict__ cond, int B, int D,
                                                                 int n_out, int b_chunk, float* __restrict__ mod,
                                                                 int32_t* __restrict__ zero_ints, int n_zero) {
  __shared__ float sc[kAdaLdsFloats];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // The block's first kernel also clears the GEMM split-K arrival counters.
  if (blockIdx.x == 0 && zero_ints)
    for (int i = threadIdx.x; i < n_zero; i += kAdaThreads) zero_ints[i] = 0;
  const int row0 = blockIdx.x * kAdaRowsPerBlock + wave * kAdaRowsPerWave;
  for (int b0 = 0; b0 < B; b0 += b_chunk) {
    const int nb = min(b_chunk, B - b0);
    __syncthreads();
    for (int e = threadIdx.x; e < nb * D; e += kAdaThreads) {
      const float z = cond[static_cast<size_t>(b0) * D + e];
      sc[e] = z / (1.0f + __expf(-z));
    }
    __syncthreads();
    float acc[kAdaRowsPerWave][kAdaMaxB];
#pragma unroll
    for (int i = 0; i < kAdaRowsPerWave; ++i)
#pragma unroll
      for (int b = 0; b < kAdaMaxB; ++b) acc[i][b] = 0.f;
    for (int k = lane * 8; k < D; k += fd::kWave * 8) {
      float s8[kAdaMaxB][8];
#pragma unroll
      for (int b = 0; b < kAdaMaxB; ++b) {
        if (b < nb) {
          const float4 lo = *reinterpret_cast<const float4*>(&sc[b * D + k]);
          const float4 hi = *reinterpret_cast<const float4*>(&sc[b * D + k + 4]);
          s8[b][0] = lo.x; s8[b][1] = lo.y; s8[b][2] = lo.z; s8[b][3] = lo.w;
          s8[b][4] = hi.x; s8[b][5] = hi.y; s8[b][6] = hi.z; s8[b][7] = hi.w;
        }
      }
#pragma unroll
      for (int i = 0; i < kAdaRowsPerWave; ++i) {
        const int j = row0 + i;
        if (j >= n_out) break;
        const uint4 wv = *reinterpret_cast<const uint4*>(W + static_cast<size_t>(j) * D + k);
        const uint32_t wr[4] = {wv.x, wv.y, wv.z, wv.w};
        float wf[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          wf[2 * q] = __uint_as_float(wr[q] << 16);
          wf[2 * q + 1] = __uint_as_float(wr[q] & 0xffff0000u);
        }
#pragma unroll
        for (int b = 0; b < kAdaMaxB; ++b) {
          if (b < nb) {
            float a = acc[i][b];
#pragma unroll
            for (int q = 0; q < 8; ++q) a += wf[q] * s8[b][q];
            acc[i][b] = a;
          }
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kAdaRowsPerWave; ++i) {
      const int j = row0 + i;
#pragma unroll
      for (int b = 0; b < kAdaMaxB; ++b) {
        if (b < nb) {
          const float s = fd::wave_sum(acc[i][b]);
          if (lane == 0 && j < n_out) mod[static_cast<size_t>(b0 + b) * n_out + j] = s + bias[j];
        }
      }
    }
  }
}

// a[i] = bf16(LN(h[i]) * (1 + scale_b) + shift_b) for i < M; one wave per row.
// VEC: float4 pieces per lane (D = 256 * VEC); VEC = 0 selects the scalar path
// for D not a multiple of 256 (lanes take every 64th element).
template <int VEC>
__global__ __launch_bounds__(256) void ln_modulate_kernel(const float* __restrict__ h,
                                                          const int32_t* __restrict__ cu_q, int B,
                                                          const int32_t* __restrict__ m_dev, int D,
                                                          const float* __restrict__ mod, int mod_stride,
                                                          int shift_off, int scale_off, uint16_t* __restrict__ a) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= *m_dev) return;
  const int b = fd::row_request(cu_q, B, row);
  const float* hr = h + static_cast<size_t>(row) * D;
  const float* shift = mod + static_cast<size_t>(b) * mod_stride + shift_off;
  const float* scale = mod + static_cast<size_t>(b) * mod_stride + scale_off;
  uint16_t* ar = a + static_cast<size_t>(row) * D;
  const float inv_d = 1.0f / static_cast<float>(D);
  if constexpr (VEC > 0) {
    float4 v[VEC];
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      v[j] = reinterpret_cast<const float4*>(hr)[lane + 64 * j];
      s += (v[j].x + v[j].y) + (v[j].z + v[j].w);
    }
    const float mean = fd::wave_sum(s) * inv_d;
    float q = 0.f;
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      const float d0 = v[j].x - mean, d1 = v[j].y - mean, d2 = v[j].z - mean, d3 = v[j].w - mean;
      q += (d0 * d0 + d1 * d1) + (d2 * d2 + d3 * d3);
    }
    const float rstd = 1.0f / sqrtf(fd::wave_sum(q) * inv_d + 1e-6f);
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      const int k = 4 * (lane + 64 * j);
      const float4 sh = *reinterpret_cast<const float4*>(shift + k);
      const float4 sc = *reinterpret_cast<const float4*>(scale + k);
      uint2 o;
      o.x = fd::pack_bf2((v[j].x - mean) * rstd * (1.f + sc.x) + sh.x, (v[j].y - mean) * rstd * (1.f + sc.y) + sh.y);
      o.y = fd::pack_bf2((v[j].z - mean) * rstd * (1.f + sc.z) + sh.z, (v[j].w - mean) * rstd * (1.f + sc.w) + sh.w);
      reinterpret_cast<uint2*>(ar)[lane + 64 * j] = o;
    }
  } else {
    float s = 0.f;
    for (int k = lane; k < D; k += 64) s += hr[k];
    const float mean = fd::wave_sum(s) * inv_d;
    float q = 0.f;
    for (int k = lane; k < D; k += 64) {
      const float d = hr[k] - mean;
      q += d * d;
    }
    const float rstd = 1.0f / sqrtf(fd::wave_sum(q) * inv_d + 1e-6f);
    for (int k = lane; k < D; k += 64) ar[k] = fd::f2bf((hr[k] - mean) * rstd * (1.f + scale[k]) + shift[k]);
  }
}

}  // namespace

namespace fdh {

hipError_t launch_adaln(const uint16_t* w, const float* b, const float* cond, int B, int D, int n_out, float* mod,
                        int32_t* zero_ints, int n_zero, hipStream_t s) {
  int b_chunk = kAdaLdsFloats / D;
  if (b_chunk > kAdaMaxB) b_chunk = kAdaMaxB;
  const int grid = (n_out + kAdaRowsPerBlock - 1) / kAdaRowsPerBlock;
  adaln_gemv_kernel<<<grid, kAdaThreads, 0, s>>>(w, b, cond, B, D, n_out, b_chunk, mod, zero_ints, n_zero);
  return hipGetLastError();
}

hipError_t launch_ln_modulate(const float* h, const int32_t* cu_q, int B, const int32_t* m, int n_max, int D,
                              const float* mod, int mod_stride, int shift_off, int scale_off, uint16_t* a,
                              hipStream_t s) {
  const int grid = (n_max + 3) / 4;
  switch (D % 256 == 0 ? D / 256 : 0) {
#define FD_LN_CASE(V)                                                                                   \
  case V:                                                                                               \
    ln_modulate_kernel<V><<<grid, 256, 0, s>>>(h, cu_q, B, m, D, mod, mod_stride, shift_off, scale_off, a); \
    break;
    FD_LN_CASE(1) FD_LN_CASE(2) FD_LN_CASE(3) FD_LN_CASE(4) FD_LN_CASE(5) FD_LN_CASE(6) FD_LN_CASE(8)
    FD_LN_CASE(12) FD_LN_CASE(16)
#undef FD_LN_CASE
    default:
      ln_modulate_kernel<0><<<grid, 256, 0, s>>>(h, cu_q, B, m, D, mod, mod_stride, shift_off, scale_off, a);
  }
  return hipGetLastError();
}

}  // namespace fdh
