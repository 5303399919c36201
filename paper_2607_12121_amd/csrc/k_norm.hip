// adaLN modulation GEMV and LayerNorm + modulate of the active rows.
#include "fd_common.h"

namespace {

constexpr int kAdaThreads = 256;
constexpr int kAdaWaves = kAdaThreads / fd::kWave;
constexpr int kAdaLdsFloats = 12288;    // at most 48 KB of SiLU(cond) per pass
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
constexpr int kAdaRows = 4;   // weight rows per wave and group (2: 6.2 us per block, 4: 5.4)

FD_DEVICE void bf16x8_to_f32(const uint4 w, float f[8]) {
  const uint32_t r[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    f[2 * q] = __uint_as_float(r[q] << 16);
    f[2 * q + 1] = __uint_as_float(r[q] & 0xffff0000u);
  }
}

// SiLU(cond) of requests b0 .. b0 + NB - 1 (zero past B) into sc[NB][D].
template <int NB>
FD_DEVICE void silu_cond_to_lds(const float* __restrict__ cond, int B, int D, int b0, float* sc) {
  __syncthreads();
  for (int e = threadIdx.x; e < NB * D; e += kAdaThreads) {
    const float z = b0 + e / D < B ? cond[static_cast<size_t>(b0) * D + e] : 0.f;
    sc[e] = z / (1.0f + __expf(-z));
  }
  __syncthreads();
}

// acc[i][b] += dot(W row i (8 bf16 at k, packed in wv[i]), SiLU(cond_b)[k .. k + 7]).
template <int NB, int R>
FD_DEVICE void ada_fma_chunk(const float* sc, int D, int k, const uint4 (&wv)[R], float (&acc)[R][NB]) {
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const float4 lo = *reinterpret_cast<const float4*>(&sc[b * D + k]);
    const float4 hi = *reinterpret_cast<const float4*>(&sc[b * D + k + 4]);
    const float s8[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
    for (int i = 0; i < R; ++i) {
      float wf[8];
      bf16x8_to_f32(wv[i], wf);
      float a = acc[i][b];
#pragma unroll
      for (int q = 0; q < 8; ++q) a += wf[q] * s8[q];
      acc[i][b] = a;
    }
  }
}

// Row j of the stacked weights (block l = j / n_out, output jj): one value per request.
template <int NB, int R>
FD_DEVICE void ada_store(const float (&acc)[R][NB], int row0, int n_rows, int n_out, int B, int b0,
                         const float* __restrict__ bias, float* __restrict__ mod) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int j = row0 + i;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const float s = fd::wave_sum(acc[i][b]);
      if (lane == 0 && j < n_rows && b0 + b < B) {
        const int l = j / n_out, jj = j - l * n_out;
        mod[(static_cast<size_t>(l) * B + b0 + b) * n_out + jj] = s + bias[j];
      }
    }
  }
}

// mod[l][b][j] = sum_k W[l][j][k] * SiLU(cond[b][k]) + bias[l][j] for n_blocks
// stacked weight matrices (W bf16 [n_blocks][n_out][D], rows contiguous across
// blocks): a stream of n_blocks * n_out weight rows, HBM-bound.  D = 512 KIT: each
// wave walks groups of kAdaRows consecutive rows (grid-stride), a lane holding 8
// consecutive k of every 512; two register buffers keep the next group's loads in
// flight while the current group is reduced.  SiLU(cond) of NB <= 2 requests sits
// in LDS; B > NB re-streams the weights per NB requests.
template <int NB, int KIT>
__global__ __launch_bounds__(kAdaThreads) void adaln_stream_kernel(const uint16_t* __restrict__ W,
                                                                   const float* __restrict__ bias,
                                                                   const float* __restrict__ cond, int B, int D,
                                                                   int n_out, int n_rows, float* __restrict__ mod) {
  constexpr int R = kAdaRows;
  extern __shared__ float sc[];   // [NB][D]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n_groups = (n_rows + R - 1) / R;
  const int stride = gridDim.x * kAdaWaves;
  auto load = [&](int grp, uint4 (&w)[KIT][R]) {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const uint16_t* r = W + static_cast<size_t>(min(grp * R + i, n_rows - 1)) * D + lane * 8;   // past the end: the last row again
#pragma unroll
      for (int t = 0; t < KIT; ++t) {
        // streaming loads: each weight row is read once per step (7.0 -> 6.1 us per block)
        const u32x4_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(r + t * 512));
        w[t][i] = make_uint4(x.x, x.y, x.z, x.w);
      }
    }
  };
  auto reduce = [&](int grp, const uint4 (&w)[KIT][R], int b0) {
    float acc[R][NB];
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[i][b] = 0.f;
#pragma unroll
    for (int t = 0; t < KIT; ++t) ada_fma_chunk<NB, R>(sc, D, t * 512 + lane * 8, w[t], acc);
    ada_store<NB, R>(acc, grp * R, n_rows, n_out, B, b0, bias, mod);
  };
  for (int b0 = 0; b0 < B; b0 += NB) {
    silu_cond_to_lds<NB>(cond, B, D, b0, sc);
    int grp = blockIdx.x * kAdaWaves + wave;
    if (grp >= n_groups) continue;
    uint4 w0[KIT][R], w1[KIT][R];
    load(grp, w0);
    for (;;) {
      const bool more0 = grp + stride < n_groups;
      if (more0) load(grp + stride, w1);
      reduce(grp, w0, b0);
      if (!more0) break;
      grp += stride;
      const bool more1 = grp + stride < n_groups;
      if (more1) load(grp + stride, w0);
      reduce(grp, w1, b0);
      if (!more1) break;
      grp += stride;
    }
  }
}

// The same product for any D (and for more than two requests per pass, where the
// streaming kernel's registers would grow past two waves per SIMD): one group of 4
// rows per wave, one k-chunk of all 4 rows at a time; blockIdx.y picks the batch
// of NB requests, so the batches of a many-request call run side by side (their
// re-reads of the same weight rows are served by L2).
constexpr int kAdaRowsPerWave = 4;
constexpr int kAdaRowsPerBlock = kAdaRowsPerWave * kAdaWaves;
template <int NB>
__global__ __launch_bounds__(kAdaThreads) void adaln_gemv_kernel(const uint16_t* __restrict__ W,
                                                                 const float* __restrict__ bias,
                                                                 const float* __restrict__ cond, int B, int D,
                                                                 int n_out, int n_rows, float* __restrict__ mod) {
  extern __shared__ float sc[];   // [NB][D]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int b0 = blockIdx.y * NB;   // < B by the grid
  silu_cond_to_lds<NB>(cond, B, D, b0, sc);
  const int n_groups = (n_rows + kAdaRowsPerBlock - 1) / kAdaRowsPerBlock;
  for (int grp = blockIdx.x; grp < n_groups; grp += gridDim.x) {   // row groups of this batch
    const int row0 = grp * kAdaRowsPerBlock + wave * kAdaRowsPerWave;
    const uint16_t* wr[kAdaRowsPerWave];
#pragma unroll
    for (int i = 0; i < kAdaRowsPerWave; ++i)
      wr[i] = W + static_cast<size_t>(min(row0 + i, n_rows - 1)) * D;   // rows past the end re-read the last
    float acc[kAdaRowsPerWave][NB];
#pragma unroll
    for (int i = 0; i < kAdaRowsPerWave; ++i)
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[i][b] = 0.f;
    for (int k = lane * 8; k < D; k += 512) {
      uint4 wv[kAdaRowsPerWave];
#pragma unroll
      for (int i = 0; i < kAdaRowsPerWave; ++i) wv[i] = *reinterpret_cast<const uint4*>(wr[i] + k);
      ada_fma_chunk<NB, kAdaRowsPerWave>(sc, D, k, wv, acc);
    }
    ada_store<NB, kAdaRowsPerWave>(acc, row0, n_rows, n_out, B, b0, bias, mod);
  }
}

// More than 24 requests: the same product on the matrix cores in fp32
// (v_mfma_f32_16x16x4f32; the bf16 weights widen exactly, so the precision is
// that of the fp32 GEMV), 16 requests per workgroup with their SiLU(cond) in LDS
// (D <= 2048), each wave 32 weight rows (two 16-row blocks), the workgroup
// walking row tiles of its request batch.  k is permuted so that a lane reads 8
// consecutive weights of its row: in MFMA step t of a 32-wide k chunk, lane group
// g (lanes 16g .. 16g + 15) supplies k = 8g + t, to both operands.  Weights are
// loaded four chunks ahead.  The grid's x extent is a multiple of the 8 XCDs, so
// all request batches of a row tile run on one XCD and share its weights in L2.
constexpr int kAdaMfmaReq = 16;
// Above this many requests the matrix-core kernel beats the GEMV (hidden 1024:
// 12 requests 68 against 50 us, 24 equal at 74, 32 75 against 80, 64 79 against
// 115); below it a few request batches leave most of the GPU idle.
constexpr int kAdaMfmaMinB = 24;
constexpr int kAdaMfmaMaxD = 2048;
constexpr int kAdaMfmaWaves = 8;
constexpr int kAdaMfmaBlk = 2;                                   // 16-row blocks per wave
constexpr int kAdaMfmaTile = kAdaMfmaWaves * 16 * kAdaMfmaBlk;   // rows per workgroup tile
constexpr int kAdaMfmaPf = 4;                                    // 32-wide k chunks of weights in flight
typedef float f32x4v_t __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(kAdaMfmaWaves * 64) void adaln_mfma_kernel(const uint16_t* __restrict__ W,
                                                                       const float* __restrict__ bias,
                                                                       const float* __restrict__ cond, int B, int D,
                                                                       int n_out, int n_rows, float* __restrict__ mod) {
  __shared__ float sc[kAdaMfmaReq * kAdaMfmaMaxD];   // SiLU(cond) [16][D]
  const int n_tiles = (n_rows + kAdaMfmaTile - 1) / kAdaMfmaTile;
  if (static_cast<int>(blockIdx.x) >= n_tiles) return;   // grid padded to whole XCD rounds
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b0 = blockIdx.y * kAdaMfmaReq;   // < B by the grid
  for (int e = tid; e < kAdaMfmaReq * D; e += kAdaMfmaWaves * 64) {
    const float z = b0 + e / D < B ? cond[static_cast<size_t>(b0) * D + e] : 0.f;
    sc[e] = z / (1.0f + __expf(-z));
  }
  __syncthreads();
  const int i16 = lane & 15, g = lane >> 4;
  const float* srow = sc + i16 * D + 8 * g;   // request b0 + i16, this lane group's k
  for (int tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    const int r0 = tile * kAdaMfmaTile + wave * 16 * kAdaMfmaBlk;
    const uint16_t* wr[kAdaMfmaBlk];
    f32x4v_t acc[kAdaMfmaBlk];
    uint4 wq[kAdaMfmaPf][kAdaMfmaBlk];   // chunks k0 + 32 u, u < kAdaMfmaPf, in flight
#pragma unroll
    for (int blk = 0; blk < kAdaMfmaBlk; ++blk) {
      wr[blk] = W + static_cast<size_t>(min(r0 + 16 * blk + i16, n_rows - 1)) * D + 8 * g;
      acc[blk] = f32x4v_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < kAdaMfmaPf; ++u) wq[u][blk] = *reinterpret_cast<const uint4*>(wr[blk] + 32 * u);
    }
    for (int k0 = 0; k0 < D; k0 += 32 * kAdaMfmaPf) {   // D is a multiple of 32 kAdaMfmaPf
#pragma unroll
      for (int u = 0; u < kAdaMfmaPf; ++u) {
        const int k = k0 + 32 * u;
        const float4 s0 = *reinterpret_cast<const float4*>(srow + k);
        const float4 s1 = *reinterpret_cast<const float4*>(srow + k + 4);
        const float s8[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
        float wf[kAdaMfmaBlk][8];
#pragma unroll
        for (int blk = 0; blk < kAdaMfmaBlk; ++blk) bf16x8_to_f32(wq[u][blk], wf[blk]);
        // refill this slot with the chunk kAdaMfmaPf ahead
        if (k + 32 * kAdaMfmaPf < D) {
#pragma unroll
          for (int blk = 0; blk < kAdaMfmaBlk; ++blk)
            wq[u][blk] = *reinterpret_cast<const uint4*>(wr[blk] + k + 32 * kAdaMfmaPf);
        }
#pragma unroll
        for (int t = 0; t < 8; ++t)
#pragma unroll
          for (int blk = 0; blk < kAdaMfmaBlk; ++blk)
            acc[blk] = __builtin_amdgcn_mfma_f32_16x16x4f32(wf[blk][t], s8[t], acc[blk], 0, 0, 0);
      }
    }
    // lane (i16, g), register r: weight row 16 blk + 4 g + r of the wave, request b0 + i16
    const int b = b0 + i16;
#pragma unroll
    for (int blk = 0; blk < kAdaMfmaBlk; ++blk)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = r0 + 16 * blk + 4 * g + r;
        if (row < n_rows && b < B) {
          const int l = row / n_out, jj = row - l * n_out;
          mod[(static_cast<size_t>(l) * B + b) * n_out + jj] = acc[blk][r] + bias[row];
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
                                                          int shift_off, int scale_off, uint16_t* __restrict__ a,
                                                          const int32_t* __restrict__ idx,
                                                          const int32_t* __restrict__ token_region,
                                                          const int32_t* __restrict__ region_req) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= *m_dev) return;
  // the row's request: through its token's region when the index list is given
  // (two table reads after idx, whatever B), else a binary search over cu_q
  const int b = B == 1 ? 0 : idx ? region_req[token_region[idx[row]]] : fd::row_request(cu_q, B, row);
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

hipError_t launch_adaln(const uint16_t* w, const float* b, const float* cond, int B, int D, int n_out, int n_blocks,
                        float* mod, hipStream_t s) {
  const int n_rows = n_out * n_blocks;
  // requests per pass: B rounded up to a power of two, at most 8 and at most what LDS holds
  const int cap = kAdaLdsFloats / D;   // >= 1 (D <= 12288)
  int nb = B <= 1 ? 1 : B <= 2 ? 2 : B <= 4 ? 4 : 8;
  while (nb > 1 && nb > cap) nb >>= 1;
  const int kit = (D % 512 == 0 && D <= 2048) ? D / 512 : 0;
  if (kit > 0 && nb <= 2) {
    // persistent: four workgroups per CU, fewer when the rows run out first
    const int groups = (n_rows + kAdaRows - 1) / kAdaRows;
    int grid = 4 * num_cus();
    if (grid > (groups + kAdaWaves - 1) / kAdaWaves) grid = (groups + kAdaWaves - 1) / kAdaWaves;
#define FD_ADA(NB, KIT)                                                                                     \
  adaln_stream_kernel<NB, KIT><<<grid, kAdaThreads, (NB) * D * sizeof(float), s>>>(w, b, cond, B, D, n_out, \
                                                                                 n_rows, mod)
#define FD_ADA_NB(NB)             \
  switch (kit) {                  \
    case 1: FD_ADA(NB, 1); break; \
    case 2: FD_ADA(NB, 2); break; \
    case 3: FD_ADA(NB, 3); break; \
    default: FD_ADA(NB, 4);       \
  }
    if (nb == 1) {
      FD_ADA_NB(1)
    } else {
      FD_ADA_NB(2)
    }
#undef FD_ADA_NB
#undef FD_ADA
  } else if (B > kAdaMfmaMinB && D <= kAdaMfmaMaxD && D % (32 * kAdaMfmaPf) == 0) {
    const int batches = (B + kAdaMfmaReq - 1) / kAdaMfmaReq;
    if (batches > 65535) return hipErrorInvalidValue;   // the grid's y extent
    // every row tile its own workgroup column (up to eight per CU in all, then
    // walked), the x extent a multiple of the 8 XCDs
    const int tiles = (n_rows + kAdaMfmaTile - 1) / kAdaMfmaTile;
    int gx = (8 * num_cus() + batches - 1) / batches;
    if (gx > tiles) gx = tiles;
    gx = (gx + 7) / 8 * 8;
    adaln_mfma_kernel<<<dim3(gx, batches), kAdaMfmaWaves * 64, 0, s>>>(w, b, cond, B, D, n_out, n_rows, mod);
  } else {
    const int batches = (B + nb - 1) / nb;
    if (batches > 65535) return hipErrorInvalidValue;   // the grid's y extent
    // about eight workgroups per CU in all; each walks row groups of its batch, so
    // the batch's SiLU(cond) is computed once per workgroup, not once per row group
    const int groups = (n_rows + kAdaRowsPerBlock - 1) / kAdaRowsPerBlock;
    int gx = (8 * num_cus() + batches - 1) / batches;
    if (gx > groups) gx = groups;
    const dim3 grid(gx, batches);
#define FD_ADA(NB) \
  adaln_gemv_kernel<NB><<<grid, kAdaThreads, (NB) * D * sizeof(float), s>>>(w, b, cond, B, D, n_out, n_rows, mod)
    switch (nb) {
      case 1: FD_ADA(1); break;
      case 2: FD_ADA(2); break;
      case 4: FD_ADA(4); break;
      default: FD_ADA(8);
    }
#undef FD_ADA
  }
  return hipGetLastError();
}

hipError_t launch_ln_modulate(const float* h, const int32_t* cu_q, int B, const int32_t* m, int n_max, int D,
                              const float* mod, int mod_stride, int shift_off, int scale_off, uint16_t* a,
                              const int32_t* idx, const int32_t* token_region, const int32_t* region_req,
                              hipStream_t s) {
  const int grid = (n_max + 3) / 4;
  switch (D % 256 == 0 ? D / 256 : 0) {
#define FD_LN_CASE(V)                                                                                   \
  case V:                                                                                               \
    ln_modulate_kernel<V><<<grid, 256, 0, s>>>(h, cu_q, B, m, D, mod, mod_stride, shift_off, scale_off, a, idx,   \
                                            token_region, region_req);                                          \
    break;
    FD_LN_CASE(1) FD_LN_CASE(2) FD_LN_CASE(3) FD_LN_CASE(4) FD_LN_CASE(5) FD_LN_CASE(6) FD_LN_CASE(8)
    FD_LN_CASE(12) FD_LN_CASE(16)
#undef FD_LN_CASE
    default:
      ln_modulate_kernel<0><<<grid, 256, 0, s>>>(h, cu_q, B, m, D, mod, mod_stride, shift_off, scale_off, a, idx,
                                                 token_region, region_req);
  }
  return hipGetLastError();
}

}  // namespace fdh
