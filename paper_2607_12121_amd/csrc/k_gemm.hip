// bf16 MFMA GEMM with fused epilogues for the DiT block on the active rows.
//
// C[M][N] = A[M][K] * B[N][K]^T, A = activations (bf16, row-major), B = weights
// ([out][in] bf16), fp32 accumulation on v_mfma_f32_32x32x16_bf16.  M (the number
// of active rows) lives on the device; the kernel is persistent: each workgroup
// walks tiles blockIdx.x, blockIdx.x + gridDim.x, ... while they exist for the
// current M, so the launch needs no host-side M.
//
// Tiling: 128x128 workgroup tile, BK = 64, 4 waves in a 2x2 grid, each wave a
// 64x64 sub-tile of 2x2 MFMA 32x32 blocks.  A and B tiles are staged in LDS,
// double-buffered, as rows of eight 16-byte chunks with chunk c of row r stored
// at c ^ (r & 7) so that the MFMA operand reads (8 consecutive rows, one chunk
// each) hit distinct banks.  The next K-slice is fetched into registers while
// the current one feeds the MFMAs.
#include "fd_common.h"

namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kThreads = 256;
constexpr int kChunks = BK / 8;                         // 16-byte chunks per tile row
constexpr int kLoadsA = BM * kChunks / kThreads;        // 4
constexpr int kLoadsB = BN * kChunks / kThreads;        // 4

struct Frag {
  f32x16_t c[2][2];
};

template <int KIND>
FD_DEVICE void epilogue(const fdh::GemmArgs& g, int row, int col, float acc) {
  const float val = acc + g.bias[col];
  if constexpr (KIND == fdh::GEMM_QKV) {
    const int D = g.D;
    if (col < D) {
      g.out_bf16[static_cast<size_t>(row) * D + col] = fd::f2bf(val);
    } else {
      const size_t tok = static_cast<size_t>(g.idx[row]);
      if (col < 2 * D)
        g.k_cache[tok * D + (col - D)] = fd::f2bf(val);
      else
        g.v_cache[tok * D + (col - 2 * D)] = fd::f2bf(val);
    }
  } else if constexpr (KIND == fdh::GEMM_RESID) {
    const int b = fd::row_request(g.cu_q, g.n_req, row);
    float* hp = g.out_f32 + static_cast<size_t>(row) * g.N + col;
    *hp = *hp + g.gate[static_cast<size_t>(b) * g.gate_stride + col] * val;
  } else if constexpr (KIND == fdh::GEMM_GELU) {
    g.out_bf16[static_cast<size_t>(row) * g.N + col] = fd::f2bf(fd::gelu_tanh(val));
  } else if constexpr (KIND == fdh::GEMM_EMBED) {
    g.out_f32[static_cast<size_t>(row) * g.N + col] = val + g.pos[static_cast<size_t>(g.idx[row]) * g.N + col];
  } else {
    g.out_f32[static_cast<size_t>(row) * g.N + col] = val;
  }
}

template <int KIND>
__global__ __launch_bounds__(kThreads, 2) void gemm_bf16_kernel(fdh::GemmArgs g) {
  __shared__ uint4 smem[2][(BM + BN) * kChunks];
  const int M = min(*g.m, g.n_max);
  const int N = g.N, K = g.K;
  const int tiles_m = (M + BM - 1) / BM;
  const int tiles_n = (N + BN - 1) / BN;
  const int total = tiles_m * tiles_n;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, lg = lane >> 5;
  const int nk = (K + BK - 1) / BK;
  const uint4 zero = make_uint4(0, 0, 0, 0);

  for (int t = blockIdx.x; t < total; t += gridDim.x) {
    const int tm = t % tiles_m, tn = t / tiles_m;
    const int m0 = tm * BM, n0 = tn * BN;
    uint4 ra[kLoadsA], rb[kLoadsB];

    auto load = [&](int k0) {
#pragma unroll
      for (int i = 0; i < kLoadsA; ++i) {
        const int c = tid + kThreads * i, row = c >> 3, ch = c & 7;
        const int gm = m0 + row, gk = k0 + ch * 8;
        ra[i] = zero;
        if (gm < M && gk < K) ra[i] = *reinterpret_cast<const uint4*>(g.act + static_cast<size_t>(gm) * K + gk);
      }
#pragma unroll
      for (int i = 0; i < kLoadsB; ++i) {
        const int c = tid + kThreads * i, row = c >> 3, ch = c & 7;
        const int gn = n0 + row, gk = k0 + ch * 8;
        rb[i] = zero;
        if (gn < N && gk < K) rb[i] = *reinterpret_cast<const uint4*>(g.wt + static_cast<size_t>(gn) * K + gk);
      }
    };
    auto store = [&](int s) {
#pragma unroll
      for (int i = 0; i < kLoadsA; ++i) {
        const int c = tid + kThreads * i, row = c >> 3, ch = c & 7;
        smem[s][row * kChunks + (ch ^ (row & 7))] = ra[i];
      }
#pragma unroll
      for (int i = 0; i < kLoadsB; ++i) {
        const int c = tid + kThreads * i, row = c >> 3, ch = c & 7;
        smem[s][(BM + row) * kChunks + (ch ^ (row & 7))] = rb[i];
      }
    };

    Frag acc;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc.c[i][j][r] = 0.f;

    load(0);
    store(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int s = kt & 1;
      const bool more = kt + 1 < nk;
      if (more) load((kt + 1) * BK);
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int ch = ks * 2 + lg;
        bf16x8_t a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const int row = wm * 64 + i * 32 + l32;
          a[i] = __builtin_bit_cast(bf16x8_t, smem[s][row * kChunks + (ch ^ (row & 7))]);
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int row = wn * 64 + j * 32 + l32;
          b[j] = __builtin_bit_cast(bf16x8_t, smem[s][(BM + row) * kChunks + (ch ^ (row & 7))]);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc.c[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc.c[i][j], 0, 0, 0);
      }
      if (more) store(s ^ 1);
      __syncthreads();
    }

    // Accumulator layout of a 32x32 block: lane holds column l32 and rows
    // 8*(r/4) + 4*lg + (r%4), r = 0..15.
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * lg + (r & 3);
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = n0 + wn * 64 + j * 32 + l32;
          if (col < N) epilogue<KIND>(g, row, col, acc.c[i][j][r]);
        }
      }
    }
  }
}

}  // namespace

namespace fdh {

hipError_t launch_gemm(GemmKind kind, const GemmArgs& a, hipStream_t s) {
  const long long tiles = static_cast<long long>((a.n_max + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  const long long cap = 2LL * num_cus();
  const int grid = static_cast<int>(tiles < cap ? (tiles < 1 ? 1 : tiles) : cap);
  switch (kind) {
    case GEMM_QKV: gemm_bf16_kernel<GEMM_QKV><<<grid, kThreads, 0, s>>>(a); break;
    case GEMM_RESID: gemm_bf16_kernel<GEMM_RESID><<<grid, kThreads, 0, s>>>(a); break;
    case GEMM_GELU: gemm_bf16_kernel<GEMM_GELU><<<grid, kThreads, 0, s>>>(a); break;
    case GEMM_EMBED: gemm_bf16_kernel<GEMM_EMBED><<<grid, kThreads, 0, s>>>(a); break;
    case GEMM_OUT: gemm_bf16_kernel<GEMM_OUT><<<grid, kThreads, 0, s>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace fdh
