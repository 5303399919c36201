// Attention of the active queries over every token of their request, K/V read
// from the per-block cache (fresh rows for active tokens, stale rows for skipped
// ones).  Flash-style: K/V tiles of 64 keys stream through LDS, the softmax is
// online in fp32 (base-2 exponent), both contractions run on
// v_mfma_f32_32x32x16_bf16.
//
// The wave computes S^T = K Q^T (keys x queries) so that each lane owns one query
// column: its row max / row sum need one cross-half exchange only, and the S^T
// accumulator is directly the B operand (P^T) of O^T = V^T P^T.  V is stored
// transposed in LDS (d-major) to serve as that product's A operand.
//
// Work item = (request, 128-query tile, head); a workgroup of 4 waves owns one
// item, 32 queries per wave.  Items are numbered tile-major over the device-side
// per-request query counts; workgroups past the last item exit at once.
#include "fd_common.h"

namespace {

constexpr int BQ = 128, BKV = 64;
constexpr int kThreads = 256;

template <int DH>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(const uint16_t* __restrict__ Q,
                                                               const uint16_t* __restrict__ Kc,
                                                               const uint16_t* __restrict__ Vc,
                                                               uint16_t* __restrict__ O, int D, int H,
                                                               const int32_t* __restrict__ cu_q,
                                                               const int32_t* __restrict__ req_tok_off, int B,
                                                               float scale_log2) {
  constexpr int KCH = DH / 8;               // 16-byte chunks per key row
  constexpr int KS = DH / 16;               // k-steps of S^T over d
  constexpr int DT = (DH + 31) / 32;        // 32-row tiles of O^T
  constexpr int KSW = KCH < 8 ? KCH : 8;    // swizzle span of K rows
  constexpr int UNITS = BKV / 4;            // 8-byte units (4 keys) per V^T row
  constexpr int LOADS = BKV * KCH / kThreads > 0 ? BKV * KCH / kThreads : 1;
  __shared__ uint4 k_s[2][BKV * KCH];
  __shared__ uint2 v_s[2][DH * UNITS];

  const int head = blockIdx.x % H;
  const int tile = blockIdx.x / H;
  int b = 0, first = 0;
  for (; b < B; ++b) {
    const int nt = (cu_q[b + 1] - cu_q[b] + BQ - 1) / BQ;
    if (tile < first + nt) break;
    first += nt;
  }
  if (b >= B) return;
  const int q_lo = cu_q[b] + (tile - first) * BQ;
  const int q_hi = cu_q[b + 1];
  const int k_lo = req_tok_off[b], k_hi = req_tok_off[b + 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, lg = lane >> 5;
  const int qrow = q_lo + wave * 32 + l32;
  const bool qvalid = qrow < q_hi;
  const size_t col0 = static_cast<size_t>(head) * DH;

  bf16x8_t qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (qvalid) v = *reinterpret_cast<const uint4*>(Q + static_cast<size_t>(qrow) * D + col0 + ks * 16 + lg * 8);
    qf[ks] = __builtin_bit_cast(bf16x8_t, v);
  }

  f32x16_t oacc[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[d][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  uint4 rk[LOADS], rv[LOADS];
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int c = tid + kThreads * i;
      rk[i] = make_uint4(0, 0, 0, 0);
      rv[i] = make_uint4(0, 0, 0, 0);
      if (c < BKV * KCH) {
        const int key = c / KCH, ch = c % KCH;
        const int gk = k0 + key;
        if (gk < k_hi) {
          const size_t off = static_cast<size_t>(gk) * D + col0 + ch * 8;
          rk[i] = *reinterpret_cast<const uint4*>(Kc + off);
          rv[i] = *reinterpret_cast<const uint4*>(Vc + off);
        }
      }
    }
  };
  auto store = [&](int s) {
    uint16_t* vt = reinterpret_cast<uint16_t*>(v_s[s]);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int c = tid + kThreads * i;
      if (c < BKV * KCH) {
        const int key = c / KCH, ch = c % KCH;
        k_s[s][key * KCH + (ch ^ (key % KSW))] = rk[i];
        const uint32_t w[4] = {rv[i].x, rv[i].y, rv[i].z, rv[i].w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int d = ch * 8 + e;
          const uint16_t val = static_cast<uint16_t>((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu));
          vt[d * BKV + (((key >> 2) ^ (d & 15)) << 2) + (key & 3)] = val;
        }
      }
    }
  };

  load(k_lo);
  store(0);
  __syncthreads();
  int it = 0;
  for (int k0 = k_lo; k0 < k_hi; k0 += BKV, ++it) {
    const int s = it & 1;
    const bool more = k0 + BKV < k_hi;
    if (more) load(k0 + BKV);

    // S^T (64 keys x 32 queries) = K Q^T, two 32-key halves
    f32x16_t sacc[2];
#pragma unroll
    for (int kh = 0; kh < 2; ++kh) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kh][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int key = kh * 32 + l32;
        const int ch = ks * 2 + lg;
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, k_s[s][key * KCH + (ch ^ (key % KSW))]);
        sacc[kh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], sacc[kh], 0, 0, 0);
      }
    }
    // online softmax over this tile for the lane's query column
    float mx = -INFINITY;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + kh * 32 + 8 * (r >> 2) + 4 * lg + (r & 3);
        const float v = key < k_hi ? sacc[kh][r] * scale_log2 : -INFINITY;
        sacc[kh][r] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);
    float rs = 0.f;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2f(sacc[kh][r] - m_new);
        sacc[kh][r] = p;
        rs += p;
      }
    rs += __shfl_xor(rs, 32, 64);
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[d][r] *= alpha;

    // P^T as bf16 B operands: k-step st = 2*kh + half covers keys 16*st .. 16*st+15
    bf16x8_t pk[4];
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        bf16x8_t p;
#pragma unroll
        for (int e = 0; e < 8; ++e) p[e] = static_cast<__bf16>(sacc[kh][half * 8 + e]);
        pk[kh * 2 + half] = p;
      }
    // O^T (d x 32 queries) += V^T P^T
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int d = dt * 32 + l32;
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        uint2 u0 = make_uint2(0, 0), u1 = make_uint2(0, 0);
        if (DH >= 32 || d < DH) {
          u0 = v_s[s][d * UNITS + ((4 * st + lg) ^ (d & 15))];
          u1 = v_s[s][d * UNITS + ((4 * st + 2 + lg) ^ (d & 15))];
        }
        const uint4 av = make_uint4(u0.x, u0.y, u1.x, u1.y);
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, av), pk[st], oacc[dt], 0, 0,
                                                           0);
      }
    }
    if (more) store(s ^ 1);
    __syncthreads();
  }

  if (!qvalid) return;
  const float inv_l = 1.0f / l_run;
  uint16_t* orow = O + static_cast<size_t>(qrow) * D + col0;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d0 = dt * 32 + 8 * r4 + 4 * lg;
      if (d0 >= DH) continue;
      uint2 o;
      o.x = fd::pack_bf2(oacc[dt][4 * r4 + 0] * inv_l, oacc[dt][4 * r4 + 1] * inv_l);
      o.y = fd::pack_bf2(oacc[dt][4 * r4 + 2] * inv_l, oacc[dt][4 * r4 + 3] * inv_l);
      *reinterpret_cast<uint2*>(orow + d0) = o;
    }
}

}  // namespace

namespace fdh {

hipError_t launch_attention(const uint16_t* q, const uint16_t* kc, const uint16_t* vc, uint16_t* o, int D, int H,
                            int dh, const int32_t* cu_q, const int32_t* req_tok_off, int B, int n_max,
                            const int32_t* m, hipStream_t s) {
  (void)m;
  // upper bound on the number of (request, query tile) pairs: every request adds
  // at most one partial tile
  const long long items = static_cast<long long>((n_max + BQ - 1) / BQ + B) * H;
  const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(dh));
  const int grid = static_cast<int>(items);
  switch (dh) {
    case 16: attn_fwd_kernel<16><<<grid, kThreads, 0, s>>>(q, kc, vc, o, D, H, cu_q, req_tok_off, B, scale_log2); break;
    case 64: attn_fwd_kernel<64><<<grid, kThreads, 0, s>>>(q, kc, vc, o, D, H, cu_q, req_tok_off, B, scale_log2); break;
    case 128: attn_fwd_kernel<128><<<grid, kThreads, 0, s>>>(q, kc, vc, o, D, H, cu_q, req_tok_off, B, scale_log2); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace fdh
