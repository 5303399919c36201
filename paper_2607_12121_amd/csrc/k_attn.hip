// Attention of the active queries over every token of their request, K/V read
// from the per-block cache (fresh rows for active tokens, stale rows for skipped
// ones).  Flash-style with an fp32 online softmax (base-2 exponent); both
// contractions run on v_mfma_f32_32x32x16_bf16.
//
// Work unit = (head, 128-query tile of one request, KV split).  A workgroup of 4
// waves owns a unit, 32 queries per wave.  Each wave computes S^T = K Q^T (keys x
// queries), so a lane owns one query column: its running max needs one
// half-wave exchange per tile and its running sum none until the end; S^T feeds
// O^T = V^T P^T directly as the B operand.
//
// K and V tiles of 64 keys stream from HBM straight into LDS (buffer_load ...
// lds) through a ring of stages, both row-major with 16-byte chunk c of key row k
// stored at c ^ (k % 8).  The V^T operand is read with ds_read_b64_tr_b16: in a
// group of 16 lanes, lane j addresses 4 consecutive d of key K0 + j/4 and every
// lane receives its own d for keys K0..K0+3, so V needs no transposing stores.
//
// When the units of a launch do not fill the CUs, every (head, query tile) is cut
// into S contiguous key ranges; each split stores its unnormalised O, max and
// sum with device-coherent stores and the last split to arrive combines them in
// split order (deterministic).  Units are numbered head-major and dealt to the 8
// XCDs in contiguous chunks so that the query tiles sharing a head's K/V run on
// the same L2.
#include "fd_common.h"

namespace {

constexpr int kXcds = 8;
constexpr int QB = 128, KB = 64;
constexpr int kWaves = 4, kThreads = kWaves * 64;
constexpr int kMaxKvSplit = 16;

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef int int32x4_t __attribute__((ext_vector_type(4)));
typedef short short4_t __attribute__((ext_vector_type(4)));

FD_DEVICE int32x4_t buffer_rsrc(const void* base) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  int32x4_t r;
  r.x = static_cast<int>(static_cast<uint32_t>(p));
  r.y = static_cast<int>(static_cast<uint32_t>(p >> 32) & 0xffffu);
  r.z = 0x7fffffff;
  r.w = 0x00020000;
  return r;
}

// 16 bytes per lane from buffer offset `voff` into LDS at lds_addr + 16 * lane.
FD_DEVICE void lds_dma16(uint32_t lds_addr, uint32_t voff, int32x4_t rsrc) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" : : "s"(lds_addr), "v"(voff), "s"(rsrc));
}

template <int N>
FD_DEVICE void wait_vm_barrier() {
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" : : "n"(N) : "memory");
}

// max / sum of v over lanes l and l ^ 32 (v_permlane32_swap exchanges the halves)
FD_DEVICE float half_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
FD_DEVICE float half_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int DH>
struct ACfg {
  static constexpr int KCH = DH / 8;                    // 16-byte chunks per key row
  static constexpr int SW = KCH < 8 ? KCH : 8;          // swizzle span
  static constexpr int TILE = KB * KCH;                 // chunks of one K or V tile
  static constexpr int STAGE = 2 * TILE;                // K tile then V tile
  static constexpr int STAGES = DH >= 128 ? 2 : 3;
  static constexpr int LOADS = STAGE / 64 / kWaves;     // 1 KB wave-loads per wave per stage
  static constexpr int KS = DH / 16;                    // k-steps of S^T over d
  static constexpr int DT = (DH + 31) / 32;             // 32-row tiles of O^T
  static_assert(STAGE % (64 * kWaves) == 0, "stage must split into whole wave-loads");
};

FD_DEVICE float split_eff(int units, int slots) {
  const int waves = (units + slots - 1) / slots;
  return static_cast<float>(units) / static_cast<float>(waves * slots);
}

FD_DEVICE int choose_kv_split(int items, int n_kv, int slots, int max_units) {
  int best = 1;
  float best_e = split_eff(items, slots);
  for (int s = 2; s <= kMaxKvSplit; ++s) {
    if (n_kv < 4 * s || items * s > max_units) break;
    const float e = split_eff(items * s, slots) - 0.03f * static_cast<float>(s - 1);
    if (e > best_e + 1e-6f) {
      best_e = e;
      best = s;
    }
  }
  return best;
}

template <int DH>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc, const uint16_t* __restrict__ Vc,
    uint16_t* __restrict__ O, int D, int H, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ req_tok_off,
    int B, int max_req_tokens, float scale_log2, float* __restrict__ partial, int32_t* __restrict__ counters,
    int max_units, int slots) {
  using C = ACfg<DH>;
  __shared__ uint4 ring[C::STAGES][C::STAGE];
  __shared__ int s_last;

  // query tiles over all requests, then units = heads x tiles x splits
  int tiles = 0;
  for (int b = 0; b < B; ++b) tiles += (cu_q[b + 1] - cu_q[b] + QB - 1) / QB;
  if (tiles == 0) return;
  const int S = choose_kv_split(H * tiles, (max_req_tokens + KB - 1) / KB, slots, max_units);
  const int units = H * tiles * S;
  const int per_xcd = (units + kXcds - 1) / kXcds;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, lg = lane >> 5;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int32x4_t rs_k = buffer_rsrc(Kc);
  const int32x4_t rs_v = buffer_rsrc(Vc);
  const uint32_t ring_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)&ring[0][0]));

  for (int u = blockIdx.x; u < per_xcd * kXcds; u += gridDim.x) {
    const int v = (u % kXcds) * per_xcd + u / kXcds;
    if (v >= units) continue;
    const int head = v / (tiles * S);
    const int item = v / S;                       // (head, tile) pair: the split counter's index
    const int tau = (v / S) % tiles;
    const int split = v % S;
    int b = 0, first = 0;
    for (;; ++b) {
      const int nt = (cu_q[b + 1] - cu_q[b] + QB - 1) / QB;
      if (tau < first + nt) break;
      first += nt;
    }
    const int q_lo = cu_q[b] + (tau - first) * QB;
    const int q_hi = cu_q[b + 1];
    const int k_beg = req_tok_off[b], k_end = req_tok_off[b + 1];
    const int n_kv = (k_end - k_beg + KB - 1) / KB;
    const int kt0 = (split * n_kv) / S, kt1 = ((split + 1) * n_kv) / S;
    const int nkt = kt1 - kt0;
    const size_t col0 = static_cast<size_t>(head) * DH;

    const int qrow = q_lo + wave * 32 + l32;
    const bool qvalid = qrow < q_hi;
    bf16x8_t qf[C::KS];
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      uint4 t = make_uint4(0, 0, 0, 0);
      if (qvalid) t = *reinterpret_cast<const uint4*>(Q + static_cast<size_t>(qrow) * D + col0 + ks * 16 + lg * 8);
      qf[ks] = __builtin_bit_cast(bf16x8_t, t);
    }

    // this lane's row and source chunk inside each of its wave-loads
    auto issue = [&](int kt, int st) {
      const int k0 = k_beg + kt * KB;
      const uint32_t buf = ring_base + static_cast<uint32_t>(st * C::STAGE * 16);
#pragma unroll
      for (int q = 0; q < C::LOADS; ++q) {
        const int blk = wave + kWaves * q;                 // 1 KB block of the stage
        const bool is_v = blk * 64 >= C::TILE;
        const int p = blk * 64 + lane - (is_v ? C::TILE : 0);
        const int r = p / C::KCH;                          // key row within the tile
        const int c = (p % C::KCH) ^ (r % C::SW);          // logical chunk
        const int key = min(k0 + r, k_end - 1);
        const uint32_t off = static_cast<uint32_t>((static_cast<size_t>(key) * D + col0 + c * 8) * 2);
        const uint32_t dst = buf + static_cast<uint32_t>((wave_u + kWaves * q) * 64 * 16);
        if (is_v)
          lds_dma16(dst, off, rs_v);
        else
          lds_dma16(dst, off, rs_k);
      }
    };

    f32x16_t oacc[C::DT];
#pragma unroll
    for (int d = 0; d < C::DT; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[d][r] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;

    // V^T operand addressing for ds_read_b64_tr_b16 (see file comment)
    const int grp = lane >> 4, jj = lane & 15;
    const int tr_key = 4 * lg + (jj >> 2);                 // + 16 * st + 8 * half
    const int tr_d = 16 * (grp & 1) + 4 * (jj & 3);       // + 32 * dt
    const bool tr_live = (DH >= 32) || (grp & 1) == 0;    // rows d >= DH are zero operand rows

#pragma unroll
    for (int p = 0; p < C::STAGES - 1; ++p)
      if (p < nkt) issue(kt0 + p, p);
    for (int it = 0; it < nkt; ++it) {
      const int younger = min(C::STAGES - 2, nkt - 1 - it);
      if (younger >= 1) wait_vm_barrier<C::LOADS>();
      else wait_vm_barrier<0>();
      if (it + C::STAGES - 1 < nkt) issue(kt0 + it + C::STAGES - 1, (it + C::STAGES - 1) % C::STAGES);
      const uint4* kt_lds = ring[it % C::STAGES];
      const uint32_t vt_addr = ring_base + static_cast<uint32_t>(((it % C::STAGES) * C::STAGE + C::TILE) * 16);
      const int k0 = k_beg + (kt0 + it) * KB;

      // S^T (64 keys x 32 queries) = K Q^T, two 32-key halves
      f32x16_t sacc[2];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[kh][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) {
          const int key = kh * 32 + l32;
          const int ch = ks * 2 + lg;
          const bf16x8_t a = __builtin_bit_cast(bf16x8_t, kt_lds[key * C::KCH + (ch ^ (key % C::SW))]);
          sacc[kh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], sacc[kh], 0, 0, 0);
        }
      }
      // keys past the request end (last tile only): -inf
      if (k0 + KB > k_end) {
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (k0 + kh * 32 + 8 * (r >> 2) + 4 * lg + (r & 3) >= k_end) sacc[kh][r] = -INFINITY;
      }
      float mx = sacc[0][0];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kh][r]);
      const float m_new = fmaxf(m_run, half_max(mx) * scale_log2);
      if (__any(m_new > m_run)) {   // rescale only when some running max grew
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int d = 0; d < C::DT; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[d][r] *= alpha;
      }
      m_run = m_new;
      bf16x8_t pk[4];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          bf16x8_t pv;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pe = __builtin_amdgcn_exp2f(fmaf(sacc[kh][half * 8 + e], scale_log2, -m_new));
            l_run += pe;
            pv[e] = static_cast<__bf16>(pe);
          }
          pk[kh * 2 + half] = pv;
        }
      // O^T (d x 32 queries) += V^T P^T; k-step st covers keys 16 st .. 16 st + 15
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt) {
#pragma unroll
        for (int st = 0; st < 4; ++st) {
          short4_t lo = {0, 0, 0, 0}, hi = {0, 0, 0, 0};
          if (tr_live) {
            const int d_s = dt * 32 + tr_d;
            const int key_lo = 16 * st + tr_key, key_hi = key_lo + 8;
            const int c_lo = (d_s >> 3) ^ (key_lo % C::SW), c_hi = (d_s >> 3) ^ (key_hi % C::SW);
            const uint32_t a_lo = vt_addr + static_cast<uint32_t>(key_lo * C::KCH * 16 + c_lo * 16 + (d_s & 7) * 2);
            const uint32_t a_hi = vt_addr + static_cast<uint32_t>(key_hi * C::KCH * 16 + c_hi * 16 + (d_s & 7) * 2);
            lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)(uintptr_t)a_lo);
            hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)(uintptr_t)a_hi);
          }
          const short lo_hi[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          bf16x8_t av;
#pragma unroll
          for (int e = 0; e < 8; ++e) av[e] = __builtin_bit_cast(__bf16, lo_hi[e]);
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pk[st], oacc[dt], 0, 0, 0);
        }
      }
    }
    __syncthreads();   // the ring is refilled by the next unit
    l_run = half_sum(l_run);

    if (S > 1) {
      // store this split's unnormalised O, max and sum (lane-major), count the arrival
      constexpr int E = C::DT * 16 + 2;
      float* slot = partial + static_cast<size_t>(v) * (E * kThreads) + tid;
#pragma unroll
      for (int d = 0; d < C::DT; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          __hip_atomic_store(slot + (d * 16 + r) * kThreads, oacc[d][r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(slot + (E - 2) * kThreads, m_run, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(slot + (E - 1) * kThreads, l_run, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (tid == 0) {
        const int prev = __hip_atomic_fetch_add(&counters[item], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = (prev == S - 1);
        if (prev == S - 1) __hip_atomic_store(&counters[item], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      __syncthreads();
      if (!s_last) continue;
      // combine the S splits in split order
      const float* base = partial + static_cast<size_t>(item) * S * (E * kThreads) + tid;
      float m_all = -INFINITY;
      for (int s2 = 0; s2 < S; ++s2)
        m_all = fmaxf(m_all, __hip_atomic_load(base + static_cast<size_t>(s2) * E * kThreads + (E - 2) * kThreads,
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      float l_all = 0.f;
#pragma unroll
      for (int d = 0; d < C::DT; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[d][r] = 0.f;
      for (int s2 = 0; s2 < S; ++s2) {
        const float* ps = base + static_cast<size_t>(s2) * E * kThreads;
        const float ms = __hip_atomic_load(ps + (E - 2) * kThreads, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const float w = (ms == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ms - m_all);
        l_all += w * __hip_atomic_load(ps + (E - 1) * kThreads, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int d = 0; d < C::DT; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            oacc[d][r] += w * __hip_atomic_load(ps + (d * 16 + r) * kThreads, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
      }
      l_run = l_all;
    }

    if (!qvalid) continue;
    const float inv_l = 1.0f / l_run;
    uint16_t* orow = O + static_cast<size_t>(qrow) * D + col0;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
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
}

}  // namespace

namespace fdh {

size_t attn_scratch_bytes(int dh) {
  const size_t units = static_cast<size_t>(gemm_max_tiles());
  const size_t e = static_cast<size_t>(((dh + 31) / 32) * 16 + 2);
  return units * e * kThreads * sizeof(float);
}

hipError_t launch_attention(const uint16_t* q, const uint16_t* kc, const uint16_t* vc, uint16_t* o, int D, int H,
                            int dh, const int32_t* cu_q, const int32_t* req_tok_off, int B, int n_max,
                            int max_req_tokens, float* partial, int32_t* counters, hipStream_t s) {
  const int slots = 2 * num_cus();
  const int max_units = (partial && counters) ? gemm_max_tiles() : 0;
  // upper bound on the units: every request adds at most one partial query tile
  const long long items = static_cast<long long>((n_max + QB - 1) / QB + B) * H;
  long long grid = items * kMaxKvSplit;
  if (grid > slots) grid = slots;
  grid = ((grid + kXcds - 1) / kXcds) * kXcds;
  const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(dh));
#define FD_ATTN_LAUNCH(DHV)                                                                                         \
  attn_fwd_kernel<DHV><<<grid, kThreads, 0, s>>>(q, kc, vc, o, D, H, cu_q, req_tok_off, B, max_req_tokens, scale_log2, \
                                                 partial, counters, max_units, slots)
  switch (dh) {
    case 16: FD_ATTN_LAUNCH(16); break;
    case 64: FD_ATTN_LAUNCH(64); break;
    case 128: FD_ATTN_LAUNCH(128); break;
    default: return hipErrorInvalidValue;
  }
#undef FD_ATTN_LAUNCH
  return hipGetLastError();
}

}  // namespace fdh
