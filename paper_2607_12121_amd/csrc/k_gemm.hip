// bf16 MFMA GEMM with fused epilogues for the DiT block on the active rows.
//
// C[M][N] = A[M][K] * B[N][K]^T, A = activations (bf16, row-major), B = weights
// ([out][in] bf16), fp32 accumulation on v_mfma_f32_32x32x16_bf16.  M (the number
// of active rows) lives on the device, so the kernels are persistent: each
// workgroup walks the work units that exist for the current M, and the launch
// needs no host-side M.
//
// Tiled kernel (K % 64 == 0): a BM x BN workgroup tile, BK = 64, WM x WN waves
// each owning a (BM/WM) x (BN/WN) block of 32x32 MFMA tiles.  Two shapes are
// built: 128x128 with 4 waves and two workgroups per CU (few active rows), and
// 256x256 with 8 waves and one workgroup per CU (many rows; half the LDS traffic
// per flop).  Tiles stream from HBM straight into LDS (buffer_load ... lds, 16
// bytes per lane) through a ring of stages with one barrier per K-step; every
// stage is issued (the last one re-issued at the tail) so the wait count is a
// constant.  In LDS each tile row is eight 16-byte chunks, chunk c of row r at
// c ^ ((r >> 1) & 7): the 16 lanes that read one MFMA fragment together hit 16
// different 16-byte bank groups.  Inside a K-step the next k16 fragments are read
// while the current MFMAs run (one read after each of the first MFMAs).  Rows
// past M (or N) re-read the last valid row; their results are never stored.
//
// Split-K (128x128 tiles only, when the tile count leaves CUs idle and K is long):
// every tile's K range is cut into S contiguous splits.  Each split stores its fp32
// tile to scratch and bumps the tile's arrival counter; the last split to arrive
// sums all S partials in split order (deterministic), runs the epilogue and
// resets the counter for the next launch.
//
// Epilogue: each wave moves one 32x32 accumulator block at a time through a
// private LDS patch and finishes 16 consecutive columns of one row per lane with
// vector loads and stores.
//
// Work units are dealt to the 8 XCDs in contiguous chunks of tile order (a WG
// runs on XCD blockIdx.x % 8), so the tiles one XCD runs concurrently share A
// and B rows in its L2.
#include "fd_common.h"

namespace {

constexpr int kXcds = 8;

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

// Epilogue on 8 consecutive columns col..col+7 of one output row (col % 8 == 0,
// col + 8 <= N): v holds the fp32 accumulators.  Vector loads and stores only.
template <int KIND>
FD_DEVICE void epilogue8(const fdh::GemmArgs& g, int row, int col, float v[8]) {
  const float4 b0 = *reinterpret_cast<const float4*>(g.bias + col);
  const float4 b1 = *reinterpret_cast<const float4*>(g.bias + col + 4);
  v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
  v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
  if constexpr (KIND == fdh::GEMM_QKV || KIND == fdh::GEMM_GELU) {
    if constexpr (KIND == fdh::GEMM_GELU) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = fd::gelu_tanh_fast(v[e]);
    }
    uint4 o;
    o.x = fd::pack_bf2(v[0], v[1]);
    o.y = fd::pack_bf2(v[2], v[3]);
    o.z = fd::pack_bf2(v[4], v[5]);
    o.w = fd::pack_bf2(v[6], v[7]);
    uint16_t* dst;
    if constexpr (KIND == fdh::GEMM_QKV) {
      const int D = g.D;
      if (col < D) {
        dst = g.out_bf16 + static_cast<size_t>(row) * D + col;
      } else {
        const size_t tok = static_cast<size_t>(g.idx[row]);
        dst = (col < 2 * D) ? g.k_cache + tok * D + (col - D) : g.v_cache + tok * D + (col - 2 * D);
      }
    } else {
      dst = g.out_bf16 + static_cast<size_t>(row) * g.N + col;
    }
    *reinterpret_cast<uint4*>(dst) = o;
  } else {
    float* hp = g.out_f32 + static_cast<size_t>(row) * g.N + col;
    float4 r0, r1;
    if constexpr (KIND == fdh::GEMM_RESID) {
      const int b = fd::row_request(g.cu_q, g.n_req, row);
      const float* gp = g.gate + static_cast<size_t>(b) * g.gate_stride + col;
      const float4 g0 = *reinterpret_cast<const float4*>(gp);
      const float4 g1 = *reinterpret_cast<const float4*>(gp + 4);
      const float4 h0 = *reinterpret_cast<const float4*>(hp);
      const float4 h1 = *reinterpret_cast<const float4*>(hp + 4);
      r0 = make_float4(h0.x + g0.x * v[0], h0.y + g0.y * v[1], h0.z + g0.z * v[2], h0.w + g0.w * v[3]);
      r1 = make_float4(h1.x + g1.x * v[4], h1.y + g1.y * v[5], h1.z + g1.z * v[6], h1.w + g1.w * v[7]);
    } else if constexpr (KIND == fdh::GEMM_EMBED) {
      const float* pp = g.pos + static_cast<size_t>(g.idx[row]) * g.N + col;
      const float4 p0 = *reinterpret_cast<const float4*>(pp);
      const float4 p1 = *reinterpret_cast<const float4*>(pp + 4);
      r0 = make_float4(v[0] + p0.x, v[1] + p0.y, v[2] + p0.z, v[3] + p0.w);
      r1 = make_float4(v[4] + p1.x, v[5] + p1.y, v[6] + p1.z, v[7] + p1.w);
    } else {
      r0 = make_float4(v[0], v[1], v[2], v[3]);
      r1 = make_float4(v[4], v[5], v[6], v[7]);
    }
    reinterpret_cast<float4*>(hp)[0] = r0;
    reinterpret_cast<float4*>(hp)[1] = r1;
  }
}

// ---------------------------------------------------------------- tiled kernel

template <int BM_, int BN_, int WM_, int WN_, int STAGES_, int OCC_, int BK_ = 64, bool SPREAD_ = false,
          int GROUP_M_ = 0>
struct TileCfg {
  static constexpr int GROUP_M = GROUP_M_;   // tile order: groups of GROUP_M row tiles (0: row tile fastest)
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, STAGES = STAGES_, OCC = OCC_, BK = BK_;
  // SPREAD: the next stage's loads are issued a share per k16 step, between the
  // MFMAs, instead of all at once after the barrier
  static constexpr bool SPREAD = SPREAD_;
  static constexpr int WAVES = WM * WN, THREADS = WAVES * 64;
  static constexpr int TM = BM / WM, TN = BN / WN, FM = TM / 32, FN = TN / 32;
  static constexpr int CPR = BK / 8;                        // 16-byte chunks per tile row
  static constexpr int RPW = 64 / CPR;                      // tile rows per 1 KB wave-load
  static constexpr int CHUNKS = (BM + BN) * CPR;            // 16-byte chunks per stage
  static constexpr int LOADS = (BM + BN) / RPW / WAVES;     // wave-loads per wave per stage
  static constexpr int LOADS_A = BM / RPW / WAVES;          // the first LOADS_A of them fetch A rows
  static_assert(BK == 64 || BK == 32, "K step of 64 (eight chunks per row) or 32 (four)");
  // chunk c of tile row r sits at c ^ swz(r): the 16 lanes reading one fragment (16
  // consecutive rows, one logical chunk) hit 16 different 16-byte bank groups
  static FD_DEVICE int swz(int r) { return BK == 64 ? (r >> 1) & 7 : (r >> 2) & 3; }
  static_assert(BM % (RPW * WAVES) == 0 && BN % (RPW * WAVES) == 0, "tile rows must split into whole wave-loads");
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile must be whole 32x32 MFMA blocks");
  static_assert(STAGES * CHUNKS * 16 <= 160 * 1024, "ring exceeds LDS");
};
using CfgSmall = TileCfg<128, 128, 2, 2, 2, 2>;
using CfgWide = TileCfg<128, 192, 2, 2, 2, 2>;     // 1.5x the columns: one round where 128x128 needs two
// half the columns: twice the tiles when few; its 24 KB stages fit three in the
// shared ring, and the third stage hides the load latency that two exposed
using CfgNarrow = TileCfg<128, 64, 2, 2, 3, 2>;
using CfgLarge = TileCfg<256, 256, 2, 4, 2, 1, 64, false, 8>;   // tile order in groups of 8 row tiles
constexpr int kSmallTile = 128 * 128;   // split-K partial tile (floats)
// LDS ring of the two-workgroups-per-CU kernel: the largest of its three tile shapes
constexpr int kSmallRing = CfgWide::STAGES * CfgWide::CHUNKS;
static_assert(kSmallRing >= CfgSmall::STAGES * CfgSmall::CHUNKS + 1 && kSmallRing >= CfgNarrow::STAGES * CfgNarrow::CHUNKS,
              "the small kernel's ring holds every shape (and the split flag past the 128x128 ring)");

constexpr int TBK = 64;
constexpr int kMaxSplit = 16;

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef int int32x4_t __attribute__((ext_vector_type(4)));

// Buffer resource of a raw byte buffer (base, no stride, 2^31-1 bytes in range).
FD_DEVICE int32x4_t buffer_rsrc(const void* base) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  int32x4_t r;
  r.x = static_cast<int>(static_cast<uint32_t>(p));
  r.y = static_cast<int>(static_cast<uint32_t>(p >> 32) & 0xffffu);
  r.z = 0x7fffffff;
  r.w = 0x00020000;
  return r;
}

// 16 bytes per lane from buffer offset `voff` into LDS at lds_addr + 16 * lane
// (lds_addr wave-uniform).  Issued as inline assembly so that the compiler does
// not wait for it before unrelated LDS reads; completion is awaited explicitly
// with s_waitcnt vmcnt before the barrier that publishes a stage.
FD_DEVICE void lds_dma16(uint32_t lds_addr, uint32_t voff, int32x4_t rsrc) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(rsrc));
}

// Wait until at most N of this wave's vector-memory operations are in flight,
// then barrier (no memory fence, so younger loads stay in flight).
template <int N>
FD_DEVICE void wait_vm_barrier() {
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" : : "n"(N) : "memory");
}


// Number of K splits (identical in every WG): split only while every unit keeps
// at least 24 K-steps and the units still fit the resident workgroup slots.
FD_DEVICE int choose_split(int tiles, int nk, int slots, int max_units) {
  int s = 1;
  while (s < kMaxSplit && tiles * (s + 1) <= slots && tiles * (s + 1) <= max_units && nk / (s + 1) >= 24) ++s;
  return s;
}

// All tiles of one GEMM with tile shape Cfg, the workgroup's LDS ring at ring_mem
// (STAGES * CHUNKS 16-byte chunks at least) and the split-K arrival flag at s_last.
template <class Cfg, int KIND>
FD_DEVICE void gemm_tiles(const fdh::GemmArgs& g, int slots, int M, uint4* ring_mem, int& s_last) {
  constexpr int BM = Cfg::BM, BN = Cfg::BN, FM = Cfg::FM, FN = Cfg::FN, TM = Cfg::TM, TN = Cfg::TN;
  constexpr int WAVES = Cfg::WAVES, THREADS = Cfg::THREADS, LOADS = Cfg::LOADS, STAGES = Cfg::STAGES;
  constexpr int PATCH = 32 * 36;   // per-wave epilogue patch (floats), row stride 36
  static_assert(WAVES * PATCH * 4 <= STAGES * Cfg::CHUNKS * 16, "epilogue patches must fit in the ring");
  const int N = g.N, K = g.K;
  const int tiles_m = (M + BM - 1) / BM;
  const int tiles_n = (N + BN - 1) / BN;
  const int tiles = tiles_m * tiles_n;
  constexpr int BK = Cfg::BK, CPR = Cfg::CPR, RPW = Cfg::RPW;
  const int nk = K / BK;
  const int S = (BM * BN == kSmallTile && g.max_units > 0) ? choose_split(tiles, nk, slots, g.max_units) : 1;
  const int units = tiles * S;
  const int per_xcd = (units + kXcds - 1) / kXcds;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / Cfg::WN, wn = wave % Cfg::WN;
  const int l32 = lane & 31, lg = lane >> 5;
  const int32x4_t rs_a = buffer_rsrc(g.act);
  const int32x4_t rs_b = buffer_rsrc(g.wt);
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t ring_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)&ring_mem[0]));

  for (int u = blockIdx.x; u < per_xcd * kXcds; u += gridDim.x) {
    const int v = (u % kXcds) * per_xcd + u / kXcds;
    if (v >= units) continue;
    const int tile = v / S, split = v - (v / S) * S;
    int tm, tn;
    if constexpr (Cfg::GROUP_M > 0) {
      // groups of GROUP_M row tiles x every column tile, row tile fastest: the tiles
      // an XCD runs at once form a GROUP_M x (concurrent / GROUP_M) rectangle that
      // shares its A and B panels in that XCD's L2
      const int per_group = Cfg::GROUP_M * tiles_n;
      const int grp = tile / per_group, r = tile - grp * per_group;
      const int gm = min(Cfg::GROUP_M, tiles_m - grp * Cfg::GROUP_M);
      tm = grp * Cfg::GROUP_M + r % gm;
      tn = r / gm;
    } else {
      tm = tile % tiles_m;
      tn = tile / tiles_m;
    }
    const int m0 = tm * BM, n0 = tn * BN;
    const int kt0 = (split * nk) / S, kt1 = ((split + 1) * nk) / S;
    const int nkt = kt1 - kt0;

    // per-lane byte offsets (k = 0) of this lane's row and source chunk in each of its wave-loads
    uint32_t off[LOADS];
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int blk = wave + WAVES * q;        // 8-row block in the concatenated A|B tile
      const int r = blk * RPW + lane / CPR;
      const int c = (lane % CPR) ^ Cfg::swz(r);
      const int gr = (q < Cfg::LOADS_A) ? min(m0 + r, M - 1) : min(n0 + (r - BM), N - 1);
      off[q] = static_cast<uint32_t>((static_cast<size_t>(gr) * K + c * 8) * 2);   // chunk = 8 bf16
    }
    // wave-loads [q0, q1) of K-step kt into stage st
    auto issue_q = [&](int kt, int st, int q0, int q1) {
      const uint32_t buf = ring_base + static_cast<uint32_t>(st * Cfg::CHUNKS * 16);
      const uint32_t kb = static_cast<uint32_t>((kt0 + kt) * BK * 2);
#pragma unroll
      for (int q = 0; q < LOADS; ++q)
        if (q >= q0 && q < q1)
          lds_dma16(buf + static_cast<uint32_t>((wave_u + WAVES * q) * 64 * 16), off[q] + kb,
                    q < Cfg::LOADS_A ? rs_a : rs_b);
    };
    auto issue = [&](int kt, int st) { issue_q(kt, st, 0, LOADS); };

    f32x16_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

#pragma unroll
    for (int p = 0; p < STAGES - 1; ++p) issue(min(p, nkt - 1), p);
    for (int it = 0; it < nkt; ++it) {
      // exactly STAGES - 2 younger stages are in flight: stage `it` has landed for every wave
      wait_vm_barrier<(STAGES - 2) * LOADS>();
      // refill the slot every wave finished reading before this barrier (a repeat at the tail)
      const int kt_next = min(it + STAGES - 1, nkt - 1), st_next = (it + STAGES - 1) % STAGES;
      if constexpr (!Cfg::SPREAD) issue(kt_next, st_next);
      const uint4* sm = ring_mem + (it % STAGES) * Cfg::CHUNKS;
      bf16x8_t a[2][FM], b[2][FN];
      auto frag = [&](int ks, int slot) {
        const int ch = ks * 2 + lg;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          const int row = wm * TM + i * 32 + l32;
          a[slot][i] = __builtin_bit_cast(bf16x8_t, sm[row * CPR + (ch ^ Cfg::swz(row))]);
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int row = BM + wn * TN + j * 32 + l32;
          b[slot][j] = __builtin_bit_cast(bf16x8_t, sm[row * CPR + (ch ^ Cfg::swz(row))]);
        }
      };
      frag(0, 0);
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        if (ks + 1 < BK / 16) frag(ks + 1, (ks + 1) & 1);
        if constexpr (Cfg::SPREAD) {
          constexpr int LQ = (LOADS + BK / 16 - 1) / (BK / 16);
          issue_q(kt_next, st_next, ks * LQ, (ks + 1) * LQ);
        }
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks & 1][i], b[ks & 1][j], acc[i][j], 0, 0, 0);
      }
      // schedule: first fragments, then per k16 step one next-step read after each of
      // the first FM + FN MFMAs, then the remaining MFMAs
      __builtin_amdgcn_sched_group_barrier(0x100, FM + FN, 0);
#pragma unroll
      for (int ks = 0; ks < BK / 16 - 1; ++ks) {
#pragma unroll
        for (int x = 0; x < FM + FN; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - (FM + FN), 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);
    }
    // the tail re-issue may still be landing: drain it before the ring is reused
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();

    if (S > 1) {
      // Store this split's tile (lane-major: element e of thread t at e * THREADS + t)
      // with device-coherent stores; once the workgroup's stores are done, thread 0
      // counts the arrival with a release read-modify-write at agent scope, and the
      // last split to arrive acquires before it reads the partials (the splits may
      // have run on other XCDs).
      float* slot = g.partial + static_cast<size_t>(v) * (BM * BN) + tid;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            __hip_atomic_store(slot + ((i * FN + j) * 16 + r) * THREADS, acc[i][j][r], __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's partials have been performed
      __syncthreads();   // ... and happen before thread 0's release below (workgroup barrier)
      if (tid == 0) {
        const int prev = __hip_atomic_fetch_add(&g.counters[tile], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        if (prev == S - 1) {
          // the last arrival: acquire every split's released partials, reset the counter
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
          __hip_atomic_store(&g.counters[tile], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        s_last = (prev == S - 1);
      }
      __syncthreads();   // thread 0's acquire happens before every thread's loads below
      if (!s_last) continue;
      // Sum the S partials (this split's included) in split order with
      // device-coherent loads: the result does not depend on which split arrived last.
      const float* base = g.partial + static_cast<size_t>(tile) * S * (BM * BN) + tid;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            acc[i][j][r] = __hip_atomic_load(base + ((i * FN + j) * 16 + r) * THREADS, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
      for (int s2 = 1; s2 < S; ++s2) {
        const float* ps = base + static_cast<size_t>(s2) * (BM * BN);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              acc[i][j][r] += __hip_atomic_load(ps + ((i * FN + j) * 16 + r) * THREADS, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
      }
    }

    // Epilogue, one 32x32 block at a time through this wave's LDS patch
    // (accumulator layout: lane holds column l32, rows 8*(r/4) + 4*lg + (r%4));
    // lane then owns row lane/2, columns 16*(lane%2) .. +15 of the block.
    float* patch = reinterpret_cast<float*>(ring_mem) + wave * PATCH;
    const int pr = lane >> 1, pc = (lane & 1) * 16;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
#pragma unroll
        for (int r = 0; r < 16; ++r) patch[(8 * (r >> 2) + 4 * lg + (r & 3)) * 36 + l32] = acc[i][j][r];
        const int row = m0 + wm * TM + i * 32 + pr, col = n0 + wn * TN + j * 32 + pc;
        const float4* src = reinterpret_cast<const float4*>(patch + pr * 36 + pc);
        float v0[8], v1[8];
        const float4 x0 = src[0], x1 = src[1], x2 = src[2], x3 = src[3];
        v0[0] = x0.x; v0[1] = x0.y; v0[2] = x0.z; v0[3] = x0.w; v0[4] = x1.x; v0[5] = x1.y; v0[6] = x1.z; v0[7] = x1.w;
        v1[0] = x2.x; v1[1] = x2.y; v1[2] = x2.z; v1[3] = x2.w; v1[4] = x3.x; v1[5] = x3.y; v1[6] = x3.z; v1[7] = x3.w;
        if (row < M) {
          if (col < N) epilogue8<KIND>(g, row, col, v0);
          if (col + 8 < N) epilogue8<KIND>(g, row, col + 8, v1);
        }
      }
    __syncthreads();   // the patches are the next unit's ring
  }
}

// Tile shape of the two-workgroups-per-CU kernel for M rows (identical in every
// WG): 128x128 whenever split-K applies; otherwise the shape whose rounds of tiles
// over the resident slots cost least, a round of 128x64 / 128x128 / 128x192 tiles
// weighted 8 / 13 / 22 (measured per-round times at 1664 rows); ties go to the
// larger tile.  0 = 128x128, 1 = 128x192, 2 = 128x64 (three-stage ring: a round
// costs 8 where its two-stage version cost 10).
FD_DEVICE int small_shape(int M, int N, int K, int slots, int max_units) {
  const int tm = (M + 127) / 128;
  const int t128 = tm * ((N + 127) / 128);
  if (max_units > 0 && choose_split(t128, K / TBK, slots, max_units) > 1) return 0;
  const int r128 = (t128 + slots - 1) / slots;
  const int r192 = (tm * ((N + 191) / 192) + slots - 1) / slots;
  const int r64 = (tm * ((N + 63) / 64) + slots - 1) / slots;
  const int c128 = 13 * r128, c192 = 22 * r192, c64 = 8 * r64;
  if (c192 <= c128 && c192 <= c64) return 1;
  if (c128 <= c64) return 0;
  return 2;
}

template <int KIND>
__global__ __launch_bounds__(256, 2) void gemm_small_kernel(fdh::GemmArgs g, int slots) {
  __shared__ uint4 ring_mem[kSmallRing];
  int& s_last = *reinterpret_cast<int*>(&ring_mem[kSmallRing - 1]);   // outside the 128x128 ring
  const int M = min(*g.m, g.n_max);
  if (M <= 0) return;
  switch (small_shape(M, g.N, g.K, slots, g.max_units)) {
    case 1: gemm_tiles<CfgWide, KIND>(g, slots, M, ring_mem, s_last); break;
    case 2: gemm_tiles<CfgNarrow, KIND>(g, slots, M, ring_mem, s_last); break;
    default: gemm_tiles<CfgSmall, KIND>(g, slots, M, ring_mem, s_last); break;
  }
}

template <int KIND>
__global__ __launch_bounds__(CfgLarge::THREADS, CfgLarge::OCC) void gemm_large_kernel(fdh::GemmArgs g, int slots) {
  __shared__ uint4 ring_mem[CfgLarge::STAGES * CfgLarge::CHUNKS];
  __shared__ int s_last;
  const int M = min(*g.m, g.n_max);
  if (M <= 0) return;
  gemm_tiles<CfgLarge, KIND>(g, slots, M, ring_mem, s_last);
}

// ---------------------------------------------------------------- simple kernel (any K % 8 == 0)

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kThreads = 256;
constexpr int kChunks = BK / 8;
constexpr int kLoadsA = BM * kChunks / kThreads;
constexpr int kLoadsB = BN * kChunks / kThreads;

template <int KIND>
__global__ __launch_bounds__(kThreads, 2) void gemm_simple_kernel(fdh::GemmArgs g) {
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

    f32x16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

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
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      }
      if (more) store(s ^ 1);
      __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * lg + (r & 3);
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = n0 + wn * 64 + j * 32 + l32;
          if (col < N) epilogue<KIND>(g, row, col, acc[i][j][r]);
        }
      }
    }
  }
}

}  // namespace

namespace fdh {

int gemm_max_tiles() { return 4 * num_cus(); }

size_t gemm_scratch_bytes() {
  const size_t units = static_cast<size_t>(gemm_max_tiles());
  return units * kSmallTile * sizeof(float) + units * sizeof(int32_t);
}

namespace {
// Row capacity (token count of the batch) from which the 256x256 tile is used.
// The active row count is only known on the device, so the choice rests on the
// capacity: at the active fractions the gate produces (20-70%), 16384 tokens give
// thousands of active rows, enough for one 256x256 tile per CU at N >= 1536.
constexpr int kLargeTileRows = 16384;

// Persistent grid: at most the resident slots, at least one workgroup per unit
// the largest unit count could need (narrowest tile, every split).
hipError_t launch_tiled(GemmKind kind, const GemmArgs& a, int max_units, bool large, hipStream_t s) {
  const int occ = large ? CfgLarge::OCC : 2;
  const int slots = num_cus() * occ;
  GemmArgs g = a;
  g.max_units = max_units;
  const int bm = large ? CfgLarge::BM : 128, bn = large ? CfgLarge::BN : CfgNarrow::BN;
  const long long tiles_max = static_cast<long long>((a.n_max + bm - 1) / bm) * ((a.N + bn - 1) / bn);
  long long grid = tiles_max * (max_units > 0 ? kMaxSplit : 1);
  if (grid > slots) grid = slots;
  grid = ((grid + kXcds - 1) / kXcds) * kXcds;
#define FD_GEMM_LAUNCH(K)                                                                      \
  if (large)                                                                                   \
    gemm_large_kernel<K><<<grid, CfgLarge::THREADS, 0, s>>>(g, slots);                         \
  else                                                                                         \
    gemm_small_kernel<K><<<grid, 256, 0, s>>>(g, slots);
  switch (kind) {
    case GEMM_QKV: FD_GEMM_LAUNCH(GEMM_QKV) break;
    case GEMM_RESID: FD_GEMM_LAUNCH(GEMM_RESID) break;
    case GEMM_GELU: FD_GEMM_LAUNCH(GEMM_GELU) break;
    case GEMM_EMBED: FD_GEMM_LAUNCH(GEMM_EMBED) break;
    case GEMM_OUT: FD_GEMM_LAUNCH(GEMM_OUT) break;
  }
#undef FD_GEMM_LAUNCH
  return hipGetLastError();
}
}  // namespace

hipError_t launch_gemm(GemmKind kind, const GemmArgs& a, hipStream_t s) {
  if (a.K % TBK == 0) {
    const int max_units = (a.partial && a.counters) ? a.max_units : 0;   // no scratch: never split
    if (a.n_max >= kLargeTileRows && a.N >= 1024) return launch_tiled(kind, a, 0, true, s);
    return launch_tiled(kind, a, max_units, false, s);
  }
  const long long tiles = static_cast<long long>((a.n_max + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  const long long cap = 2LL * num_cus();
  const int grid = static_cast<int>(tiles < cap ? (tiles < 1 ? 1 : tiles) : cap);
  switch (kind) {
    case GEMM_QKV: gemm_simple_kernel<GEMM_QKV><<<grid, kThreads, 0, s>>>(a); break;
    case GEMM_RESID: gemm_simple_kernel<GEMM_RESID><<<grid, kThreads, 0, s>>>(a); break;
    case GEMM_GELU: gemm_simple_kernel<GEMM_GELU><<<grid, kThreads, 0, s>>>(a); break;
    case GEMM_EMBED: gemm_simple_kernel<GEMM_EMBED><<<grid, kThreads, 0, s>>>(a); break;
    case GEMM_OUT: gemm_simple_kernel<GEMM_OUT><<<grid, kThreads, 0, s>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace fdh
