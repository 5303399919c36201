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
// every tile's K range is cut into S contiguous splits, each storing its fp32 tile
// to scratch; a second kernel sums the S partials in split order (deterministic)
// and runs the epilogue.  No workgroup waits for another: the kernel boundary
// orders the partial stores before the sums.
//
// The MFMA takes the weight fragment as its first operand, so each accumulator
// block is the transposed output block: a lane holds one output row and four runs
// of four consecutive columns.  The epilogue works from those registers (no LDS):
// fp32 outputs as float4, bf16 outputs as 16-byte runs after exchanging halves
// between lanes l and l + 32; per-row operands (token, request) are loaded before
// the K loop, and the gated residual keeps the next block's loads in flight.
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

// Epilogue of one 32x32 output block held transposed in a wave's accumulator (the
// MFMA takes the weight fragment as its first operand): lane (l32, lg) holds output
// row `row` and, in registers 4q .. 4q+3, columns c_q = cb + 8q + 4lg .. +3.  Every
// lane runs it (the bf16 kinds exchange halves between lanes l and l + 32); rows
// past M and columns past N (N % 16 == 0) are not stored (with kAlwaysStore, the
// bf16 kinds issue every store and send those lanes' data to `spare`).  The
// accumulators started at the bias, or at 0 with the block's 32 bias values at
// lds_bias.  tok: the row's token (QKV, EMBED).  RESID has its own pipelined loop
// in the caller.
template <int KIND, bool kAlwaysStore = false>
FD_DEVICE void epilogue_block(const fdh::GemmArgs& g, bool row_ok, int row, int cb, int lg, int tok, const f32x16_t& acc,
                              float4* spare = nullptr, const float* lds_bias = nullptr) {
  const int N = g.N;
  float v[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) v[e] = acc[e];
  if (lds_bias) {   // the bias of the block's columns from LDS (the accumulators started at 0)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 b = *reinterpret_cast<const float4*>(lds_bias + 8 * q + 4 * lg);
      v[4 * q + 0] += b.x; v[4 * q + 1] += b.y; v[4 * q + 2] += b.z; v[4 * q + 3] += b.w;
    }
  }
  if constexpr (KIND == fdh::GEMM_QKV || KIND == fdh::GEMM_GELU) {
    if constexpr (KIND == fdh::GEMM_GELU) {
#pragma unroll
      for (int e = 0; e < 16; ++e) v[e] = fd::gelu_tanh_fast(v[e]);
    }
    uint32_t pk[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) pk[e] = fd::pack_bf2(v[2 * e], v[2 * e + 1]);
    uint16_t* base;
    int c0 = cb;
    if constexpr (KIND == fdh::GEMM_QKV) {
      const int D = g.D;
      if (cb < D) {
        base = g.out_bf16 + static_cast<size_t>(row) * D;
      } else {
        base = (cb < 2 * D ? g.k_cache : g.v_cache) + static_cast<size_t>(tok) * D;
        c0 = cb - (cb < 2 * D ? D : 2 * D);
      }
    } else {
      base = g.out_bf16 + static_cast<size_t>(row) * N;
    }
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      // lanes 0-31 gather columns 16p .. 16p+7 of the block, lanes 32-63 16p+8 .. 16p+15
      const auto lo = __builtin_amdgcn_permlane32_swap(pk[4 * p + 0], pk[4 * p + 2], false, false);
      const auto hi = __builtin_amdgcn_permlane32_swap(pk[4 * p + 1], pk[4 * p + 3], false, false);
      const uint4 o = make_uint4(lo[0], hi[0], lo[1], hi[1]);
      const int off = 16 * p + 8 * lg;
      if constexpr (kAlwaysStore) {
        // one store instruction whatever the row: lanes past M or N write the spare slot
        uint4* dst = (row_ok && cb + off < N) ? reinterpret_cast<uint4*>(base + c0 + off) : reinterpret_cast<uint4*>(spare);
        *dst = o;
      } else if (row_ok && cb + off < N) {
        *reinterpret_cast<uint4*>(base + c0 + off) = o;
      }
    }
  } else {
    float* out = g.out_f32 + static_cast<size_t>(row) * N;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c = cb + 8 * q + 4 * lg;
      if (!row_ok || c >= N) continue;
      float4 r = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
      if constexpr (KIND == fdh::GEMM_EMBED) {
        const float4 pp = *reinterpret_cast<const float4*>(g.pos + static_cast<size_t>(tok) * N + c);
        r.x += pp.x; r.y += pp.y; r.z += pp.z; r.w += pp.w;
      }
      *reinterpret_cast<float4*>(out + c) = r;
    }
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
constexpr int kSideChunks = 4 * 1024 / 16;   // two 1 KB bias slots and two 1 KB token slots (256x256 tile)
// LDS ring of the two-workgroups-per-CU kernel: the largest of its three tile shapes
constexpr int kSmallRing = CfgWide::STAGES * CfgWide::CHUNKS;
static_assert(kSmallRing >= CfgSmall::STAGES * CfgSmall::CHUNKS + 1 && kSmallRing >= CfgNarrow::STAGES * CfgNarrow::CHUNKS,
              "the small kernel's ring holds every shape (and the split flag past the 128x128 ring)");

constexpr int TBK = 64;
constexpr int kMaxSplit = 16;
constexpr int kMinSplitSteps = 24;   // K-steps every split keeps

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef int int32x4_t __attribute__((ext_vector_type(4)));

// Buffer resource of a raw byte buffer (base, no stride, `bytes` in range: loads
// past it return zeros).
FD_DEVICE int32x4_t buffer_rsrc(const void* base, uint32_t bytes = 0x7fffffffu) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  int32x4_t r;
  r.x = static_cast<int>(static_cast<uint32_t>(p));
  r.y = static_cast<int>(static_cast<uint32_t>(p >> 32) & 0xffffu);
  r.z = static_cast<int>(bytes);
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
  while (s < kMaxSplit && tiles * (s + 1) <= slots && tiles * (s + 1) <= max_units && nk / (s + 1) >= kMinSplitSteps) ++s;
  return s;
}

// Epilogue of a wave's FM x FN accumulator blocks, straight from the registers:
// acc[i][j] is the transposed 32x32 block at rows row0 + 32i, columns cw + 32j (see
// epilogue_block); rtok / rreq are the token / request of row row0 + 32i.
template <int FM, int FN, int KIND>
FD_DEVICE void tile_epilogue(const fdh::GemmArgs& g, int M, int row0, int cw, int lg, const int (&rtok)[FM],
                             const int (&rreq)[FM], const f32x16_t (&acc)[FM][FN]) {
  const int N = g.N;
  if constexpr (KIND == fdh::GEMM_RESID) {
    // h += gate * acc (the bias is in acc): the next block's h and gate rows are loaded before
    // this block's stores, so each wave keeps two blocks of loads in flight
    constexpr int NB = FM * FN;
    float4 hb[2][4], gb[2][4];
    auto load_blk = [&](int bi, int sl) {
      const int i = bi / FN, j = bi - (bi / FN) * FN;
      const int r = min(row0 + 32 * i, M - 1);
      const float* hp = g.out_f32 + static_cast<size_t>(r) * N;
      const float* gp = g.gate + static_cast<size_t>(rreq[i]) * g.gate_stride;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = min(cw + 32 * j + 8 * q + 4 * lg, N - 4);
        hb[sl][q] = *reinterpret_cast<const float4*>(hp + c);
        gb[sl][q] = *reinterpret_cast<const float4*>(gp + c);
      }
    };
    load_blk(0, 0);
#pragma unroll
    for (int bi = 0; bi < NB; ++bi) {
      if (bi + 1 < NB) load_blk(bi + 1, (bi + 1) & 1);
      const int i = bi / FN, j = bi - (bi / FN) * FN, sl = bi & 1;
      const int row = row0 + 32 * i;
      float* hp = g.out_f32 + static_cast<size_t>(row) * N;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = cw + 32 * j + 8 * q + 4 * lg;
        const float4 h4 = hb[sl][q], g4 = gb[sl][q];
        const float4 r4 = make_float4(h4.x + g4.x * acc[i][j][4 * q + 0], h4.y + g4.y * acc[i][j][4 * q + 1],
                                      h4.z + g4.z * acc[i][j][4 * q + 2], h4.w + g4.w * acc[i][j][4 * q + 3]);
        if (row < M && c < N) *reinterpret_cast<float4*>(hp + c) = r4;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        epilogue_block<KIND>(g, row0 + 32 * i < M, row0 + 32 * i, cw + 32 * j, lg, rtok[i], acc[i][j]);
  }
}

// Token and request of this lane's output rows row0 + 32i (clamped to M - 1).
template <int FM, int KIND>
FD_DEVICE void row_operands(const fdh::GemmArgs& g, int M, int row0, int (&rtok)[FM], int (&rreq)[FM]) {
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int r = min(row0 + 32 * i, M - 1);
    rtok[i] = (KIND == fdh::GEMM_QKV || KIND == fdh::GEMM_EMBED) ? g.idx[r] : 0;
    rreq[i] = (KIND == fdh::GEMM_RESID) ? fd::row_request(g.cu_q, g.n_req, r) : 0;
  }
}

// All tiles of one GEMM with tile shape Cfg, the workgroup's LDS ring at ring_mem
// (STAGES * CHUNKS 16-byte chunks, followed by kSideChunks more for the bias and
// token slots of the 256x256 bf16-output kinds).
//
// Units follow each other without a drain of the output stores: on the 256x256
// tile with a bf16 output (QKV, GELU) the next unit's first stage, bias and row
// tokens (copied into the LDS slots of the unit's parity) are issued before this
// unit's epilogue, whose stores all issue (rows past M go to a spare slot), so the
// next unit's first wait leaves exactly those stores in flight (vector memory
// operations complete in issue order).  That path issues no other vector memory
// operation the compiler would wait for.
template <class Cfg, int KIND>
FD_DEVICE void gemm_tiles(const fdh::GemmArgs& g, int slots, int M, uint4* ring_mem) {
  constexpr int BM = Cfg::BM, BN = Cfg::BN, FM = Cfg::FM, FN = Cfg::FN, TM = Cfg::TM, TN = Cfg::TN;
  constexpr int WAVES = Cfg::WAVES, THREADS = Cfg::THREADS, LOADS = Cfg::LOADS, STAGES = Cfg::STAGES;
  constexpr bool kOverlap = BM * BN == 256 * 256 && (KIND == fdh::GEMM_QKV || KIND == fdh::GEMM_GELU);
  constexpr int kEpiStores = 2 * FM * FN;   // stores of one unit's epilogue_block<KIND, true> calls
  const int N = g.N, K = g.K;
  const int tiles_m = (M + BM - 1) / BM;
  const int tiles_n = (N + BN - 1) / BN;
  const int tiles = tiles_m * tiles_n;
  constexpr int BK = Cfg::BK, CPR = Cfg::CPR, RPW = Cfg::RPW;
  const int nk = K / BK;
  const int S = (BM * BN == kSmallTile && g.max_units > 0) ? choose_split(tiles, nk, slots, g.max_units) : 1;
  const int units = tiles * S;
  const int per_xcd = (units + kXcds - 1) / kXcds;
  constexpr bool overlap = kOverlap;   // g.partial (required) holds the spare slot of skipped stores
  static_assert(!kOverlap || (BN == 256 && BM == 256), "one 16-byte copy per lane covers a slot");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / Cfg::WN, wn = wave % Cfg::WN;
  const int l32 = lane & 31, lg = lane >> 5;
  const int32x4_t rs_a = buffer_rsrc(g.act);
  const int32x4_t rs_b = buffer_rsrc(g.wt);
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t ring_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)&ring_mem[0]));

  // Work unit u of this workgroup (u = blockIdx.x, + gridDim.x, ...).  gridDim.x is
  // a multiple of kXcds, so v grows with u and the valid units form a prefix.
  struct Unit { int v, split, m0, n0, kt0, nkt; };
  auto unit_at = [&](int u, Unit& t) -> bool {
    if (u >= per_xcd * kXcds) return false;
    t.v = (u % kXcds) * per_xcd + u / kXcds;
    if (t.v >= units) return false;
    const int tile = t.v / S;
    t.split = t.v - tile * S;
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
    t.m0 = tm * BM;
    t.n0 = tn * BN;
    t.kt0 = (t.split * nk) / S;
    t.nkt = ((t.split + 1) * nk) / S - t.kt0;
    return true;
  };
  // per-lane byte offsets (k = 0) of this lane's row and source chunk in each of its wave-loads
  auto offsets = [&](const Unit& t, uint32_t (&o)[LOADS]) {
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int blk = wave + WAVES * q;        // 8-row block in the concatenated A|B tile
      const int r = blk * RPW + lane / CPR;
      const int c = (lane % CPR) ^ Cfg::swz(r);
      const int gr = (q < Cfg::LOADS_A) ? min(t.m0 + r, M - 1) : min(t.n0 + (r - BM), N - 1);
      o[q] = static_cast<uint32_t>((static_cast<size_t>(gr) * K + c * 8) * 2);   // chunk = 8 bf16
    }
  };
  // wave-loads [q0, q1) of K-step kt of a unit (offsets o, first K-step kt0) into stage st
  auto issue_q = [&](const uint32_t (&o)[LOADS], int kt0, int kt, int st, int q0, int q1) {
    const uint32_t buf = ring_base + static_cast<uint32_t>(st * Cfg::CHUNKS * 16);
    const uint32_t kb = static_cast<uint32_t>((kt0 + kt) * BK * 2);
#pragma unroll
    for (int q = 0; q < LOADS; ++q)
      if (q >= q0 && q < q1)
        lds_dma16(buf + static_cast<uint32_t>((wave_u + WAVES * q) * 64 * 16), o[q] + kb, q < Cfg::LOADS_A ? rs_a : rs_b);
  };
  auto prologue = [&](const Unit& t, const uint32_t (&o)[LOADS]) {
#pragma unroll
    for (int p = 0; p < STAGES - 1; ++p) issue_q(o, t.kt0, min(p, t.nkt - 1), p, 0, LOADS);
  };
  // the bias of this lane's columns (split 0 only; the accumulators start there),
  // or, with overlap, zeros, and the tile's bias (wave 0) and row tokens (wave 1, QKV)
  // copied into the LDS slots of the unit's parity ahead of the unit's first stage
  // (bytes past the arrays read as zeros)
  const int32x4_t rs_bias = buffer_rsrc(g.bias, static_cast<uint32_t>(N) * 4);
  const int32x4_t rs_idx = buffer_rsrc(g.idx, static_cast<uint32_t>(g.n_max) * 4);
  const uint32_t side_base = ring_base + static_cast<uint32_t>(STAGES * Cfg::CHUNKS * 16);
  int parity = 0;
  auto bias_of = [&](const Unit& t, float4 (&bq)[FN][4]) {
    if (overlap) {
      if (wave_u == 0)
        lds_dma16(side_base + static_cast<uint32_t>(parity * 1024), static_cast<uint32_t>(t.n0 + 4 * lane) * 4, rs_bias);
      if (KIND == fdh::GEMM_QKV && wave_u == 1)
        lds_dma16(side_base + static_cast<uint32_t>(2048 + parity * 1024), static_cast<uint32_t>(t.m0 + 4 * lane) * 4, rs_idx);
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) bq[j][q] = make_float4(0.f, 0.f, 0.f, 0.f);
      return;
    }
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        bq[j][q] = t.split == 0 ? *reinterpret_cast<const float4*>(g.bias + min(t.n0 + wn * TN + 32 * j + 8 * q + 4 * lg, N - 4))
                                : make_float4(0.f, 0.f, 0.f, 0.f);
  };

  Unit cur;
  int u = blockIdx.x;
  if (!unit_at(u, cur)) return;
  uint32_t off[LOADS];
  offsets(cur, off);
  // this lane's output rows (one per 32-row block) and their token / request,
  // loaded before the K loop so that the epilogue never waits on them
  int rtok[FM], rreq[FM];
  if constexpr (!overlap) row_operands<FM, KIND>(g, M, cur.m0 + wm * TM + l32, rtok, rreq);
  float4 bq[FN][4];
  bias_of(cur, bq);
  prologue(cur, off);
  bool stores_in_flight = false;   // the previous unit's epilogue stores follow this unit's first stage
  for (;;) {
    f32x16_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[i][j][4 * q + 0] = bq[j][q].x;
          acc[i][j][4 * q + 1] = bq[j][q].y;
          acc[i][j][4 * q + 2] = bq[j][q].z;
          acc[i][j][4 * q + 3] = bq[j][q].w;
        }

    const int nkt = cur.nkt, kt0 = cur.kt0;
    for (int it = 0; it < nkt; ++it) {
      // exactly STAGES - 2 younger stages (and, in the first step, the previous
      // unit's epilogue stores) are in flight: stage `it` has landed for every wave
      if (kOverlap && it == 0 && stores_in_flight)
        wait_vm_barrier<(STAGES - 2) * LOADS + kEpiStores>();
      else
        wait_vm_barrier<(STAGES - 2) * LOADS>();
      // refill the slot every wave finished reading before this barrier (a repeat at the tail)
      const int kt_next = min(it + STAGES - 1, nkt - 1), st_next = (it + STAGES - 1) % STAGES;
      if constexpr (!Cfg::SPREAD) issue_q(off, kt0, kt_next, st_next, 0, LOADS);
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
          issue_q(off, kt0, kt_next, st_next, ks * LQ, (ks + 1) * LQ);
        }
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[ks & 1][j], a[ks & 1][i], acc[i][j], 0, 0, 0);
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

    const int row0 = cur.m0 + wm * TM + l32, cw = cur.n0 + wn * TN;
    Unit nxt;
    u += gridDim.x;
    const bool more = unit_at(u, nxt);
    if (S > 1) {
      // Store this split's fp32 tile for splitk_reduce_kernel (float4 r4 of block
      // (i, j) of thread t at float4 index ((i * FN + j) * 4 + r4) * THREADS + t).
      f32x4_t* slot = reinterpret_cast<f32x4_t*>(g.partial + static_cast<size_t>(cur.v) * (BM * BN)) + tid;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4)
            slot[((i * FN + j) * 4 + r4) * THREADS] =
                f32x4_t{acc[i][j][4 * r4], acc[i][j][4 * r4 + 1], acc[i][j][4 * r4 + 2], acc[i][j][4 * r4 + 3]};
    } else if constexpr (overlap) {
      // the next unit's copies go first; then every epilogue store issues
      const float* side = reinterpret_cast<const float*>(ring_mem + STAGES * Cfg::CHUNKS);
      const float* bias_lds = side + parity * 256 + wn * TN;
      const int* tok_lds = reinterpret_cast<const int*>(side + 512 + parity * 256) + wm * TM + l32;
      int tok[FM];
#pragma unroll
      for (int i = 0; i < FM; ++i) tok[i] = KIND == fdh::GEMM_QKV ? tok_lds[32 * i] : 0;
      if (more) {
        parity ^= 1;
        offsets(nxt, off);
        bias_of(nxt, bq);
        prologue(nxt, off);
      }
      float4* spare = reinterpret_cast<float4*>(g.partial) + tid;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          epilogue_block<KIND, true>(g, row0 + 32 * i < M, row0 + 32 * i, cw + 32 * j, lg, tok[i], acc[i][j], spare,
                                     bias_lds + 32 * j);
      if (!more) return;
      stores_in_flight = true;
      cur = nxt;
      continue;
    } else {
      tile_epilogue<FM, FN, KIND>(g, M, row0, cw, lg, rtok, rreq, acc);
    }
    if (!more) return;
    cur = nxt;
    offsets(cur, off);
    if constexpr (!overlap) row_operands<FM, KIND>(g, M, cur.m0 + wm * TM + l32, rtok, rreq);
    bias_of(cur, bq);
    prologue(cur, off);
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
  const int M = min(*g.m, g.n_max);
  if (M <= 0) return;
  switch (small_shape(M, g.N, g.K, slots, g.max_units)) {
    case 1: gemm_tiles<CfgWide, KIND>(g, slots, M, ring_mem); break;
    case 2: gemm_tiles<CfgNarrow, KIND>(g, slots, M, ring_mem); break;
    default: gemm_tiles<CfgSmall, KIND>(g, slots, M, ring_mem); break;
  }
}

template <int KIND>
__global__ __launch_bounds__(CfgLarge::THREADS, CfgLarge::OCC) void gemm_large_kernel(fdh::GemmArgs g, int slots) {
  __shared__ uint4 ring_mem[CfgLarge::STAGES * CfgLarge::CHUNKS + kSideChunks];   // ring + bias and token slots
  const int M = min(*g.m, g.n_max);
  if (M <= 0) return;
  gemm_tiles<CfgLarge, KIND>(g, slots, M, ring_mem);
}

// Split-K reduction: when the GEMM above split its 128x128 tiles (same M, shape and
// split count, recomputed here), the S partial tiles are summed in split order
// (deterministic) and the epilogue runs with the GEMM's thread geometry, one
// workgroup per (tile, 32x32 block of every wave): four per tile, so that each
// thread keeps all of its S partial loads in flight.  The kernel boundary orders
// the partial stores before these loads.
template <int KIND>
__global__ __launch_bounds__(CfgSmall::THREADS) void splitk_reduce_kernel(fdh::GemmArgs g, int slots) {
  using Cfg = CfgSmall;
  constexpr int FM = Cfg::FM, FN = Cfg::FN, NB = FM * FN, THREADS = Cfg::THREADS;
  const int M = min(*g.m, g.n_max);
  if (M <= 0) return;
  const int tiles_m = (M + Cfg::BM - 1) / Cfg::BM, tiles_n = (g.N + Cfg::BN - 1) / Cfg::BN;
  const int tiles = tiles_m * tiles_n;
  const int S = choose_split(tiles, g.K / TBK, slots, g.max_units);
  if (S == 1) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / Cfg::WN, wn = wave % Cfg::WN, l32 = lane & 31, lg = lane >> 5;
  for (int w = blockIdx.x; w < tiles * NB; w += gridDim.x) {
    const int tile = w / NB, bi = w - tile * NB, i = bi / FN, j = bi - (bi / FN) * FN;
    const int m0 = (tile % tiles_m) * Cfg::BM, n0 = (tile / tiles_m) * Cfg::BN;
    const int row0 = m0 + wm * Cfg::TM + 32 * i + l32;
    int rtok[1], rreq[1];
    row_operands<1, KIND>(g, M, row0, rtok, rreq);
    const f32x4_t* base = reinterpret_cast<const f32x4_t*>(g.partial + static_cast<size_t>(tile) * S * kSmallTile) +
                          static_cast<size_t>(bi * 4) * THREADS + tid;
    f32x16_t acc[1][1];
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[0][0][e] = 0.f;
    // four splits' loads at a time, summed in split order (the first add is onto 0)
    for (int s0 = 0; s0 < S; s0 += 4) {
      f32x4_t p[4][4];
#pragma unroll
      for (int sp = 0; sp < 4; ++sp)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
          p[sp][r4] = (s0 + sp < S) ? base[static_cast<size_t>(s0 + sp) * (kSmallTile / 4) + r4 * THREADS] : f32x4_t{};
#pragma unroll
      for (int sp = 0; sp < 4; ++sp)
        if (s0 + sp < S) {
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4)
            for (int e = 0; e < 4; ++e) acc[0][0][4 * r4 + e] += p[sp][r4][e];
        }
    }
    tile_epilogue<1, 1, KIND>(g, M, row0, n0 + wn * Cfg::TN + 32 * j, lg, rtok, rreq, acc);
  }
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
  return units * kSmallTile * sizeof(float);
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
  // the split-K reduction, launched whenever K is long enough for a split (it
  // returns at once when the device-side M gave S = 1)
  const bool may_split = !large && max_units > 0 && (a.K / TBK) >= 2 * kMinSplitSteps;
  const long long red_units = static_cast<long long>((a.n_max + 127) / 128) * ((a.N + 127) / 128) * CfgSmall::FM * CfgSmall::FN;
  const int red_grid = static_cast<int>(red_units < 4 * slots ? red_units : 4 * slots);
  switch (kind) {
    case GEMM_QKV: FD_GEMM_LAUNCH(GEMM_QKV) break;
    case GEMM_RESID: FD_GEMM_LAUNCH(GEMM_RESID) break;
    case GEMM_GELU: FD_GEMM_LAUNCH(GEMM_GELU) break;
    case GEMM_EMBED: FD_GEMM_LAUNCH(GEMM_EMBED) break;
    case GEMM_OUT: FD_GEMM_LAUNCH(GEMM_OUT) break;
  }
#undef FD_GEMM_LAUNCH
  if (may_split) {
    switch (kind) {
      case GEMM_QKV: splitk_reduce_kernel<GEMM_QKV><<<red_grid, CfgSmall::THREADS, 0, s>>>(g, slots); break;
      case GEMM_RESID: splitk_reduce_kernel<GEMM_RESID><<<red_grid, CfgSmall::THREADS, 0, s>>>(g, slots); break;
      case GEMM_GELU: splitk_reduce_kernel<GEMM_GELU><<<red_grid, CfgSmall::THREADS, 0, s>>>(g, slots); break;
      case GEMM_EMBED: splitk_reduce_kernel<GEMM_EMBED><<<red_grid, CfgSmall::THREADS, 0, s>>>(g, slots); break;
      case GEMM_OUT: splitk_reduce_kernel<GEMM_OUT><<<red_grid, CfgSmall::THREADS, 0, s>>>(g, slots); break;
    }
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_gemm(GemmKind kind, const GemmArgs& a, hipStream_t s) {
  if (a.K % TBK == 0) {
    const int max_units = a.partial ? a.max_units : 0;   // no scratch: never split
    if (a.n_max >= kLargeTileRows && a.N >= 1024) {
      // the bf16-output kinds send the stores of rows past M to a spare slot in the scratch
      if ((kind == GEMM_QKV || kind == GEMM_GELU) && !a.partial) return hipErrorInvalidValue;
      return launch_tiled(kind, a, 0, true, s);
    }
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
