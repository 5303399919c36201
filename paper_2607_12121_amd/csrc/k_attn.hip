// Attention of the active queries over every token of their request, K/V read
// from the per-block cache (fresh rows for active tokens, stale rows for skipped
// ones).  Flash-style with an fp32 online softmax (base-2 exponent); both
// contractions run on v_mfma_f32_32x32x16_bf16.
//
// Work item = (head, query tile of one request).  Head dim 64 and 128: one
// workgroup of 8 waves per CU (two per SIMD) works on 256 queries at a time, 32
// per wave; head dim 16: 4 waves, two workgroups per CU.  Each wave computes
// S^T = K Q^T (keys x queries), so a lane owns one query column: its running max
// needs one half-wave exchange per tile and its running sum none until the end;
// S^T feeds O^T = V^T P^T directly as the B operand.  Every head dim runs a
// software pipeline: the iteration of key tile t issues the MFMAs of S(t + 1) and
// of O += V P(t) as jobs between the element pairs of tile t's softmax, so one
// wave's softmax runs beside MFMAs of its own and of the other wave on the SIMD.
// (The code also supports two 32-query groups per wave sharing every K/V
// fragment read; one group measured faster once the loop is pipelined.)
//
// K and V tiles of 64 keys stream from HBM straight into LDS (buffer_load ...
// lds), both row-major in 16-byte chunks: head dim 128 in two-slot rings of their
// own (K two tiles ahead, V one), the others in one ring of K|V stages.  K rows are
// read as MFMA A fragments (16 consecutive keys, one chunk): chunk c of key row
// k sits at c ^ fk(k).  V^T is read with ds_read_b64_tr_b16: in a group of 16
// lanes, lane j addresses 4 consecutive d of key K0 + j/4 and every lane
// receives its own d for keys K0..K0+3, so V needs no transposing stores; one
// read covers 4 keys x 4 chunks per half-wave, placed at c ^ fv(k).  Both
// swizzles make every 16-lane (K) or 32-lane (V) read hit distinct banks.
//
// Schedule: the key tiles of all (head, query tile) items, head-major, form one
// range cut into equal contiguous shares, one per workgroup of the persistent grid;
// a share that ends inside an item leaves a piece of it to the next share.  Each
// piece of a cut item stores its O divided by its own sum (bf16), its max and its
// sum (fp32), and a second kernel merges the pieces in key order, each weighted by
// 2^(max - overall max) * sum (deterministic for a given grid); no workgroup
// waits for another.  Shares are dealt to the 8 XCDs in contiguous chunks so that
// the query tiles sharing a head's K/V run on the same L2.  Head dim 128 and
// launches without scratch for a partial per piece use runs of whole items.
#include <type_traits>

#include "fd_common.h"

namespace {

constexpr int kXcds = 8;
constexpr int KB = 64;                    // keys per tile
constexpr int kMaxThreads = 512;        // largest workgroup (the partial slots are per thread)
constexpr int kMaxQG = 2;

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef int int32x4_t __attribute__((ext_vector_type(4)));
typedef short short4_t __attribute__((ext_vector_type(4)));
using fd::bf16x2_t;

FD_DEVICE int32x4_t buffer_rsrc(const void* base) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  int32x4_t r;
  r.x = static_cast<int>(static_cast<uint32_t>(p));
  r.y = static_cast<int>(static_cast<uint32_t>(p >> 32) & 0xffffu);
  r.z = 0x7fffffff;
  r.w = 0x00020000;
  return r;
}

// 16 bytes per lane from buffer offset voff + soff (soff wave-uniform) into LDS at
// lds_addr + 16 * lane.
FD_DEVICE void lds_dma16(uint32_t lds_addr, uint32_t voff, int32x4_t rsrc, uint32_t soff = 0) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff));
}

template <int N>
FD_DEVICE void wait_vm_barrier() {
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" : : "n"(N) : "memory");
}

// max / sum of v over lanes l and l ^ 32 (v_permlane32_swap exchanges the halves)
FD_DEVICE float half_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
// NaN-propagating maximum (v_maximum3_f32 when nested): unlike fmaxf it needs no
// canonicalisation of MFMA results
FD_DEVICE float max3(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}
FD_DEVICE float half_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int DH>
struct ACfg {
  // 32-query groups per wave (two would share every K/V fragment read, half the LDS
  // reads per MFMA, but the pipeline's registers then leave one wave per SIMD, whose
  // softmax no other wave hides: measured slower)
  static constexpr int QG = 1;
  // Waves per workgroup.  Head dim 64 and 128: eight (two per SIMD) in one workgroup
  // per CU, so every K/V tile brought into LDS serves 256 queries (half the LDS
  // writes per query of two four-wave workgroups; video attention -8%, image -9%);
  // head dim 16: four, two workgroups per CU.
  static constexpr int WAVES = DH >= 64 ? 8 : 4;
  static constexpr int THREADS = WAVES * 64;
  static constexpr int QB = WAVES * QG * 32;            // queries per unit
  static constexpr int KCH = DH / 8;                    // 16-byte chunks per key row
  static constexpr int TILE = KB * KCH;                 // chunks of one K or V tile
  static constexpr int STAGE = 2 * TILE;                // K tile then V tile
  // Software pipeline: S of tile t + 1 next to the softmax of tile t.  Head dim <= 64:
  // a ring of four K|V stages.  Head dim 128: K and V in two-slot rings of their own
  // (K two tiles ahead, V one), 64 KB, so that two workgroups share a CU.
  static constexpr bool PIPE = true;
  static constexpr bool SPLIT = DH >= 128;
  static constexpr int RING = 2;                         // slots of each split ring (3: modulo spills; 4: equal to 2)
  static constexpr int STAGES = SPLIT ? RING : 4;        // ring memory: STAGES x (K tile + V tile)
  static constexpr int LOADS = STAGE / 64 / WAVES;      // 1 KB wave-loads per wave per stage
  static constexpr int KS = DH / 16;                    // k16 steps of S^T over d
  static constexpr int DT = (DH + 31) / 32;             // 32-row tiles of O^T
  static constexpr int OCC = 8 / WAVES;                 // workgroups per CU
  static constexpr int WPE = WAVES * OCC / 4;           // waves per SIMD
  static_assert(THREADS <= kMaxThreads, "partial slots sized for kMaxThreads");
  static_assert(STAGE % (64 * WAVES) == 0, "stage must split into whole wave-loads");
  // split rings: the first half of a wave's loads fetch K blocks, the second half V blocks
  static_assert(!SPLIT || (LOADS % 2 == 0 && TILE / 64 == WAVES * LOADS / 2), "K/V halves of the wave-loads");
  // K: 16 consecutive rows at one chunk -> distinct 16-byte bank groups
  static constexpr __host__ __device__ int fk(int r) {
    return KCH >= 16 ? (r & 15) : KCH == 8 ? ((r >> 1) & 7) : ((r >> 3) & (KCH - 1));
  }
  // V: 4 consecutive rows x one aligned block of 4 chunks -> distinct bank groups
  static constexpr __host__ __device__ int fv(int r) { return KCH >= 16 ? 4 * (r & 3) : KCH == 8 ? 4 * ((r >> 1) & 1) : 0; }
  // the read addressing folds these into per-lane bases plus constants: fk is the
  // same for key l and l + 32, fv the same for keys k, k + 8 and k + 16 st (k < 8)
  static constexpr bool swizzle_folds() {
    for (int r = 0; r < 32; ++r)
      if (fk(r) != fk(r + 32)) return false;
    for (int k = 0; k < 8; ++k)
      for (int st = 0; st < 4; ++st)
        if (fv(k + 16 * st) != fv(k) || fv(k + 16 * st + 8) != fv(k)) return false;
    return true;
  }
  static_assert(swizzle_folds(), "swizzle must fold into constant offsets");
};

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
FD_DEVICE bf16x8_t lds_read16(uint32_t addr) {
  return __builtin_bit_cast(bf16x8_t, *(__attribute__((address_space(3))) const u32x4_t*)(uintptr_t)addr);
}

constexpr int kMaxSchedRequests = fdh::kMaxAttnRequests;
// Up to this many requests the merge pass walks them instead of building the
// tables (a kernel of its own, without the tables' LDS): most of its workgroups
// only look up their share and exit, and for a handful of requests the walk
// costs less than the table build and its barriers.
constexpr int kWalkRequests = 16;

// Per-request prefix tables of the schedule, built once per workgroup: wpre[b] =
// tile-steps (query tiles x key tiles, one head) of the requests before b, tpre[b]
// = their query tiles; entry B holds the totals.
struct SchedTables {
  long long wpre[kMaxSchedRequests + 1];
  int tpre[kMaxSchedRequests + 1];
};

// One exclusive scan over the requests: each thread sums a contiguous run of them,
// the runs' sums are scanned within each wave (shuffles) and across the waves
// (LDS), and each thread then writes its run's prefixes.  O(B / threads + log)
// steps per workgroup instead of a walk over every request.
template <int THREADS>
FD_DEVICE void build_sched_tables(SchedTables& t, const int32_t* __restrict__ cu_q,
                                  const int32_t* __restrict__ req_tok_off, int B, int QB) {
  constexpr int NW = THREADS / 64;
  __shared__ long long s_w[NW];
  __shared__ int s_t[NW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int per = (B + THREADS - 1) / THREADS;
  const int b0 = min(tid * per, B), b1 = min(b0 + per, B);
  auto tiles_of = [&](int b) { return (cu_q[b + 1] - cu_q[b] + QB - 1) / QB; };
  auto keys_of = [&](int b) { return (req_tok_off[b + 1] - req_tok_off[b] + KB - 1) / KB; };
  int st = 0;
  long long sw = 0;
  for (int b = b0; b < b1; ++b) {
    const int nt = tiles_of(b);
    st += nt;
    sw += static_cast<long long>(nt) * keys_of(b);
  }
  int it = st;
  long long iw = sw;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int yt = __shfl_up(it, o, 64);
    const long long yw = __shfl_up(iw, o, 64);
    if (lane >= o) {
      it += yt;
      iw += yw;
    }
  }
  if (lane == 63) {
    s_t[wave] = it;
    s_w[wave] = iw;
  }
  __syncthreads();
  int pt = it - st;
  long long pw = iw - sw;
  for (int w = 0; w < wave; ++w) {
    pt += s_t[w];
    pw += s_w[w];
  }
  for (int b = b0; b < b1; ++b) {
    t.tpre[b] = pt;
    t.wpre[b] = pw;
    const int nt = tiles_of(b);
    pt += nt;
    pw += static_cast<long long>(nt) * keys_of(b);
  }
  if (b0 < b1 && b1 == B) {
    t.tpre[B] = pt;
    t.wpre[B] = pw;
  }
  __syncthreads();
}

// A wave-uniform value read from LDS, moved to a scalar register so that the loop
// bounds and branches derived from it stay scalar.
FD_DEVICE int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }
FD_DEVICE long long uniform(long long v) {
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(v)));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(v >> 32)));
  return static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Schedule: the key tiles of every item, items head-major, form one range of
// `work` tile-steps cut into G contiguous shares, one per workgroup, numbered so
// that each XCD gets consecutive shares (the query tiles of a head share its K/V
// in that XCD's L2).  With cuts the shares are equal: a share covers the end of
// one item, whole items and the start of another, and an item covered by
// several shares is a cut item whose pieces attn_combine_kernel merges.  A share
// w holds at most two pieces of cut items: the continuation of an item begun in
// an earlier share (scratch slot 2w) and the first piece of an item that goes on
// into later shares (slot 2w + 1; when that item starts at the share's start
// there is no continuation and slot 2w stays unused).  Without cuts every share
// boundary is rounded up to the next item start.  Requests are found by binary
// search in the workgroup's prefix tables.
template <int QB, bool TABLES>
struct AttnSched {
  const SchedTables* t;         // TABLES: the workgroup's prefix tables
  const int32_t* cu_q;          // else the requests are walked
  const int32_t* req_tok_off;
  int B, G;
  int tiles;              // query tiles over all requests
  long long work_head;    // tile-steps of one head (key tiles summed over every query tile)
  long long work;         // ... of every head
  bool cut;

  FD_DEVICE AttnSched(const SchedTables* tab, const int32_t* cq, const int32_t* rto, int B_, int H, int G_,
                      int max_units)
      : t(tab), cu_q(cq), req_tok_off(rto), B(B_), G(G_), tiles(0), work_head(0) {
    if constexpr (TABLES) {
      tiles = uniform(t->tpre[B]);
      work_head = uniform(t->wpre[B]);
    } else {
      for (int b = 0; b < B; ++b) {
        const int nt = (cu_q[b + 1] - cu_q[b] + QB - 1) / QB;
        tiles += nt;
        work_head += static_cast<long long>(nt) * ((req_tok_off[b + 1] - req_tok_off[b] + KB - 1) / KB);
      }
    }
    work = work_head * H;
    // Shares may cut items when the scratch holds two partials per share and
    // every share gets a tile-step; otherwise every share is a run of whole items.
    cut = max_units >= 2 * G && work >= static_cast<long long>(G) && G % kXcds == 0;
  }
  // the share run by workgroup `blk`
  FD_DEVICE int share(int blk) const { return (G % kXcds == 0) ? (blk % kXcds) * (G / kXcds) + blk / kXcds : blk; }
  // tile-step q < work: its item's first tile-step and key tiles, head, request,
  // the request's first query tile and the query tile
  FD_DEVICE void locate(long long q, long long& i_start, int& nkv, int& head, int& b, int& first, int& tau) const {
    head = static_cast<int>(q / work_head);
    long long r = q - static_cast<long long>(head) * work_head;
    if constexpr (!TABLES) {   // few requests: walk them (requests without tile-steps are passed over)
      b = 0;
      first = 0;
      nkv = 1;
      for (; b < B; ++b) {
        const int nt = (cu_q[b + 1] - cu_q[b] + QB - 1) / QB;
        nkv = (req_tok_off[b + 1] - req_tok_off[b] + KB - 1) / KB;
        const long long span = static_cast<long long>(nt) * nkv;
        if (r < span) break;
        r -= span;
        first += nt;
      }
      tau = first + static_cast<int>(r / nkv);
      i_start = q - r % nkv;
      return;
    }
    // the request: the largest b < B with wpre[b] <= r, which has tile-steps
    // (wpre[b + 1] > r); requests without any are passed over
    int lo = 0, hi = B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (uniform(t->wpre[mid]) <= r) lo = mid; else hi = mid - 1;
    }
    b = lo;
    first = uniform(t->tpre[b]);
    const int nt = uniform(t->tpre[b + 1]) - first;
    const long long w0 = uniform(t->wpre[b]);
    nkv = static_cast<int>((uniform(t->wpre[b + 1]) - w0) / nt);
    r -= w0;
    tau = first + static_cast<int>(r / nkv);
    i_start = q - r % nkv;
  }
  FD_DEVICE long long bound(long long x) const {   // first tile-step of share x (x <= G)
    const long long q = x * work / G;
    if (cut || q >= work) return q;
    long long i_start;
    int nkv, head, b, first, tau;
    locate(q, i_start, nkv, head, b, first, tau);
    return i_start == q ? q : i_start + nkv;
  }
  FD_DEVICE int share_of(long long q) const {   // the share holding tile-step q
    int x = static_cast<int>(q * G / work);
    while (x + 1 < G && bound(x + 1) <= q) ++x;
    return x;
  }
  // scratch slot of piece j of a cut item whose first piece is in share f
  FD_DEVICE static int slot_of(int f, int j) { return j == 0 ? 2 * f + 1 : 2 * (f + j); }
};

// Normalised O^T block rows of one 32-query group to bf16 O (row qrow, head
// columns col0 ...) and the query's base-2 log-sum-exp of the scaled scores
// (softmax = exp2(s * scale_log2 - lse)); lane (l32, lg) holds query l32 and, in
// register 4 r4 + e of block dt, d = 32 dt + 8 r4 + 4 lg + e.
template <int DH>
FD_DEVICE void store_o(uint16_t* __restrict__ O, float* __restrict__ lse, int D, int H, int head, int qrow, int lg,
                       const f32x16_t (&oacc)[ACfg<DH>::DT], float m, float l) {
  if (lse && lg == 0) lse[static_cast<size_t>(qrow) * H + head] = m + __log2f(l);
  const float inv_l = 1.0f / l;
  uint16_t* orow = O + static_cast<size_t>(qrow) * D + static_cast<size_t>(head) * DH;
#pragma unroll
  for (int dt = 0; dt < ACfg<DH>::DT; ++dt)
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

template <int DH>
__global__ __launch_bounds__(ACfg<DH>::THREADS) __attribute__((amdgpu_waves_per_eu(ACfg<DH>::WPE, ACfg<DH>::WPE))) void attn_fwd_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc, const uint16_t* __restrict__ Vc,
    uint16_t* __restrict__ O, int D, int H, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ req_tok_off,
    int B, float scale_log2, float* __restrict__ partial, int max_units, float* __restrict__ lse) {
  using C = ACfg<DH>;
  constexpr int DT = C::DT, KS = C::KS, KCH = C::KCH, STAGES = C::STAGES, LOADS = C::LOADS, QG = C::QG, QB = C::QB;
  __shared__ uint4 ring[STAGES][C::STAGE];
  __shared__ SchedTables tabs;

  build_sched_tables<C::THREADS>(tabs, cu_q, req_tok_off, B, QB);
  const AttnSched<QB, true> sch(&tabs, cu_q, req_tok_off, B, H, static_cast<int>(gridDim.x), max_units);
  if (sch.tiles == 0) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, lg = lane >> 5;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  // waves w and w + WAVES/2 share a SIMD: the second one issues first when both
  // are ready, so the pair drifts apart instead of contending for the same pipe
  // at the same time (image -2%, video -1%)
  if (wave_u >= C::WAVES / 2) __builtin_amdgcn_s_setprio(1);
  const int32x4_t rs_k = buffer_rsrc(Kc);
  const int32x4_t rs_v = buffer_rsrc(Vc);
  const uint32_t ring_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)&ring[0][0]));

  // V^T operand addressing for ds_read_b64_tr_b16 (see file comment)
  const int grp = lane >> 4, jj = lane & 15;
  const int tr_key = 4 * lg + (jj >> 2);                 // + 16 * st + 8 * half
  const int tr_d = 16 * (grp & 1) + 4 * (jj & 3);       // + 32 * dt
  const bool tr_live = (DH >= 32) || (grp & 1) == 0;    // rows d >= DH are zero operand rows
  // per-lane LDS byte offsets inside a tile: K fragment of k16 step ks (key l32), V^T
  // fragment of 32-row block dt (keys tr_key + 16 st (+ 8)); the swizzles of those keys
  // do not depend on the half, st or the +8 (checked below)
  uint32_t k_off[ACfg<DH>::KS], v_off[ACfg<DH>::DT];
#pragma unroll
  for (int ks = 0; ks < ACfg<DH>::KS; ++ks)
    k_off[ks] = static_cast<uint32_t>((l32 * ACfg<DH>::KCH + ((ks * 2 + lg) ^ ACfg<DH>::fk(l32))) * 16);
#pragma unroll
  for (int dt = 0; dt < ACfg<DH>::DT; ++dt) {
    const int d_s = dt * 32 + tr_d;
    v_off[dt] = static_cast<uint32_t>(tr_key * ACfg<DH>::KCH * 16 + ((d_s >> 3) ^ ACfg<DH>::fv(tr_key)) * 16 + (d_s & 7) * 2);
  }

  // One piece of work: key tiles [kt0, kt1) of query tile tau (of request b, whose
  // first query tile is number `first`) under head `head`; piece `piece` of the
  // `npieces` that cover this (head, tile) item in key order, the first of them in
  // share `share0`.
  auto run_piece = [&](const int head, const int tau, const int b, const int first, const int kt0, const int kt1,
                       const int piece, const int npieces, const int share0) {
    const int q_lo = cu_q[b] + (tau - first) * QB;
    const int q_hi = cu_q[b + 1];
    const int k_beg = req_tok_off[b], k_end = req_tok_off[b + 1];
    const int nkt = kt1 - kt0;
    const size_t col0 = static_cast<size_t>(head) * DH;
    const uint32_t col2 = static_cast<uint32_t>(col0 * 2);

    bf16x8_t qf[QG][KS];
#pragma unroll
    for (int g = 0; g < QG; ++g) {
      const int qrow = q_lo + wave * (32 * QG) + g * 32 + l32;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        uint4 t = make_uint4(0, 0, 0, 0);
        if (qrow < q_hi) t = *reinterpret_cast<const uint4*>(Q + static_cast<size_t>(qrow) * D + col0 + ks * 16 + lg * 8);
        qf[g][ks] = __builtin_bit_cast(bf16x8_t, t);
      }
    }

    // DMA of one stage: wave-load q covers 64 consecutive chunks (RPL rows) of the K|V
    // stage.  A tile whose keys all lie inside the request adds a wave-uniform byte
    // offset to per-lane offsets fixed for the unit; only a ragged last tile clamps
    // its rows per lane.
    constexpr int RPL = 64 / KCH, TILE_BLKS = C::TILE / 64;
    const int n_full = (k_end - k_beg) / KB;
    uint32_t dma_off[LOADS];
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int blk = wave + C::WAVES * q;
      const bool is_v = blk >= TILE_BLKS;
      const int r = (blk - (is_v ? TILE_BLKS : 0)) * RPL + lane / KCH;   // key row within the tile
      const int c = (lane % KCH) ^ (is_v ? C::fv(r) : C::fk(r));
      dma_off[q] = static_cast<uint32_t>(k_beg + r) * static_cast<uint32_t>(2 * D) + col2 + static_cast<uint32_t>(c * 16);
    }
    // wave-loads q in [Q0, Q1) of key tile kt (global index): K blocks to kbuf, V
    // blocks to vbuf, 1 KB per block
    auto issue_q = [&](int kt, uint32_t kbuf, uint32_t vbuf, auto q0_tag, auto q1_tag) {
      constexpr int Q0 = decltype(q0_tag)::value, Q1 = decltype(q1_tag)::value;
      if (kt < n_full) {
        const uint32_t soff = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(kt * KB * 2 * D));
#pragma unroll
        for (int q = Q0; q < Q1; ++q) {
          const int blk = wave_u + C::WAVES * q;            // wave-uniform
          const bool is_v = blk >= TILE_BLKS;
          const uint32_t dst = is_v ? vbuf + static_cast<uint32_t>((blk - TILE_BLKS) * 64 * 16)
                                    : kbuf + static_cast<uint32_t>(blk * 64 * 16);
          lds_dma16(dst, dma_off[q], is_v ? rs_v : rs_k, soff);
        }
      } else {
        const int k0 = k_beg + kt * KB;
#pragma unroll
        for (int q = Q0; q < Q1; ++q) {
          const int blk = wave_u + C::WAVES * q;            // wave-uniform
          const bool is_v = blk >= TILE_BLKS;
          const int r = (blk - (is_v ? TILE_BLKS : 0)) * RPL + lane / KCH;
          const int c = (lane % KCH) ^ (is_v ? C::fv(r) : C::fk(r));
          const int key = min(k0 + r, k_end - 1);
          const uint32_t off = static_cast<uint32_t>(key) * static_cast<uint32_t>(2 * D) + col2 + static_cast<uint32_t>(c * 16);
          const uint32_t dst = is_v ? vbuf + static_cast<uint32_t>((blk - TILE_BLKS) * 64 * 16)
                                    : kbuf + static_cast<uint32_t>(blk * 64 * 16);
          lds_dma16(dst, off, is_v ? rs_v : rs_k);
        }
      }
    };
    using IQ0 = std::integral_constant<int, 0>;
    using IQH = std::integral_constant<int, LOADS / 2>;
    using IQL = std::integral_constant<int, LOADS>;
    // LDS byte address of local key tile t's K and V
    auto k_addr = [&](int t) -> uint32_t {
      return C::SPLIT ? ring_base + static_cast<uint32_t>((t % C::RING) * C::TILE * 16)
                      : ring_base + static_cast<uint32_t>((t % STAGES) * C::STAGE * 16);
    };
    auto v_addr = [&](int t) -> uint32_t {
      return C::SPLIT ? ring_base + static_cast<uint32_t>((C::RING + t % C::RING) * C::TILE * 16)
                      : ring_base + static_cast<uint32_t>(((t % STAGES) * C::STAGE + C::TILE) * 16);
    };
    // combined ring: key tile kt into stage st; split rings: K or V of local tile t
    auto issue = [&](int kt, int st) {
      const uint32_t buf = ring_base + static_cast<uint32_t>(st * C::STAGE * 16);
      issue_q(kt, buf, buf + static_cast<uint32_t>(C::TILE * 16), IQ0{}, IQL{});
    };
    auto issue_k = [&](int t) { issue_q(kt0 + min(t, nkt - 1), k_addr(t), 0u, IQ0{}, IQH{}); };
    auto issue_v = [&](int t) { issue_q(kt0 + min(t, nkt - 1), 0u, v_addr(t), IQH{}, IQL{}); };

    f32x16_t oacc[QG][DT];
#pragma unroll
    for (int g = 0; g < QG; ++g)
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[g][d][r] = 0.f;
    float m_run[QG], l_run[QG];
#pragma unroll
    for (int g = 0; g < QG; ++g) {
      m_run[g] = -INFINITY;
      l_run[g] = 0.f;
    }
    typedef f32x16_t SAcc[QG][2];
    typedef bf16x8_t PAcc[QG][4];

    // S^T (64 keys x 32 queries per group) of tile t = K Q^T; each K fragment feeds every group
    auto s_tile = [&](int t, SAcc& sacc, auto ks_lo_tag, auto ks_hi_tag) {
      constexpr int KS_LO = decltype(ks_lo_tag)::value, KS_HI = decltype(ks_hi_tag)::value;
      const uint32_t kt_addr = k_addr(t);
      const f32x16_t zero = {};
#pragma unroll
      for (int ks = KS_LO; ks < KS_HI; ++ks)
#pragma unroll
        for (int kh = 0; kh < 2; ++kh) {
          // fk(l32 + 32 kh) = fk(l32): the half is a constant offset
          const bf16x8_t a = lds_read16(kt_addr + k_off[ks] + static_cast<uint32_t>(kh * 32 * KCH * 16));
#pragma unroll
          for (int g = 0; g < QG; ++g)   // the first k16 step starts from the constant zero accumulator
            sacc[g][kh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[g][ks], ks == 0 ? zero : sacc[g][kh], 0, 0, 0);
        }
    };

    // Online softmax of tile t, part 1: running max and (rarely) the rescale of O.
    // MASK: the tile holds keys past the request end (scores -inf).
    auto softmax_max = [&](int t, SAcc& sacc, float (&m_new)[QG], auto mask_tag) {
      constexpr bool MASK = decltype(mask_tag)::value;
      if constexpr (MASK) {
        const int lim = k_end - (k_beg + (kt0 + t) * KB) - 4 * lg;   // this lane's keys below lim are valid
#pragma unroll
        for (int g = 0; g < QG; ++g)
#pragma unroll
          for (int kh = 0; kh < 2; ++kh)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              if (kh * 32 + 8 * (r >> 2) + (r & 3) >= lim) sacc[g][kh][r] = -INFINITY;
      }
#pragma unroll
      for (int g = 0; g < QG; ++g) {
        // four independent max3 chains over the 32 scores of this lane
        float mx[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int kh = c >> 1, r0 = 8 * (c & 1);
          mx[c] = __builtin_elementwise_maximum(sacc[g][kh][r0], sacc[g][kh][r0 + 1]);
#pragma unroll
          for (int r = r0 + 2; r < r0 + 8; r += 2) mx[c] = max3(mx[c], sacc[g][kh][r], sacc[g][kh][r + 1]);
        }
        const float m_tile = half_max(__builtin_elementwise_maximum(__builtin_elementwise_maximum(mx[0], mx[1]),
                                                                   __builtin_elementwise_maximum(mx[2], mx[3]))) *
                             scale_log2;
        // Lazy rescaling: the subtracted max only moves when the tile max exceeds it by
        // more than 8 (P <= 2^8 otherwise); softmax does not depend on that constant.
        const bool grow = m_tile > m_run[g] + 8.0f;
        m_new[g] = grow ? m_tile : m_run[g];
        if (__any(grow)) {
          const float alpha = __builtin_amdgcn_exp2f(m_run[g] - m_new[g]);
          l_run[g] *= alpha;
#pragma unroll
          for (int d = 0; d < DT; ++d)
#pragma unroll
            for (int r = 0; r < 16; ++r) oacc[g][d][r] *= alpha;
        }
        m_run[g] = m_new[g];
      }
    };
    // part 2: P = exp2(S scale - m) packed to bf16 pairs (the B operand of O^T), row sums
    auto softmax_p = [&](SAcc& sacc, PAcc& pk, const float (&m_new)[QG]) {
#pragma unroll
      for (int g = 0; g < QG; ++g) {
        float lsum = 0.f;
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            bf16x8_t pv;
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
              const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[g][kh][half * 8 + e], scale_log2, -m_new[g]));
              const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[g][kh][half * 8 + e + 1], scale_log2, -m_new[g]));
              const fd::f32x2_t f = {p0, p1};
              const bf16x2_t pb = __builtin_convertvector(f, bf16x2_t);
              // the row sum is taken over the rounded P that the PV product uses
              lsum = __builtin_amdgcn_fdot2_f32_bf16(pb, bf16x2_t{(__bf16)1.0f, (__bf16)1.0f}, lsum, false);
              pv[e] = pb[0];
              pv[e + 1] = pb[1];
            }
            pk[g][kh * 2 + half] = pv;
          }
        l_run[g] += lsum;
      }
    };

    // O^T (d x 32 queries) += V^T P^T for tile t; k-step st covers keys 16 st .. 16 st + 15
    auto pv_tile = [&](int t, PAcc& pk) {
      const uint32_t vt_addr = v_addr(t);
#pragma unroll
      for (int st = 0; st < 4; ++st) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          short4_t lo = {0, 0, 0, 0}, hi = {0, 0, 0, 0};
          if (tr_live) {
            // fv(key) is the same for keys 16 st + tr_key and that + 8: st and hi are constant offsets
            const uint32_t a_lo = vt_addr + v_off[dt] + static_cast<uint32_t>(16 * st * KCH * 16);
            const uint32_t a_hi = a_lo + static_cast<uint32_t>(8 * KCH * 16);
            lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)(uintptr_t)a_lo);
            hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)(uintptr_t)a_hi);
          }
          const short lo_hi[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          bf16x8_t av;
#pragma unroll
          for (int e = 0; e < 8; ++e) av[e] = __builtin_bit_cast(__bf16, lo_hi[e]);
#pragma unroll
          for (int g = 0; g < QG; ++g) oacc[g][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pk[g][st], oacc[g][dt], 0, 0, 0);
        }
      }
    };

    // Software pipeline over the key tiles: iteration t computes S of tile t + 1 on
    // the MFMA pipe while the VALU runs the softmax of tile t, then O += V P of tile
    // t.  The ring: stages are issued STAGES - 1 ahead (re-issued at the tail so the
    // wait count is constant); iteration t refills the slot of tile t - 1, which
    // every wave finished before the iteration's barrier.
    constexpr int AHEAD_WAIT = C::PIPE ? (STAGES - 3) * LOADS : 0;   // younger loads allowed while tile t + 1 must have landed
    SAcc sa, sb;
    PAcc pk;
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using IK = std::integral_constant<int, KS>;
    const bool ragged = (k_beg + kt1 * KB > k_end);   // only the piece's last tile can hold keys past the end
    auto body = [&](int t, SAcc& cur, SAcc& nxt) {
      if constexpr (C::SPLIT) {
        // K of tile t + 1 and V of tile t (issued RING - 1 iterations ago) have landed,
        // and every wave is done with K of tile t and V of tile t - 1, whose slots refill
        wait_vm_barrier<(C::RING - 2) * LOADS>();
        issue_k(t + C::RING);
        issue_v(t + C::RING - 1);
      } else {
        wait_vm_barrier<AHEAD_WAIT>();
        issue(kt0 + min(t + STAGES - 1, nkt - 1), (t + STAGES - 1) % STAGES);
      }
      float m_new[QG];
      s_tile(t + 1, nxt, I0{}, I1{});
      softmax_max(t, cur, m_new, std::integral_constant<bool, false>{});
      {
        // Hand-interleaved block: the P math of tile t (16 element pairs per query
        // group, quarter-major: quarter st of every group before quarter st + 1) with
        // MFMA jobs after each pair: first the rest of S(t + 1), then PV(t) per 16-key
        // step once that quarter of P exists in every group.  A job is one LDS operand
        // read feeding the MFMAs of all QG groups.  The order is pinned per pair.
        const uint32_t kt_addr = k_addr(t + 1);
        const uint32_t vt_addr = v_addr(t);
        constexpr int NS = (KS - 1) * 2, NP = DT * 4, NJ = NS + NP;
        constexpr int NPAIR = 16 * QG;
        constexpr int PER = (NJ + NPAIR - 1) / NPAIR;
        // job j = its LDS operand read (fetch) and its MFMAs (run); reads run two jobs ahead
        auto fetch = [&](int j) -> u32x4_t {
          if (j < NS) {
            const int ks = 1 + j / 2, kh = j % 2;
            return __builtin_bit_cast(u32x4_t, lds_read16(kt_addr + k_off[ks] + static_cast<uint32_t>(kh * 32 * KCH * 16)));
          }
          const int st = (j - NS) / DT, dt = (j - NS) % DT;
          short4_t lo = {0, 0, 0, 0}, hi = {0, 0, 0, 0};
          if (tr_live) {
            const uint32_t a_lo = vt_addr + v_off[dt] + static_cast<uint32_t>(16 * st * KCH * 16);
            const uint32_t a_hi = a_lo + static_cast<uint32_t>(8 * KCH * 16);
            lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)(uintptr_t)a_lo);
            hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)(uintptr_t)a_hi);
          }
          const short lo_hi[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          return __builtin_bit_cast(u32x4_t, lo_hi);
        };
        auto run = [&](int j, u32x4_t op) {
          const bf16x8_t a = __builtin_bit_cast(bf16x8_t, op);
          if (j < NS) {
            const int ks = 1 + j / 2, kh = j % 2;
#pragma unroll
            for (int g = 0; g < QG; ++g)
              nxt[g][kh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[g][ks], nxt[g][kh], 0, 0, 0);
          } else {
            const int st = (j - NS) / DT, dt = (j - NS) % DT;
#pragma unroll
            for (int g = 0; g < QG; ++g)
              oacc[g][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pk[g][st], oacc[g][dt], 0, 0, 0);
          }
        };
        // earliest pair after which job j may run: S jobs at once, PV(st) after the last
        // pair of quarter st
        auto earliest = [&](int j) { return j < NS ? 0 : 4 * QG * ((j - NS) / DT + 1) - 1; };
        float lsum[QG][4];   // four independent chains of row-sum dot products
#pragma unroll
        for (int g = 0; g < QG; ++g)
#pragma unroll
          for (int c = 0; c < 4; ++c) lsum[g][c] = 0.f;
        int cursor = 0;
        u32x4_t op0 = fetch(0), op1 = fetch(1);   // operands of jobs cursor and cursor + 1
        auto next_job = [&]() {
          const u32x4_t op2 = cursor + 2 < NJ ? fetch(cursor + 2) : op1;
          run(cursor++, op0);
          op0 = op1;
          op1 = op2;
        };
#pragma unroll
        for (int pp = 0; pp < NPAIR; ++pp) {
          const int st = pp / (4 * QG), g = (pp / 4) % QG, e = 2 * (pp % 4);
          const int kh = st / 2, half = st % 2;
          const float p0 = __builtin_amdgcn_exp2f(fmaf(cur[g][kh][half * 8 + e], scale_log2, -m_new[g]));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(cur[g][kh][half * 8 + e + 1], scale_log2, -m_new[g]));
          const fd::f32x2_t f = {p0, p1};
          const bf16x2_t pb = __builtin_convertvector(f, bf16x2_t);
          lsum[g][pp % 4] = __builtin_amdgcn_fdot2_f32_bf16(pb, bf16x2_t{(__bf16)1.0f, (__bf16)1.0f}, lsum[g][pp % 4], false);
          pk[g][st][e] = pb[0];
          pk[g][st][e + 1] = pb[1];
#pragma unroll
          for (int k = 0; k < PER; ++k)
            if (cursor < NJ && earliest(cursor) <= pp) next_job();
          __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int k = 0; k < NJ; ++k)
          if (cursor < NJ) next_job();
#pragma unroll
        for (int g = 0; g < QG; ++g) l_run[g] += (lsum[g][0] + lsum[g][1]) + (lsum[g][2] + lsum[g][3]);
      }
    };
    auto tail = [&](int t, SAcc& cur, bool masked) {
      if constexpr (C::SPLIT) wait_vm_barrier<(C::RING - 2) * LOADS>();   // V of tile t has landed
      float m_new[QG];
      if (masked)
        softmax_max(t, cur, m_new, std::integral_constant<bool, true>{});
      else
        softmax_max(t, cur, m_new, std::integral_constant<bool, false>{});
      softmax_p(cur, pk, m_new);
      pv_tile(t, pk);
    };
    if constexpr (C::PIPE) {
      if constexpr (C::SPLIT) {
#pragma unroll
        for (int p = 0; p + 1 < C::RING; ++p) {
          issue_k(p);
          issue_v(p);
        }
        issue_k(C::RING - 1);
        wait_vm_barrier<(C::RING - 1) * LOADS>();   // K of tile 0 has landed
      } else {
#pragma unroll
        for (int p = 0; p < STAGES - 1; ++p) issue(kt0 + min(p, nkt - 1), p);
        wait_vm_barrier<(STAGES - 2) * LOADS>();
      }
      s_tile(0, sa, I0{}, IK{});
      int t = 0;
      for (; t + 2 <= nkt - 1; t += 2) {
        body(t, sa, sb);
        body(t + 1, sb, sa);
      }
      if (t < nkt - 1) {
        body(t, sa, sb);
        tail(t + 1, sb, ragged);
      } else {
        tail(t, sa, ragged);
      }
    } else {
      // plain loop: the ring is issued STAGES - 1 ahead, tile t is complete after the wait
      issue(kt0, 0);
      const int n_plain = ragged ? nkt - 1 : nkt;
      for (int t = 0; t < n_plain; ++t) {
        wait_vm_barrier<0>();
        issue(kt0 + min(t + 1, nkt - 1), (t + 1) % STAGES);
        s_tile(t, sa, I0{}, IK{});
        float m_new[QG];
        softmax_max(t, sa, m_new, std::integral_constant<bool, false>{});
        softmax_p(sa, pk, m_new);
        pv_tile(t, pk);
      }
      if (ragged) {   // the masked last tile, outside the loop
        wait_vm_barrier<0>();
        s_tile(nkt - 1, sa, I0{}, IK{});
        float m_new[QG];
        softmax_max(nkt - 1, sa, m_new, std::integral_constant<bool, true>{});
        softmax_p(sa, pk, m_new);
        pv_tile(nkt - 1, pk);
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();   // the ring is refilled by the next unit
#pragma unroll
    for (int g = 0; g < QG; ++g) l_run[g] = half_sum(l_run[g]);

    if (npieces > 1) {
      // a piece of a cut item: O / sum rounded to bf16 (a convex combination of V
      // rows, so bf16 keeps its range) and (max, sum) in fp32 for
      // attn_combine_kernel, lane-major (the four bf16 of quad q of thread t at
      // 8-byte word q * THREADS + t, then, past the slot's O area, the (max, sum)
      // pair of group g at float2 g * THREADS + t)
      constexpr int E = QG * (DT * 16 + 2);
      float* slot = partial + static_cast<size_t>(AttnSched<QB, true>::slot_of(share0, piece)) * (E * C::THREADS);
      uint2* quads = reinterpret_cast<uint2*>(slot) + tid;
      fd::f32x2_t* ml = reinterpret_cast<fd::f32x2_t*>(slot + QG * DT * 16 * C::THREADS) + tid;
#pragma unroll
      for (int g = 0; g < QG; ++g) {
        const float inv = l_run[g] > 0.f ? 1.0f / l_run[g] : 0.f;
#pragma unroll
        for (int d = 0; d < DT; ++d)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4)
            quads[((g * DT + d) * 4 + r4) * C::THREADS] =
                make_uint2(fd::pack_bf2(oacc[g][d][4 * r4] * inv, oacc[g][d][4 * r4 + 1] * inv),
                           fd::pack_bf2(oacc[g][d][4 * r4 + 2] * inv, oacc[g][d][4 * r4 + 3] * inv));
        ml[g * C::THREADS] = fd::f32x2_t{m_run[g], l_run[g]};
      }
      return;
    }
#pragma unroll
    for (int g = 0; g < QG; ++g) {
      const int qrow = q_lo + wave * (32 * QG) + g * 32 + l32;
      if (qrow < q_hi) store_o<DH>(O, lse, D, H, head, qrow, lg, oacc[g], m_run[g], l_run[g]);
    }
  };

  const int w = sch.share(static_cast<int>(blockIdx.x));
  long long p = sch.bound(w);
  const long long p_end = sch.bound(w + 1);
  while (p < p_end) {
    long long i_start;
    int nkv, head, b, first, tau;
    sch.locate(p, i_start, nkv, head, b, first, tau);
    if (b >= B) break;   // unreachable: p < work
    const long long i_end = i_start + nkv;
    const int kt0 = static_cast<int>(p - i_start);
    const int kt1 = static_cast<int>((p_end < i_end ? p_end : i_end) - i_start);
    int f = w, l = w;
    if (sch.cut) {
      f = sch.share_of(i_start);
      l = sch.share_of(i_end - 1);
    }
    run_piece(head, tau, b, first, kt0, kt1, w - f, l - f + 1, f);
    p = i_start + kt1;
  }
}

// The pieces of the cut items, merged in key order (deterministic for a given
// grid): workgroup x of the attention's grid takes the cut item whose first piece
// share x holds, if any, with the attention's thread geometry.  The kernel
// boundary orders the pieces' stores before these loads.
template <int DH, bool TABLES>
FD_DEVICE void combine_items(uint16_t* __restrict__ O, int D, int H, const int32_t* __restrict__ cu_q,
                             const int32_t* __restrict__ req_tok_off, int B, const float* __restrict__ partial,
                             int max_units, float* __restrict__ lse, const SchedTables* tabs) {
  using C = ACfg<DH>;
  constexpr int DT = C::DT, QG = C::QG, QB = C::QB, E = QG * (DT * 16 + 2);
  const AttnSched<QB, TABLES> sch(tabs, cu_q, req_tok_off, B, H, static_cast<int>(gridDim.x), max_units);
  if (sch.tiles == 0 || !sch.cut) return;
  const int x = sch.share(static_cast<int>(blockIdx.x));
  const long long p0 = sch.bound(x), p_end = sch.bound(x + 1);
  if (p_end <= p0) return;
  // the item of the share's last tile-step: cut with its first piece here iff it
  // starts in this share and goes on past it
  long long i_start;
  int nkv, head, b, first, tau;
  sch.locate(p_end - 1, i_start, nkv, head, b, first, tau);
  if (b >= B || i_start < p0 || i_start + nkv <= p_end) return;
  const int npieces = sch.share_of(i_start + nkv - 1) - x + 1;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, lg = lane >> 5;
  const int q_lo = cu_q[b] + (tau - first) * QB, q_hi = cu_q[b + 1];
  auto slot = [&](int j) { return partial + static_cast<size_t>(AttnSched<QB, true>::slot_of(x, j)) * (E * C::THREADS); };
  auto ml_of = [&](int j, int g) {
    return reinterpret_cast<const fd::f32x2_t*>(slot(j) + QG * DT * 16 * C::THREADS)[g * C::THREADS + tid];
  };
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    const int qrow = q_lo + wave * (32 * QG) + g * 32 + l32;
    // the pieces' maxima four at a time, then their O two at a time (in key order),
    // each batch's loads in flight before their first use
    float m_all = -INFINITY;
    for (int j0 = 0; j0 < npieces; j0 += 4) {
      float mj[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) mj[k] = j0 + k < npieces ? ml_of(j0 + k, g)[0] : -INFINITY;
#pragma unroll
      for (int k = 0; k < 4; ++k) m_all = fmaxf(m_all, mj[k]);
    }
    float l_all = 0.f;
    f32x16_t oacc[DT];
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[d][r] = 0.f;
    for (int j0 = 0; j0 < npieces; j0 += 2) {
      uint2 pv[2][DT * 4];
      fd::f32x2_t mls[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const bool has = j0 + k < npieces;
        const uint2* quads = reinterpret_cast<const uint2*>(slot(has ? j0 + k : j0)) + tid;
#pragma unroll
        for (int q = 0; q < DT * 4; ++q) pv[k][q] = quads[(g * DT * 4 + q) * C::THREADS];
        mls[k] = has ? ml_of(j0 + k, g) : fd::f32x2_t{-INFINITY, 0.f};
      }
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        // the piece's O is normalised by its own sum: weight exp2(m_k - m) * l_k
        const float wl = (mls[k][0] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mls[k][0] - m_all) * mls[k][1];
        l_all += wl;
#pragma unroll
        for (int d = 0; d < DT; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const uint2 w2 = pv[k][d * 4 + r / 4];
            const uint32_t wd = (r % 4) < 2 ? w2.x : w2.y;
            const float o = (r % 2) == 0 ? __uint_as_float(wd << 16) : __uint_as_float(wd & 0xffff0000u);
            oacc[d][r] += wl * o;
          }
      }
    }
    if (qrow < q_hi) store_o<DH>(O, lse, D, H, head, qrow, lg, oacc, m_all, l_all);
  }
}

// TABLES: the requests are located in per-workgroup prefix tables (more than
// kWalkRequests requests), else walked (no LDS, no barrier).
template <int DH, bool TABLES>
__global__ __launch_bounds__(ACfg<DH>::THREADS) void attn_combine_kernel(
    uint16_t* __restrict__ O, int D, int H, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ req_tok_off,
    int B, const float* __restrict__ partial, int max_units, float* __restrict__ lse) {
  if constexpr (TABLES) {
    __shared__ SchedTables tabs;
    build_sched_tables<ACfg<DH>::THREADS>(tabs, cu_q, req_tok_off, B, ACfg<DH>::QB);
    combine_items<DH, true>(O, D, H, cu_q, req_tok_off, B, partial, max_units, lse, &tabs);
  } else {
    combine_items<DH, false>(O, D, H, cu_q, req_tok_off, B, partial, max_units, lse, nullptr);
  }
}

}  // namespace

namespace fdh {

// Partial slots: two per share of a grid of at most two workgroups per CU.
size_t attn_scratch_bytes(int dh) {
  const size_t units = static_cast<size_t>(gemm_max_tiles());
  const size_t e = static_cast<size_t>(kMaxQG * (((dh + 31) / 32) * 16 + 2));
  return units * e * kMaxThreads * sizeof(float);
}

hipError_t launch_attention(const uint16_t* q, const uint16_t* kc, const uint16_t* vc, uint16_t* o, int D, int H,
                            int dh, const int32_t* cu_q, const int32_t* req_tok_off, int B, int n_max,
                            int max_req_tokens, float* partial, float* lse, hipStream_t s) {
  if (B < 1 || B > kMaxSchedRequests) return hipErrorInvalidValue;   // the schedule tables' size
  const int occ = dh >= 128 ? ACfg<128>::OCC : ACfg<64>::OCC;
  const int slots = occ * num_cus();
  // head dim 128: every workgroup runs whole (head, query tile) items (cut items
  // measured no faster: the kernel runs at the power limit); smaller heads cut items
  // into pieces that attn_combine_kernel merges
  const int max_units = (partial && dh < 128) ? gemm_max_tiles() : 0;
  // persistent grid: the resident slots, fewer when even one key tile per share
  // would leave some idle (upper bound on the items: every request adds at most
  // one partial query tile)
  const int qb = dh >= 128 ? ACfg<128>::QB : ACfg<64>::QB;
  const long long items = static_cast<long long>((n_max + qb - 1) / qb + B) * H;
  long long grid = items * ((max_req_tokens + KB - 1) / KB);
  if (grid > slots) grid = slots;
  if (grid < 1) grid = 1;
  grid = ((grid + kXcds - 1) / kXcds) * kXcds;
  const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(dh));
#define FD_ATTN_LAUNCH(DHV)                                                                                         \
  attn_fwd_kernel<DHV><<<grid, ACfg<DHV>::THREADS, 0, s>>>(q, kc, vc, o, D, H, cu_q, req_tok_off, B, scale_log2, partial, \
                                                           max_units, lse);                                           \
  if (max_units > 0 && B > kWalkRequests)                                                                             \
    attn_combine_kernel<DHV, true><<<grid, ACfg<DHV>::THREADS, 0, s>>>(o, D, H, cu_q, req_tok_off, B, partial,          \
                                                                       max_units, lse);                                 \
  else if (max_units > 0)                                                                                             \
    attn_combine_kernel<DHV, false><<<grid, ACfg<DHV>::THREADS, 0, s>>>(o, D, H, cu_q, req_tok_off, B, partial,         \
                                                                        max_units, lse)
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
