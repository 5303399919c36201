// Recursive load-aware patch partitioning (the Patch Partitioner, Sec. 3.1):
// every request's tokens are bisected by the Otsu threshold of their integer
// saliency into a focus set (saliency >= theta) and a context set, which get r_f
// and R - r_f of the node's R regions, until every node holds one region.
//
// Since every split is a threshold on saliency, every node of the recursion is
// the set of tokens whose saliency lies in an interval of the request's sorted
// distinct values: a node is a range [a, b) of that list.  With exact prefix
// counts PC and sums PS over the list, the class counts and sums of the
// candidate split at list position p (focus = values >= v_p) are
// PC[p] - PC[a] and PS[p] - PS[a], so one node costs one pass over its distinct
// values and none over its tokens.  A node with a single distinct value has no
// split; its tokens are cut into R chunks of consecutive token indices.
//
// One workgroup per request runs the whole recursion: the 16-bit value
// histogram (two bins per LDS word, counts below 2^16), the distinct-value list
// with its prefix counts and sums (global workspace), one level of splits at a
// time with the workgroup's waves shared among the nodes, and the region of every token.  No host round trip.
#include "fd_common.h"

namespace {

constexpr int kPartThreads = 1024;
constexpr int kPartWaves = kPartThreads / fd::kWave;
constexpr int kValues = 65536;                  // saliency is uint16
constexpr int kValWords = kValues / 2;          // two 16-bit bins per word
constexpr int kWordsPerThread = kValWords / kPartThreads;
// One pad word after every 32: a thread's 32 consecutive words then start 33
// words after its neighbour's, so a wave's reads of them hit distinct banks.
constexpr int kBinWords = kValWords + kValWords / 32;

FD_DEVICE int bin_word(int w) { return w + (w >> 5); }

enum : uint8_t { kNone = 0, kSplit = 1, kLeaf = 2, kChunk = 3 };

struct PartReqs {
  int32_t tok_off[fd::kMaxPartRequests + 1];   // request token ranges
  int32_t reg_off[fd::kMaxPartRequests + 1];   // request region ranges
};

struct PartWs {
  int32_t* dv;        // [N]     distinct values of each request, ascending
  int32_t* node_of;   // [N]     node of each distinct value
  int32_t* pc;        // [N + B] tokens below each distinct value (exclusive prefix)
  int64_t* ps;        // [N + B] saliency sum below each distinct value
};

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

template <typename T>
FD_DEVICE T wave_scan_incl(T v, int lane) {
#pragma unroll
  for (int o = 1; o < fd::kWave; o <<= 1) {
    const T u = __shfl_up(v, o, fd::kWave);
    if (lane >= o) v += u;
  }
  return v;
}

// Exclusive workgroup scan of (x, y, z) in thread order; totals in tx, ty, tz.
// Called by every thread of the workgroup.
FD_DEVICE void block_scan3(int& x, int& y, int64_t& z, int& tx, int& ty, int64_t& tz, int* sx, int* sy,
                           int64_t* sz) {
  const int lane = threadIdx.x & (fd::kWave - 1), wave = threadIdx.x / fd::kWave;
  const int ix = wave_scan_incl(x, lane), iy = wave_scan_incl(y, lane);
  const int64_t iz = wave_scan_incl(z, lane);
  if (lane == fd::kWave - 1) {
    sx[wave] = ix;
    sy[wave] = iy;
    sz[wave] = iz;
  }
  __syncthreads();
  int bx = 0, by = 0;
  int64_t bz = 0;
  tx = 0;
  ty = 0;
  tz = 0;
  for (int w = 0; w < kPartWaves; ++w) {
    if (w == wave) {
      bx = tx;
      by = ty;
      bz = tz;
    }
    tx += sx[w];
    ty += sy[w];
    tz += sz[w];
  }
  x = bx + ix - x;
  y = by + iy - y;
  z = bz + iz - z;
  __syncthreads();
}

// Regions given to the focus set: the r in 1 .. R-1 nearest to R n_f / n (ties
// to the smaller r), kept within [max(1, R - n_c), min(R - 1, n_f)] so that no
// region is empty.
FD_DEVICE int focus_share(int64_t n_f, int64_t n_c, int R) {
  const double x = static_cast<double>(static_cast<int64_t>(R) * n_f) / static_cast<double>(n_f + n_c);
  int64_t r = static_cast<int64_t>(floor(x));
  if (x - static_cast<double>(r) > 0.5) ++r;
  if (r < 1) r = 1;
  if (r < R - n_c) r = R - n_c;
  if (r > R - 1) r = R - 1;
  if (r > n_f) r = n_f;
  return static_cast<int>(r);
}

__global__ __launch_bounds__(kPartThreads) void partition_kernel(const uint16_t* __restrict__ saliency,
                                                                 PartReqs reqs, PartWs ws,
                                                                 int32_t* __restrict__ region) {
  __shared__ uint32_t s_bins[kBinWords];   // value counts, then value -> distinct index (padded)
  __shared__ int32_t s_a[fd::kMaxPartRegions], s_b[fd::kMaxPartRegions], s_rn[fd::kMaxPartRegions];
  __shared__ int16_t s_todo[fd::kMaxPartRegions];
  __shared__ uint8_t s_kind[fd::kMaxPartRegions];
  __shared__ int s_sx[kPartWaves], s_sy[kPartWaves];
  __shared__ int64_t s_sz[kPartWaves];
  __shared__ int s_ntodo;
  __shared__ double s_best[kPartWaves];
  __shared__ int s_bp[kPartWaves];
  __shared__ int64_t s_nc[kPartWaves];

  const int req = blockIdx.x;
  const int T0 = reqs.tok_off[req], n = reqs.tok_off[req + 1] - T0;
  const int G0 = reqs.reg_off[req], R = reqs.reg_off[req + 1] - G0;
  const uint16_t* sal = saliency + T0;
  int32_t* dv = ws.dv + T0;
  int32_t* node_of = ws.node_of + T0;
  int32_t* pc = ws.pc + T0 + req;
  int64_t* ps = ws.ps + T0 + req;
  const int tid = threadIdx.x, lane = tid & (fd::kWave - 1), wave = tid / fd::kWave;

  // histogram of the request's saliency values
  for (int w = tid; w < kBinWords; w += kPartThreads) s_bins[w] = 0;
  __syncthreads();
  for (int t = tid; t < n; t += kPartThreads) {
    const int v = sal[t];
    atomicAdd(&s_bins[bin_word(v >> 1)], 1u << ((v & 1) * 16));
  }
  __syncthreads();

  // distinct values in ascending order with exclusive prefix counts and sums;
  // every bin word is replaced by the distinct indices of its two values
  const int w0 = tid * kWordsPerThread, p0 = bin_word(w0);
  int nz = 0, cnt = 0;
  int64_t sum = 0;
  for (int j = 0; j < kWordsPerThread; ++j) {
    const uint32_t word = s_bins[p0 + j];
    const int c0 = static_cast<int>(word & 0xffffu), c1 = static_cast<int>(word >> 16);
    const int v = 2 * (w0 + j);
    nz += (c0 > 0) + (c1 > 0);
    cnt += c0 + c1;
    sum += static_cast<int64_t>(c0) * v + static_cast<int64_t>(c1) * (v + 1);
  }
  int U, n_all;
  int64_t s_all;
  block_scan3(nz, cnt, sum, U, n_all, s_all, s_sx, s_sy, s_sz);
  for (int j = 0; j < kWordsPerThread; ++j) {
    const uint32_t word = s_bins[p0 + j];
    uint32_t map = 0;
    for (int h = 0; h < 2; ++h) {
      const int c = static_cast<int>((word >> (16 * h)) & 0xffffu);
      if (c == 0) continue;
      const int v = 2 * (w0 + j) + h;
      dv[nz] = v;
      pc[nz] = cnt;
      ps[nz] = sum;
      map |= static_cast<uint32_t>(nz) << (16 * h);
      ++nz;
      cnt += c;
      sum += static_cast<int64_t>(c) * v;
    }
    s_bins[p0 + j] = map;
  }
  if (tid == 0) {
    pc[U] = n_all;
    ps[U] = s_all;
  }
  for (int f = tid; f < R; f += kPartThreads) s_kind[f] = kNone;
  __syncthreads();
  if (tid == 0) {
    s_a[0] = 0;
    s_b[0] = U;
    s_rn[0] = R;
    s_kind[0] = R > 1 ? kSplit : kLeaf;
  }
  __syncthreads();

  // One level of splits per pass.  A node owns the region ids [f, f + rn[f]) and
  // only the thread that splits it writes entries inside that range.  Every
  // pass splits or ends each node it takes, so at most R passes run.  With K
  // nodes to split, a group of wpn = 16 / K waves (a power of two, at least 1)
  // scans each node's candidates; groups take the nodes in rounds.
  for (int level = 0; level <= R; ++level) {
    if (wave == 0) {
      int k = 0;
      for (int f0 = 0; f0 < R; f0 += fd::kWave) {
        const int f = f0 + lane;
        const bool p = f < R && s_kind[f] == kSplit;
        const uint64_t m = __ballot(p);
        if (p) s_todo[k + __popcll(m & ((1ull << lane) - 1))] = static_cast<int16_t>(f);
        k += __popcll(m);
      }
      if (lane == 0) s_ntodo = k;
    }
    __syncthreads();
    const int K = s_ntodo;
    if (K == 0) break;
    int wpn = kPartWaves;
    while (wpn > 1 && wpn * K > kPartWaves) wpn >>= 1;
    const int groups = kPartWaves / wpn, sub = wave % wpn, stride = wpn * fd::kWave;
    for (int j0 = 0; j0 < K; j0 += groups) {
      const int j = j0 + wave / wpn;
      int f = 0, a = 0, b = 0;
      if (j < K) {
        f = s_todo[j];
        a = s_a[f];
        b = s_b[f];
      }
      const int pa = j < K ? pc[a] : 0;
      const int64_t sa = j < K ? ps[a] : 0;
      const int64_t nn = j < K ? pc[b] - pa : 0, tot = j < K ? ps[b] - sa : 0;
      double best = -1.0;
      int bp = b;
      int64_t bnc = 0;   // context count of the best split
      if (j < K) {
#pragma clang fp contract(off)
        // between-class variance w_f w_c (mu_f - mu_c)^2 of the split at each
        // distinct value but the smallest, from exact integer counts and sums;
        // four candidates' prefix loads in flight per lane, ascending order kept
        for (int p0 = a + 1 + sub * fd::kWave + lane; p0 < b; p0 += 4 * stride) {
          int64_t ncs[4], scs[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int p = p0 + u * stride;
            ncs[u] = p < b ? pc[p] : 0;
            scs[u] = p < b ? ps[p] : 0;
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int p = p0 + u * stride;
            if (p >= b) continue;
            const int64_t n_c = ncs[u] - pa, s_c = scs[u] - sa;
            const int64_t n_f = nn - n_c, s_f = tot - s_c;
            const double wf = static_cast<double>(n_f) / static_cast<double>(nn);
            const double wc = static_cast<double>(n_c) / static_cast<double>(nn);
            const double d = static_cast<double>(s_f) / static_cast<double>(n_f) -
                             static_cast<double>(s_c) / static_cast<double>(n_c);
            const double sb = wf * wc * (d * d);
            if (sb > best) {
              best = sb;
              bp = p;
              bnc = n_c;
            }
          }
        }
      }
      // the largest variance wins, ties to the smallest threshold
      for (int o = fd::kWave / 2; o > 0; o >>= 1) {
        const double ob = __shfl_xor(best, o, fd::kWave);
        const int op = __shfl_xor(bp, o, fd::kWave);
        const int64_t onc = __shfl_xor(bnc, o, fd::kWave);
        if (ob > best || (ob == best && op < bp)) {
          best = ob;
          bp = op;
          bnc = onc;
        }
      }
      if (lane == 0) {
        s_best[wave] = best;
        s_bp[wave] = bp;
        s_nc[wave] = bnc;
      }
      __syncthreads();
      if (j < K && sub == 0 && lane == 0) {
        const int Rn = s_rn[f];
        if (b - a == 1) {   // one saliency value: no split
          s_kind[f] = kChunk;
        } else {
          for (int w = wave + 1; w < wave + wpn; ++w)
            if (s_best[w] > best || (s_best[w] == best && s_bp[w] < bp)) {
              best = s_best[w];
              bp = s_bp[w];
              bnc = s_nc[w];
            }
          const int rf = focus_share(nn - bnc, bnc, Rn);
          s_a[f] = bp;
          s_b[f] = b;
          s_rn[f] = rf;
          s_kind[f] = rf > 1 ? kSplit : kLeaf;
          s_a[f + rf] = a;
          s_b[f + rf] = bp;
          s_rn[f + rf] = Rn - rf;
          s_kind[f + rf] = Rn - rf > 1 ? kSplit : kLeaf;
        }
      }
      __syncthreads();
    }
  }

  // node of every distinct value
  for (int f = wave; f < R; f += kPartWaves) {
    const uint8_t kind = s_kind[f];
    if (kind != kLeaf && kind != kChunk) continue;
    for (int k = s_a[f] + lane; k < s_b[f]; k += fd::kWave) node_of[k] = f;
  }
  __syncthreads();

  // tokens of one-region nodes
  for (int t = tid; t < n; t += kPartThreads) {
    const int v = sal[t];
    const int k = static_cast<int>((s_bins[bin_word(v >> 1)] >> ((v & 1) * 16)) & 0xffffu);
    const int f = node_of[k];
    if (s_kind[f] == kLeaf) region[T0 + t] = G0 + f;
  }

  // tokens of a node with one value: chunk floor(rank R_f / n_f), rank in token
  // order among the tokens of that value
  for (int f = 0; f < R; ++f) {
    if (s_kind[f] != kChunk) continue;
    const int k = s_a[f];
    const int v = dv[k], nf = pc[k + 1] - pc[k], Rn = s_rn[f];
    int base = 0;
    for (int t0 = 0; t0 < n; t0 += kPartThreads) {
      const int t = t0 + tid;
      const int in = (t < n && sal[t] == v) ? 1 : 0;
      int rank = in, zero = 0, n_in, n_zero;
      int64_t z = 0, n_z;
      block_scan3(rank, zero, z, n_in, n_zero, n_z, s_sx, s_sy, s_sz);
      if (in) region[T0 + t] = G0 + f + static_cast<int>(static_cast<int64_t>(base + rank) * Rn / nf);
      base += n_in;
    }
  }
}

}  // namespace

namespace fdh {

size_t partition_ws_bytes(int n_tokens, int n_requests) {
  const size_t N = static_cast<size_t>(n_tokens), B = static_cast<size_t>(n_requests);
  return 2 * align256(N * 4) + align256((N + B) * 4) + align256((N + B) * 8);
}

hipError_t launch_partition(int n_requests, const int32_t* req_tok_off, const int32_t* req_reg_off,
                            const uint16_t* saliency, int32_t* region, void* ws, hipStream_t s) {
  PartReqs reqs{};
  for (int b = 0; b <= n_requests; ++b) {
    reqs.tok_off[b] = req_tok_off[b];
    reqs.reg_off[b] = req_reg_off[b];
  }
  const size_t N = static_cast<size_t>(req_tok_off[n_requests]), B = static_cast<size_t>(n_requests);
  uintptr_t p = reinterpret_cast<uintptr_t>(ws);
  PartWs w;
  w.dv = reinterpret_cast<int32_t*>(p);
  p += align256(N * 4);
  w.node_of = reinterpret_cast<int32_t*>(p);
  p += align256(N * 4);
  w.pc = reinterpret_cast<int32_t*>(p);
  p += align256((N + B) * 4);
  w.ps = reinterpret_cast<int64_t*>(p);
  partition_kernel<<<n_requests, kPartThreads, 0, s>>>(saliency, reqs, w, region);
  return hipGetLastError();
}

}  // namespace fdh
