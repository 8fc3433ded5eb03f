// Curvature-guided subgraph draws on gfx950.
//
// Section 3.2 turns the normalised node scores of Eq. 7 and edge scores of Eq. 8 into
// sampling distributions; Section 4 trains on GraphSAINT-style subgraphs drawn from
// them.  This file draws indices from such a distribution and assembles the subgraph.
//
//   k_scan_up / k_scan_mid / k_scan_down   exclusive prefix sums over 4096-item tiles:
//        of W_i = floor(P_i * 2^62) (uint64, the integer CDF of a draw) or of 0/1 flags
//        (uint32, the new numbering of the kept nodes and edges)
//   k_draw        target t = floor(X T / 2^128) from two SplitMix64 words, then the
//                 item i with C_i <= t < C_{i+1} by binary search
//   k_mark, k_edges_of_nodes, k_nodes_of_edges, k_emit_nodes, k_emit_edges
//                 subgraph assembly: the subgraph induced on the drawn nodes, or the
//                 drawn edges with their endpoints
//
// Every sum here is an exact integer sum, so no result depends on the order in which
// the scan combines partial sums: draws and subgraphs repeat bit for bit and match
// any other exact evaluation of the same definition.
#include <hip/hip_runtime.h>

#include "erc_common.h"

namespace erc {
namespace {

constexpr int kItems = 16;              // items per thread of a scan tile
constexpr int kTile = kBlock * kItems;  // items per block of a scan
static_assert(kTile == kScanTile, "scan tile must match the host sizing");
constexpr int kPad = kItems + 1;        // LDS row pitch of one thread's items

// SplitMix64 output finaliser (Steele, Lea & Flood 2014), as for the projection signs.
__device__ __forceinline__ uint64_t sm_final(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

// Item loaders: a probability becomes its integer weight (and flags a value outside
// [0, 1]); a flag is its own value.
__device__ __forceinline__ uint64_t load_item(const double* P, int64_t i, uint32_t* status) {
  const double p = P[i];
  if (!(p >= 0.0 && p <= 1.0)) {  // also catches NaN
    atomicOr(status, kDrawBadProb);
    return 0;
  }
  // p * 2^62 is exact (a power-of-two scaling) and below 2^63; the conversion of its
  // integer part is exact too
  return static_cast<uint64_t>(p * 0x1p62);
}
__device__ __forceinline__ uint32_t load_item(const uint32_t* F, int64_t i, uint32_t*) {
  return F[i];
}

template <typename U>
__device__ __forceinline__ U wave_sum(U x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// Exclusive scan of one value per thread over the block, in thread order; `total`
// receives the block sum.
template <typename U>
__device__ __forceinline__ U block_exclusive_scan(U x, U* s_wave, U& total) {
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  U inc = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const U y = __shfl_up(inc, off);
    if (lane >= off) inc += y;
  }
  if (lane == 63) s_wave[wv] = inc;
  __syncthreads();
  U before = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kWavesPerBlock; ++w) {
    const U s = s_wave[w];
    if (w < wv) before += s;
    total += s;
  }
  __syncthreads();
  return before + inc - x;
}

// Pass 1: block b stores the sum of its tile in bsum[b] (and, for probabilities, the
// fp64 sum of the tile in psum[b], summed in a fixed order).
template <typename U, typename In>
__global__ __launch_bounds__(kBlock) void k_scan_up(const In* __restrict__ in, int64_t N,
                                                    U* __restrict__ bsum,
                                                    double* __restrict__ psum,
                                                    uint32_t* status) {
  constexpr bool kProb = sizeof(In) == sizeof(double);
  __shared__ U s_u[kWavesPerBlock];
  __shared__ double s_d[kWavesPerBlock];
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kTile;
  U acc = 0;
  double pacc = 0.0;
#pragma unroll 4
  for (int k = 0; k < kItems; ++k) {
    const int64_t i = t0 + k * kBlock + threadIdx.x;
    if (i < N) {
      acc += static_cast<U>(load_item(in, i, status));
      if constexpr (kProb) pacc += static_cast<double>(in[i]);
    }
  }
  acc = wave_sum(acc);
  if constexpr (kProb) pacc = wave_sum(pacc);
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  if (lane == 0) {
    s_u[wv] = acc;
    s_d[wv] = pacc;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    U t = 0;
    double d = 0.0;
    for (int w = 0; w < kWavesPerBlock; ++w) {
      t += s_u[w];
      d += s_d[w];
    }
    bsum[blockIdx.x] = t;
    if constexpr (kProb) psum[blockIdx.x] = d;
  }
}

// Pass 2 (one block): exclusive scan of the nb block sums in place; the grand total
// goes to *total.  For probabilities the fp64 sum must not exceed 1.5 (the integer
// weights then sum below 2^63, so no 64-bit sum above can have wrapped) and must not
// be all zero.
template <typename U>
__global__ __launch_bounds__(kBlock) void k_scan_mid(U* __restrict__ bsum, int64_t nb,
                                                     const double* __restrict__ psum,
                                                     U* __restrict__ total, uint32_t* status) {
  __shared__ U s_wave[kWavesPerBlock];
  __shared__ double s_d[kWavesPerBlock];
  U carry = 0;
  for (int64_t c0 = 0; c0 < nb; c0 += kBlock) {
    const int64_t i = c0 + threadIdx.x;
    const U x = i < nb ? bsum[i] : U(0);
    U tot;
    const U ex = block_exclusive_scan(x, s_wave, tot);
    if (i < nb) bsum[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) *total = carry;
  if (psum != nullptr) {
    double d = 0.0;
    for (int64_t i = threadIdx.x; i < nb; i += kBlock) d += psum[i];
    d = wave_sum(d);
    if ((threadIdx.x & 63) == 0) s_d[threadIdx.x >> 6] = d;
    __syncthreads();
    if (threadIdx.x == 0) {
      double all = 0.0;
      for (int w = 0; w < kWavesPerBlock; ++w) all += s_d[w];
      if (!(all <= 1.5)) atomicOr(status, kDrawSumTooLarge);
      if (carry == 0) atomicOr(status, kDrawAllZero);
    }
  }
}

// Pass 3: out[i] = (exclusive prefix of block b) + (prefix of i within the tile).  The
// tile is staged through LDS so that loads and stores stay coalesced while each thread
// scans kItems consecutive items; out may alias a flag input.
template <typename U, typename In>
__global__ __launch_bounds__(kBlock) void k_scan_down(const In* in, int64_t N,
                                                      const U* __restrict__ bsum, U* out,
                                                      uint32_t* status) {
  __shared__ U s_tile[kBlock * kPad];
  __shared__ U s_wave[kWavesPerBlock];
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kTile;
#pragma unroll 4
  for (int k = 0; k < kItems; ++k) {
    const int loc = k * kBlock + threadIdx.x;
    const int64_t i = t0 + loc;
    s_tile[(loc / kItems) * kPad + loc % kItems] =
        i < N ? static_cast<U>(load_item(in, i, status)) : U(0);
  }
  __syncthreads();
  U* mine = s_tile + threadIdx.x * kPad;
  U run = 0;
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const U x = mine[j];
    mine[j] = run;
    run += x;
  }
  U tot;
  const U off = block_exclusive_scan(run, s_wave, tot) + bsum[blockIdx.x];
#pragma unroll
  for (int j = 0; j < kItems; ++j) mine[j] += off;
  __syncthreads();
#pragma unroll 4
  for (int k = 0; k < kItems; ++k) {
    const int loc = k * kBlock + threadIdx.x;
    const int64_t i = t0 + loc;
    if (i < N) out[i] = s_tile[(loc / kItems) * kPad + loc % kItems];
  }
}

// One thread per draw.  X = x_hi 2^64 + x_lo from outputs 2d and 2d+1 of SplitMix64
// started at `base`; t = floor(X T / 2^128) = hi64(x_hi T + hi64(x_lo T)) is uniform
// on [0, T), and the drawn item is the last i with C_i <= t.
__global__ __launch_bounds__(kBlock) void k_draw(const uint64_t* __restrict__ C, int64_t N,
                                                 int64_t draws, uint64_t base,
                                                 const uint32_t* __restrict__ status,
                                                 int64_t* __restrict__ idx) {
  const uint32_t st = *status;
  const uint64_t T = C[N];
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t d = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; d < draws;
       d += stride) {
    if (st != 0u) {
      idx[d] = -1;
      continue;
    }
    const uint64_t ctr = 2ull * static_cast<uint64_t>(d);
    const uint64_t xh = sm_final(base + (ctr + 1ull) * kGolden);
    const uint64_t xl = sm_final(base + (ctr + 2ull) * kGolden);
    const uint64_t a_lo = xh * T;
    const uint64_t a_hi = __umul64hi(xh, T);
    const uint64_t s = a_lo + __umul64hi(xl, T);
    const uint64_t t = a_hi + (s < a_lo ? 1ull : 0ull);
    int64_t lo = 0, hi = N;  // C[lo] <= t < C[hi]
    while (hi - lo > 1) {
      const int64_t mid = lo + ((hi - lo) >> 1);
      if (C[mid] <= t) lo = mid;
      else hi = mid;
    }
    idx[d] = lo;
  }
}

__global__ __launch_bounds__(kBlock) void k_mark(const int64_t* __restrict__ idx,
                                                 int64_t count, int64_t N,
                                                 uint32_t* __restrict__ flag,
                                                 uint32_t* status) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t d = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; d < count;
       d += stride) {
    const int64_t i = idx[d];
    if (i < 0 || i >= N) atomicOr(status, kSubBadIndex);
    else flag[i] = 1u;  // repeated indices store the same value
  }
}

// Walk the upper (u < v) entries of every row by edge pieces; e is the canonical id.
// A group of kPieceLanes lanes takes one piece, so a wavefront works on several short
// rows at once and their chains of dependent loads overlap.
constexpr int kPieceLanes = 16;
template <typename F>
__device__ __forceinline__ void for_upper_entries(const DevGraph& g, F f) {
  constexpr int kGroups = 64 / kPieceLanes;
  const int lane = threadIdx.x & 63;
  const int sub = lane % kPieceLanes;
  const int64_t ng = static_cast<int64_t>(gridDim.x) * kWavesPerBlock * kGroups;
  for (int64_t t = (static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6)) *
                       kGroups + lane / kPieceLanes;
       t < g.npiece; t += ng) {
    const int u = g.piece_row[t];
    const int64_t pb = g.piece_beg[t], pe = g.piece_end[t];
    const int64_t upos = g.rowptr[u + 1] - (g.ubase[u + 1] - g.ubase[u]);
    const int64_t ebase = g.ubase[u] + (pb - upos);
    for (int64_t pos = pb + sub; pos < pe; pos += kPieceLanes) f(u, g.col[pos], ebase + (pos - pb));
  }
}

__global__ __launch_bounds__(kBlock) void k_edges_of_nodes(DevGraph g,
                                                           const uint32_t* __restrict__ nflag,
                                                           uint32_t* __restrict__ eflag) {
  for_upper_entries(g, [&](int u, int v, int64_t e) { eflag[e] = nflag[u] & nflag[v]; });
}

__global__ __launch_bounds__(kBlock) void k_nodes_of_edges(DevGraph g,
                                                           const uint32_t* __restrict__ eflag,
                                                           uint32_t* __restrict__ nflag) {
  for_upper_entries(g, [&](int u, int v, int64_t e) {
    if (eflag[e] != 0u) {
      nflag[u] = 1u;
      nflag[v] = 1u;
    }
  });
}

__global__ __launch_bounds__(kBlock) void k_emit_nodes(const uint32_t* __restrict__ npos,
                                                       int64_t n, int32_t* __restrict__ nodes) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n; i += stride)
    if (npos[i + 1] != npos[i]) nodes[npos[i]] = static_cast<int32_t>(i);
}

__global__ __launch_bounds__(kBlock) void k_emit_edges(DevGraph g,
                                                       const uint32_t* __restrict__ npos,
                                                       const uint32_t* __restrict__ epos,
                                                       int64_t* __restrict__ edges,
                                                       int32_t* __restrict__ uo,
                                                       int32_t* __restrict__ vo) {
  for_upper_entries(g, [&](int u, int v, int64_t e) {
    const uint32_t k = epos[e];
    if (epos[e + 1] != k) {
      edges[k] = e;
      uo[k] = static_cast<int32_t>(npos[u]);
      vo[k] = static_cast<int32_t>(npos[v]);
    }
  });
}

int grid_for_items(int64_t count, int64_t cap) {
  const int64_t g = (count + kBlock - 1) / kBlock;
  return static_cast<int>(g < 1 ? 1 : (g > cap ? cap : g));
}
int grid_for_pieces(const DevGraph& g) {
  const int64_t per_block = kWavesPerBlock * (64 / kPieceLanes);
  const int64_t b = (g.npiece + per_block - 1) / per_block;
  return static_cast<int>(b < 1 ? 1 : (b > 8192 ? 8192 : b));
}

#define ERC_DLAUNCH(kernel, grid, stream, ...) \
  hipLaunchKernelGGL(kernel, dim3(grid), dim3(kBlock), 0, stream, __VA_ARGS__)

// Exclusive scan of N items of `in` into out[0..N), block sums in bsum (scan_blocks(N)
// entries), grand total in *total.
template <typename U, typename In>
hipError_t scan(const In* in, int64_t N, U* bsum, double* psum, U* out, U* total,
                uint32_t* status, hipStream_t s) {
  const int64_t nb = scan_blocks(N);
  if (N > 0) ERC_DLAUNCH((k_scan_up<U, In>), nb, s, in, N, bsum, psum, status);
  ERC_DLAUNCH((k_scan_mid<U>), 1, s, bsum, nb, psum, total, status);
  if (N > 0) ERC_DLAUNCH((k_scan_down<U, In>), nb, s, in, N, bsum, out, status);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_draw(const double* prob, int64_t N, int64_t draws, uint64_t base,
                       const DrawWork& w, int64_t* idx, hipStream_t s) {
  hipError_t e = scan<uint64_t, double>(prob, N, w.bsum, w.psum, w.cdf, w.cdf + N, w.status, s);
  if (e != hipSuccess) return e;
  if (draws > 0) ERC_DLAUNCH(k_draw, grid_for_items(draws, 8192), s, w.cdf, N, draws, base,
                             w.status, idx);
  return hipGetLastError();
}

hipError_t launch_subgraph(const DevGraph& g, int items, const int64_t* idx, int64_t count,
                           const SubgraphWork& w, int32_t* nodes, int64_t* edges, int32_t* uo,
                           int32_t* vo, hipStream_t s) {
  // flags start at zero (the extra slot at index n or m included)
  hipError_t e = launch_fill_u32(w.npos, 0u, g.n + 1, s);
  if (e == hipSuccess) e = launch_fill_u32(w.epos, 0u, g.m + 1, s);
  if (e != hipSuccess) return e;
  if (items == 0) {
    if (count > 0) ERC_DLAUNCH(k_mark, grid_for_items(count, 8192), s, idx, count,
                               static_cast<int64_t>(g.n), w.npos, w.status);
    if (g.npiece > 0) ERC_DLAUNCH(k_edges_of_nodes, grid_for_pieces(g), s, g, w.npos, w.epos);
  } else {
    if (count > 0) ERC_DLAUNCH(k_mark, grid_for_items(count, 8192), s, idx, count, g.m,
                               w.epos, w.status);
    if (g.npiece > 0) ERC_DLAUNCH(k_nodes_of_edges, grid_for_pieces(g), s, g, w.epos, w.npos);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // in-place exclusive scans: npos[i] = new id of node i, npos[n] = kept nodes
  e = scan<uint32_t, uint32_t>(w.npos, g.n, w.bsum, nullptr, w.npos, w.npos + g.n, w.status, s);
  if (e == hipSuccess)
    e = scan<uint32_t, uint32_t>(w.epos, g.m, w.bsum, nullptr, w.epos, w.epos + g.m, w.status, s);
  if (e != hipSuccess) return e;
  ERC_DLAUNCH(k_emit_nodes, grid_for_items(g.n, 8192), s, w.npos, static_cast<int64_t>(g.n),
              nodes);
  if (g.npiece > 0)
    ERC_DLAUNCH(k_emit_edges, grid_for_pieces(g), s, g, w.npos, w.epos, edges, uo, vo);
  return hipGetLastError();
}

}  // namespace erc
