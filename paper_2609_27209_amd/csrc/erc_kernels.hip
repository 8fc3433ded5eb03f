// HIP kernels for gfx950 (CDNA4, wave64) of the resistance-curvature path.
//
//   k_rhs        Y = B^T W^{1/2} Q for one column block (Section 3.1.2; Algorithm 1,
//                forming Y^(t)); also initialises the CG state z = 0, r = p = Y.
//   k_spmm       q = (L + delta I) p, with the fused dot products p.q, r.q, q.q
//                (Eq. 5; the matrix-free operator of Section 3.1.3).
//   k_update     z += alpha p, r -= alpha q, p = r + beta p, and r.r (column-wise CG,
//                Section 3.1.3; Algorithm 1).
//   k_edge_dist  R_e += sum_c (z_uc - z_vc)^2 (Eq. 6; Algorithm 1, edge blocks).
//   k_node_p, k_edge_kappa   node and edge curvature (Eq. 2).
//   k_minmax, k_node_w, k_edge_w, k_normalise   sampling probabilities (Eqs. 7, 8).
//
// Layout: every n x kb block (z, r, p, q) is row-major with kb a power of two, so one
// row is 64..1024 bytes.  In the gather kernels a row is read by LPN lanes with one
// 16-byte load each and a wavefront covers NPW = 64 / LPN neighbours per instruction.
//
// Determinism: no floating-point atomics anywhere.  Each block reduces its partial
// sums in a fixed order and the grid combines block partials through a fixed-fan-in
// tree (tree_sum): an integer ticket only elects which block performs each level, the
// summation order is a function of the grid size alone.  Results are therefore
// bit-identical from run to run.
#include <hip/hip_runtime.h>

#include "erc_common.h"

namespace erc {
namespace {

template <typename T>
struct __attribute__((aligned(16))) V {
  static constexpr int N = 16 / sizeof(T);
  T x[N];
};

template <typename T>
__device__ __forceinline__ V<T> ldv(const T* p) {
  return *reinterpret_cast<const V<T>*>(p);
}
template <typename T>
__device__ __forceinline__ void stv(T* p, const V<T>& v) {
  *reinterpret_cast<V<T>*>(p) = v;
}
// Non-temporal 16-byte loads and stores for data that is streamed once per launch, so
// the L2 keeps the rows that neighbour gathers reuse.
template <typename T>
struct NtVec;
template <>
struct NtVec<float> {
  typedef float type __attribute__((ext_vector_type(4)));
};
template <>
struct NtVec<double> {
  typedef double type __attribute__((ext_vector_type(2)));
};
template <typename T>
__device__ __forceinline__ V<T> ldv_nt(const T* p) {
  typedef typename NtVec<T>::type E;
  const E e = __builtin_nontemporal_load(reinterpret_cast<const E*>(p));
  V<T> v;
#pragma unroll
  for (int k = 0; k < V<T>::N; ++k) v.x[k] = e[k];
  return v;
}
template <typename T>
__device__ __forceinline__ void stv_nt(T* p, const V<T>& v) {
  typedef typename NtVec<T>::type E;
  E e;
#pragma unroll
  for (int k = 0; k < V<T>::N; ++k) e[k] = v.x[k];
  __builtin_nontemporal_store(e, reinterpret_cast<E*>(p));
}

// fp64 accumulator of one lane's V<T>::N columns: the SpMM's block tasks and split rows
// (the rows above a thousand entries) sum in fp64 whatever the working precision.
template <typename T>
struct A64 {
  double x[V<T>::N];
};
template <typename T>
__device__ __forceinline__ A64<T> azero() {
  A64<T> a;
#pragma unroll
  for (int k = 0; k < V<T>::N; ++k) a.x[k] = 0.0;
  return a;
}

template <typename T>
__device__ __forceinline__ V<T> vzero() {
  V<T> v;
#pragma unroll
  for (int k = 0; k < V<T>::N; ++k) v.x[k] = T(0);
  return v;
}

__device__ __forceinline__ double readlane_f64(double x, int k) {
  const long long b = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_readlane(static_cast<int>(b & 0xffffffffll), k);
  const int hi = __builtin_amdgcn_readlane(static_cast<int>(b >> 32), k);
  return __longlong_as_double((static_cast<long long>(hi) << 32) |
                              (static_cast<unsigned int>(lo)));
}

__device__ __forceinline__ uint64_t readlane_u64(uint64_t x, int k) {
  const unsigned lo = static_cast<unsigned>(__builtin_amdgcn_readlane(static_cast<int>(x & 0xffffffffull), k));
  const unsigned hi = static_cast<unsigned>(__builtin_amdgcn_readlane(static_cast<int>(x >> 32), k));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// SplitMix64 output finaliser (Steele, Lea & Flood 2014).
__device__ __forceinline__ uint64_t splitmix_final(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
// Output number `ctr` of SplitMix64 started from state `base`.
__device__ __forceinline__ uint64_t splitmix_at(uint64_t base, uint64_t ctr) {
  return splitmix_final(base + (ctr + 1ull) * 0x9E3779B97F4A7C15ull);
}

// ---------------------------------------------------------------------------------
// Inner products are accumulated in at least twice the working precision: fp32
// products are exact in fp64 and are summed in fp64; fp64 products are split exactly
// (fma) and summed as double-double pairs (Knuth's TwoSum), so the CG coefficients do
// not inherit the summation error of a plain fp64 sum.
struct DDv {
  double s, c;  // value s + c
};

__device__ __forceinline__ void two_sum_d(double a, double b, double& s, double& e) {
#pragma clang fp contract(off)
  s = a + b;
  const double z = s - a;
  e = (a - (s - z)) + (b - z);
}

__device__ __forceinline__ DDv dd_add(const DDv& a, const DDv& b) {
#pragma clang fp contract(off)
  double s, e;
  two_sum_d(a.s, b.s, s, e);
  DDv r;
  r.s = s;
  r.c = (a.c + b.c) + e;
  return r;
}

__device__ __forceinline__ DDv dd_mul_d(const DDv& a, double b) {
#pragma clang fp contract(off)
  const double p = a.s * b;
  const double pe = fma(a.s, b, -p);
  const double c = pe + a.c * b;
  DDv r;
  two_sum_d(p, c, r.s, r.c);
  return r;
}

__device__ __forceinline__ double dd_value(const DDv& a) { return a.s + a.c; }

template <typename T>
struct Dot;
template <>
struct Dot<float> {
  double s = 0.0;
  __device__ __forceinline__ void add(float x, float y) {
    s = fma(static_cast<double>(x), static_cast<double>(y), s);  // exact product, one rounding
  }
  __device__ __forceinline__ DDv get() const { return DDv{s, 0.0}; }
  __device__ __forceinline__ static DDv one(float x, float y) {
    return DDv{static_cast<double>(x) * static_cast<double>(y), 0.0};
  }
};
template <>
struct Dot<double> {
  double s = 0.0, c = 0.0;
  __device__ __forceinline__ void add(double x, double y) {
#pragma clang fp contract(off)
    const double p = x * y;
    const double pe = fma(x, y, -p);
    double t, e;
    two_sum_d(s, p, t, e);
    s = t;
    c += e + pe;
  }
  __device__ __forceinline__ DDv get() const { return DDv{s, c}; }
  __device__ __forceinline__ static DDv one(double x, double y) {
#pragma clang fp contract(off)
    const double p = x * y;
    return DDv{p, fma(x, y, -p)};
  }
};

// ---------------------------------------------------------------------------------
// Deterministic grid reduction.  `in` (LDS, nval doubles) holds this block's values.
// Returns true in exactly one block, with the grid totals in `out` (LDS).  All threads
// of every block must call it.  Tickets are left at zero for the next launch.
template <class Op>
__device__ bool tree_reduce(const Tree& t, int nval, const double* in, double* out) {
  __shared__ int s_last;
  const int tid = threadIdx.x;
  if (gridDim.x == 1) {
    for (int v = tid; v < nval; v += blockDim.x) out[v] = in[v];
    __syncthreads();
    return true;
  }
  for (int v = tid; v < nval; v += blockDim.x)
    t.lvl0[static_cast<size_t>(blockIdx.x) * nval + v] = in[v];
  int cnt = gridDim.x;
  int idx = blockIdx.x;
  const double* src = t.lvl0;
  uint32_t* tick = t.tick;
  for (int level = 0;; ++level) {
    const int ng = (cnt + kTreeFan - 1) / kTreeFan;
    const int grp = idx / kTreeFan;
    const int gsize = min(kTreeFan, cnt - grp * kTreeFan);
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = (atomicAdd(&tick[grp], 1u) == static_cast<unsigned>(gsize - 1));
    __syncthreads();
    if (!s_last) return false;
    __threadfence();
    double* dst = (ng == 1) ? out : (level == 0 ? t.lvl1 : t.lvl2) + static_cast<size_t>(grp) * nval;
    for (int v = tid; v < nval; v += blockDim.x) {
      const double* b = src + static_cast<size_t>(grp) * kTreeFan * nval + v;
      double s = b[0];
      for (int k = 1; k < gsize; ++k) s = Op::apply(s, b[static_cast<size_t>(k) * nval]);
      dst[v] = s;
    }
    if (tid == 0) tick[grp] = 0u;
    if (ng == 1) {
      __syncthreads();
      return true;
    }
    src = (level == 0) ? t.lvl1 : t.lvl2;
    tick += ng;
    cnt = ng;
    idx = grp;
  }
}
struct OpSum {
  __device__ static double apply(double a, double b) { return a + b; }
};
struct OpMax {
  __device__ static double apply(double a, double b) { return a > b ? a : b; }
};

// The same tree for compensated pairs: `in`/`out` are LDS arrays of nval pairs and the
// level buffers hold nval pairs per block.
__device__ bool tree_sum_dd(const Tree& t, int nval, const DDv* in, DDv* out) {
  __shared__ int s_last;
  const int tid = threadIdx.x;
  if (gridDim.x == 1) {
    for (int v = tid; v < nval; v += blockDim.x) out[v] = in[v];
    __syncthreads();
    return true;
  }
  DDv* l0 = reinterpret_cast<DDv*>(t.lvl0);
  for (int v = tid; v < nval; v += blockDim.x) l0[static_cast<size_t>(blockIdx.x) * nval + v] = in[v];
  int cnt = gridDim.x;
  int idx = blockIdx.x;
  const DDv* src = l0;
  uint32_t* tick = t.tick;
  for (int level = 0;; ++level) {
    const int ng = (cnt + kTreeFan - 1) / kTreeFan;
    const int grp = idx / kTreeFan;
    const int gsize = min(kTreeFan, cnt - grp * kTreeFan);
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = (atomicAdd(&tick[grp], 1u) == static_cast<unsigned>(gsize - 1));
    __syncthreads();
    if (!s_last) return false;
    __threadfence();
    DDv* lvl = reinterpret_cast<DDv*>(level == 0 ? t.lvl1 : t.lvl2);
    DDv* dst = (ng == 1) ? out : lvl + static_cast<size_t>(grp) * nval;
    for (int v = tid; v < nval; v += blockDim.x) {
      const DDv* b = src + static_cast<size_t>(grp) * kTreeFan * nval + v;
      DDv acc = b[0];
      for (int k = 1; k < gsize; ++k) acc = dd_add(acc, b[static_cast<size_t>(k) * nval]);
      dst[v] = acc;
    }
    if (tid == 0) tick[grp] = 0u;
    if (ng == 1) {
      __syncthreads();
      return true;
    }
    src = lvl;
    tick += ng;
    cnt = ng;
    idx = grp;
  }
}

// ---------------------------------------------------------------------------------
// Neighbour gather of one row range: acc += w_ij (p_i - p_j) over CSR entries
// [beg, end) of row i, in the working precision (acc a V<T>) or with each term formed
// and added in fp64 (acc an A64<T>: the block tasks, whose rows hold thousands to tens
// of thousands of entries, where an fp32 sum loses the small differences between a hub
// and its neighbours).  Lane (grp, sub) handles neighbour slot grp of each step and
// columns [sub*VEC, sub*VEC + VEC).  Each lane issues kInflight row loads (half as many
// with fp64 sums) before it consumes them, so a wavefront keeps kInflight * 1 KB of
// gathers in flight.  Slots past
// the end read p_i with weight 0, which adds exactly zero.
#ifndef ERC_SPMM_INFLIGHT
#define ERC_SPMM_INFLIGHT 8
#endif
constexpr int kInflight = ERC_SPMM_INFLIGHT;
// Short-row chunks whose longest row exceeds this many entries are gathered one row at
// a time by the whole wavefront instead of one row per lane group.
#ifndef ERC_WAVE_ROW_MIN
#define ERC_WAVE_ROW_MIN 32
#endif
constexpr int kWaveRowMin = ERC_WAVE_ROW_MIN;

template <typename T, int LPN, bool W, typename ACC>
__device__ __forceinline__ void gather_row(const int32_t* __restrict__ col,
                                           const T* __restrict__ wgt, const T* __restrict__ P,
                                           int i, int64_t beg, int64_t end, const V<T>& pi,
                                           ACC& acc, int lane) {
  constexpr bool D = sizeof(ACC) > sizeof(V<T>);  // fp64 sums of an fp32 row
  constexpr int VEC = V<T>::N;
  constexpr int KB = LPN * VEC;
  constexpr int NPW = 64 / LPN;
  const int grp = lane / LPN;
  const int sub = lane % LPN;
  for (int64_t base = beg; base < end; base += 64) {
    const int cnt = static_cast<int>(min(static_cast<int64_t>(64), end - base));
    int myj = i;
    T myw = T(0);
    if (lane < cnt) {
      myj = col[base + lane];
      if (W) myw = wgt[base + lane];
    }
    const int steps = (cnt + NPW - 1) / NPW;
    // fewer rows in flight with fp64 sums, which hold twice the accumulator registers
    // (a quarter for weighted rows at 8 lanes per row, the instantiation closest to the
    // register cap: it spilled 35 registers at half, 19 at a quarter)
    constexpr int NI = D ? ((W && LPN == 8) ? kInflight / 4 : kInflight / 2) : kInflight;
    for (int st = 0; st < steps; st += NI) {
      V<T> pj[NI];
      T wj[NI];
#pragma unroll
      for (int u = 0; u < NI; ++u) {
        const int k = (st + u) * NPW + grp;
        int j = __shfl(myj, k & 63);
        wj[u] = W ? __shfl(myw, k & 63) : T(1);
        if (k >= cnt) {
          j = i;
          wj[u] = T(0);
        }
        pj[u] = ldv(P + static_cast<int64_t>(j) * KB + sub * VEC);
      }
#pragma unroll
      for (int u = 0; u < NI; ++u) {
        if constexpr (D) {
          const double w64 = W ? static_cast<double>(wj[u]) : 1.0;
#pragma unroll
          for (int v = 0; v < VEC; ++v)
            acc.x[v] += w64 * (static_cast<double>(pi.x[v]) - static_cast<double>(pj[u].x[v]));
        } else if (W) {
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc.x[v] += wj[u] * (pi.x[v] - pj[u].x[v]);
        } else {
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc.x[v] += pi.x[v] - pj[u].x[v];
        }
      }
    }
  }
}

// Sum acc over the NPW neighbour groups of the wavefront (xor butterfly: every lane
// ends with the same, order-fixed total).
template <typename T, int LPN, typename ACC>
__device__ __forceinline__ void reduce_groups(ACC& acc) {
#pragma unroll
  for (int off = LPN; off < 64; off <<= 1) {
#pragma unroll
    for (int v = 0; v < V<T>::N; ++v) acc.x[v] += __shfl_xor(acc.x[v], off);
  }
}

struct SpmmArgs {
  DevGraph g;
  const void* p;
  const void* r;
  void* q;
  void* chunkbuf;
  double* mega_dots;  // nmega x 3 x kb pairs
  double* part;       // grid x 3 x kb pairs: this launch's block partials
  const int32_t* gate;
  double delta;
  const void* minv;   // Jacobi variant: 1/(d_i + delta) per row (else nullptr)
};

// q = (L + delta I) p for a block of kb = LPN*VEC columns, plus per-column p.q, r.q,
// q.q accumulated in at least twice the working precision (with the Jacobi variant the
// last two are weighted by m_i = 1/(d_i + delta): (m r).q and (m q).q).  Block tasks (long rows,
// split over the 4 waves of a block and, beyond one block's share, over several
// blocks) run first; then each wave walks its own contiguous range of short rows.  A row
// split over several blocks only stores its chunk sums here; k_mega_fin, the next
// launch on the stream, adds them, so no block needs a device-scope fence.
template <typename T, int LPN, bool W>
// At most 128 VGPRs (four waves per SIMD): the 32-column instantiation would take 138
// and fall to three waves, which costs more than its few spilled registers.
__global__ __launch_bounds__(kBlock, 4) void k_spmm(SpmmArgs a) {
  constexpr int VEC = V<T>::N;
  constexpr int KB = LPN * VEC;
  if (*a.gate == 0) return;
  __shared__ DDv s_dots[kWavesPerBlock][3 * KB];
  // the block tasks' per-wave sums share the LDS of the dot partials, which are written
  // only after the last task's closing barrier
  static_assert(sizeof(A64<T>) * kWavesPerBlock * LPN <= sizeof(DDv) * kWavesPerBlock * 3 * KB,
                "block-task sums must fit the dot partials' LDS");
  A64<T> (*s_acc)[LPN] = reinterpret_cast<A64<T> (*)[LPN]>(&s_dots[0][0]);

  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int sub = lane % LPN;
  const T* __restrict__ P = static_cast<const T*>(a.p);
  const T* __restrict__ Rr = static_cast<const T*>(a.r);
  T* __restrict__ Q = static_cast<T*>(a.q);
  const T* __restrict__ wgt = static_cast<const T*>(a.g.w);
  const T* __restrict__ minv = static_cast<const T*>(a.minv);
  const bool pc = minv != nullptr;
  const T dlt = static_cast<T>(a.delta);

  // p.q, r.q, q.q partials of the rows this lane's group finishes (block tasks are
  // finished by group 0 of wave 0)
  Dot<T> ldots[3 * VEC];

  // finish one row in group-0 lanes: q = delta p_i + acc (a block task's fp64 sum is
  // rounded once), store, and accumulate the dots into this lane's partials
  auto finish = [&](int i, const V<T>& pi, const auto& acc) {
    V<T> qv;
    const int64_t off = static_cast<int64_t>(i) * KB + sub * VEC;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      if constexpr (sizeof(acc) > sizeof(V<T>))
        qv.x[v] = static_cast<T>(a.delta * static_cast<double>(pi.x[v]) + acc.x[v]);
      else
        qv.x[v] = dlt * pi.x[v] + acc.x[v];
    }
    stv_nt(Q + off, qv);
    const V<T> ri = ldv_nt(Rr + off);
    const T mi = pc ? minv[i] : T(1);
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      ldots[v].add(pi.x[v], qv.x[v]);
      ldots[VEC + v].add(pc ? ri.x[v] * mi : ri.x[v], qv.x[v]);
      ldots[2 * VEC + v].add(pc ? qv.x[v] * mi : qv.x[v], qv.x[v]);
    }
  };

  // 1. block-cooperative tasks
  for (int t = blockIdx.x; t < a.g.ntask; t += gridDim.x) {
    const int i = a.g.task_row[t];
    const int mh = a.g.task_mega[t];
    const int64_t tb = a.g.task_beg[t];
    const int64_t len = a.g.task_end[t] - tb;
    const int64_t wb = tb + (len * wv) / kWavesPerBlock;
    const int64_t we = tb + (len * (wv + 1)) / kWavesPerBlock;
    const V<T> pi = ldv(P + static_cast<int64_t>(i) * KB + sub * VEC);
    A64<T> acc = azero<T>();
    gather_row<T, LPN, W>(a.g.col, wgt, P, i, wb, we, pi, acc, lane);
    reduce_groups<T, LPN>(acc);
    if (lane < LPN) s_acc[wv][sub] = acc;
    __syncthreads();
    A64<T> tot = azero<T>();
    if (wv == 0 && lane < LPN) {
#pragma unroll
      for (int w = 0; w < kWavesPerBlock; ++w) {
        const A64<T> x = s_acc[w][sub];
#pragma unroll
        for (int v = 0; v < VEC; ++v) tot.x[v] += x.x[v];
      }
    }
    if (wv == 0 && lane < LPN) {
      if (mh < 0) {
        finish(i, pi, tot);
      } else {
        // one chunk of a split row: its fp64 sum goes to the row's chunk slot, k_mega_fin
        // adds the chunks
        double* cb = static_cast<double*>(a.chunkbuf) + a.g.mega_chunk0[mh] * static_cast<int64_t>(KB) +
                     static_cast<int64_t>(a.g.task_chunk[t]) * KB + sub * VEC;
#pragma unroll
        for (int v = 0; v < VEC; ++v) cb[v] = tot.x[v];
      }
    }
    __syncthreads();
  }

  // 2. this wave's short rows, NPW at a time: lane group g owns row lo + g (+ NPW ...),
  // loads its own neighbour indices LPN at a time and gathers kInflight rows of p per
  // step, so a wavefront has NPW rows and NPW * kInflight gathers in flight and needs
  // no cross-group reduction per row.  A chunk whose longest row has more than
  // kWaveRowMin entries would leave the other groups idle; its rows are gathered one at
  // a time by the whole wavefront instead.
  {
    constexpr int NPW = 64 / LPN;
    const int grp = lane / LPN;
    const int gw = blockIdx.x * kWavesPerBlock + wv;
    const int lo = a.g.wave_lo[gw];
    const int hi = a.g.wave_lo[gw + 1];
    const LightRow* __restrict__ LR = a.g.light;
    // each group's next light row is loaded one step ahead, so a step starts with the
    // row id and CSR range at hand; groups past the end repeat the wave's last row
    // with no entries
    LightRow nxt{};
    if (lo < hi) nxt = LR[min(lo + grp, hi - 1)];
    for (int k0 = lo; k0 < hi; k0 += NPW) {
      const int k = k0 + grp;
      const bool valid = k < hi;
      const LightRow cur = nxt;
      if (k0 + NPW < hi) nxt = LR[min(k + NPW, hi - 1)];
      const int i = cur.row;
      const int64_t b = cur.beg;
      const int deg = valid ? cur.deg : 0;
      int dmax = deg;
#pragma unroll
      for (int off = LPN; off < 64; off <<= 1) dmax = max(dmax, __shfl_xor(dmax, off));
      if (dmax > kWaveRowMin) {
        // a chunk with a long row: the whole wavefront takes its rows one at a time
        const int kn = min(NPW, hi - k0);
        for (int r = 0; r < kn; ++r) {
          const LightRow lr = LR[k0 + r];
          const int ir = lr.row;
          const V<T> pir = ldv(P + static_cast<int64_t>(ir) * KB + sub * VEC);
          V<T> accr = vzero<T>();
          gather_row<T, LPN, W>(a.g.col, wgt, P, ir, lr.beg, lr.beg + lr.deg, pir, accr, lane);
          reduce_groups<T, LPN>(accr);
          if (lane < LPN) finish(ir, pir, accr);
        }
        continue;
      }
      const V<T> pi = ldv(P + static_cast<int64_t>(i) * KB + sub * VEC);
      V<T> acc = vzero<T>();
      for (int base = 0; base < dmax; base += LPN) {
        const int t = base + sub;
        int myj = i;
        T myw = T(0);
        if (t < deg) {
          myj = a.g.col[b + t];
          if (W) myw = wgt[b + t];
        }
        const int cnt = min(LPN, dmax - base);
        for (int u0 = 0; u0 < cnt; u0 += kInflight) {
          V<T> pj[kInflight];
          T wj[kInflight];
#pragma unroll
          for (int u = 0; u < kInflight; ++u) {
            const int tt = u0 + u;
            const int src = grp * LPN + (tt & (LPN - 1));
            int j = __shfl(myj, src);
            wj[u] = W ? __shfl(myw, src) : T(1);
            if (tt >= LPN || base + tt >= deg) {
              j = i;
              wj[u] = T(0);
            }
            pj[u] = ldv(P + static_cast<int64_t>(j) * KB + sub * VEC);
          }
#pragma unroll
          for (int u = 0; u < kInflight; ++u) {
            if (W) {
#pragma unroll
              for (int v = 0; v < VEC; ++v) acc.x[v] += wj[u] * (pi.x[v] - pj[u].x[v]);
            } else {
#pragma unroll
              for (int v = 0; v < VEC; ++v) acc.x[v] += pi.x[v] - pj[u].x[v];
            }
          }
        }
      }
      if (valid) {
        const int64_t off = static_cast<int64_t>(i) * KB + sub * VEC;
        V<T> qv;
#pragma unroll
        for (int v = 0; v < VEC; ++v) qv.x[v] = dlt * pi.x[v] + acc.x[v];
        stv_nt(Q + off, qv);
        const V<T> ri = ldv_nt(Rr + off);
        const T mi = pc ? minv[i] : T(1);
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
          ldots[v].add(pi.x[v], qv.x[v]);
          ldots[VEC + v].add(pc ? ri.x[v] * mi : ri.x[v], qv.x[v]);
          ldots[2 * VEC + v].add(pc ? qv.x[v] * mi : qv.x[v], qv.x[v]);
        }
      }
    }
  }

  // 3. block partials: fold the lane groups (xor butterfly on compensated pairs), then
  // the waves in order, then store this block's pairs for the finishing launch
  {
#pragma unroll
    for (int d = 0; d < 3 * VEC; ++d) {
      DDv x = ldots[d].get();
#pragma unroll
      for (int off = LPN; off < 64; off <<= 1) {
        DDv y;
        y.s = __shfl_xor(x.s, off);
        y.c = __shfl_xor(x.c, off);
        x = dd_add(x, y);
      }
      if (lane < LPN) s_dots[wv][(d / VEC) * KB + sub * VEC + (d % VEC)] = x;
    }
  }

  __syncthreads();
  for (int v = threadIdx.x; v < 3 * KB; v += kBlock) {
    DDv acc = s_dots[0][v];
#pragma unroll
    for (int w = 1; w < kWavesPerBlock; ++w) acc = dd_add(acc, s_dots[w][v]);
    s_dots[0][v] = acc;
  }
  __syncthreads();
  DDv* part = reinterpret_cast<DDv*>(a.part) + static_cast<int64_t>(blockIdx.x) * 3 * KB;
  for (int v = threadIdx.x; v < 3 * KB; v += kBlock) part[v] = s_dots[0][v];
}

// Rows split over several blocks of the SpMM: one wavefront per row adds the row's
// fp64 chunk sums in chunk order (the order the chunks cover the row), forms q_i =
// delta p_i + sum, and stores the row's p.q, r.q, q.q terms as its own compensated pairs
// (nmega x 3 x kb), which k_fin_col adds to the column totals.  Running in the launch
// after the SpMM makes the chunk sums visible without a device-scope fence.
template <typename T, int LPN>
__global__ __launch_bounds__(64) void k_mega_fin(SpmmArgs a) {
  constexpr int VEC = V<T>::N;
  constexpr int KB = LPN * VEC;
  if (*a.gate == 0) return;
  const int mh = blockIdx.x;
  const int sub = threadIdx.x;
  if (sub >= LPN) return;
  const int i = a.g.mega_row[mh];
  const int nch = a.g.mega_nchunk[mh];
  const double* __restrict__ cb =
      static_cast<const double*>(a.chunkbuf) + a.g.mega_chunk0[mh] * static_cast<int64_t>(KB);
  A64<T> rs = azero<T>();
  for (int k = 0; k < nch; ++k) {
    const double* x = cb + static_cast<int64_t>(k) * KB + sub * VEC;
#pragma unroll
    for (int v = 0; v < VEC; ++v) rs.x[v] += x[v];
  }
  const T* __restrict__ P = static_cast<const T*>(a.p);
  const T* __restrict__ Rr = static_cast<const T*>(a.r);
  T* __restrict__ Q = static_cast<T*>(a.q);
  const T* __restrict__ minv = static_cast<const T*>(a.minv);
  const bool pc = minv != nullptr;
  const int64_t off = static_cast<int64_t>(i) * KB + sub * VEC;
  const V<T> pi = ldv(P + off);
  V<T> qv;
#pragma unroll
  for (int v = 0; v < VEC; ++v)
    qv.x[v] = static_cast<T>(a.delta * static_cast<double>(pi.x[v]) + rs.x[v]);
  stv_nt(Q + off, qv);
  const V<T> ri = ldv_nt(Rr + off);
  const T mi = pc ? minv[i] : T(1);
  DDv* dst = reinterpret_cast<DDv*>(a.mega_dots) + static_cast<int64_t>(mh) * 3 * KB;
#pragma unroll
  for (int v = 0; v < VEC; ++v) {
    dst[sub * VEC + v] = Dot<T>::one(pi.x[v], qv.x[v]);
    dst[KB + sub * VEC + v] = Dot<T>::one(pc ? ri.x[v] * mi : ri.x[v], qv.x[v]);
    dst[2 * KB + sub * VEC + v] = Dot<T>::one(pc ? qv.x[v] * mi : qv.x[v], qv.x[v]);
  }
}

// Level-1 sum of the block partials written by the previous launch: block b of this
// small grid adds partials [32 b, 32 b + 32) in order; the blocks then meet in the
// ticket tree.  Reading the partials in a separate launch makes them visible without a
// device-scope fence in every block of the large kernel.  Returns true in the block
// that holds the totals (`out`, LDS).
__device__ bool reduce_partials(const DDv* __restrict__ part, int nparts, int nval,
                                const Tree& t, DDv* in, DDv* out) {
  const int b0 = blockIdx.x * kTreeFan;
  const int nb = min(kTreeFan, nparts - b0);
  for (int v = threadIdx.x; v < nval; v += blockDim.x) {
    DDv acc = part[static_cast<int64_t>(b0) * nval + v];
    for (int k = 1; k < nb; ++k) acc = dd_add(acc, part[static_cast<int64_t>(b0 + k) * nval + v]);
    in[v] = acc;
  }
  __syncthreads();
  return tree_sum_dd(t, nval, in, out);
}

struct FinArgs {
  const double* part;
  int nparts;        // blocks of the launch that wrote `part`
  Tree tree;
  ColState cs;
  double tol2;
  int ncols;
  int pc;            // Jacobi variant: the partials also hold y.M^-1 y
};

struct IterArgs {
  const double* part_s;  // SpMM block partials: p.q, r.q, q.q (3 kb pairs per block)
  int nparts_s;
  const double* part_u;  // update block partials: r.r (and r.M^-1 r): 1 or 2 kb pairs
  int nparts_u;
  int pc;                // Jacobi variant: the update also reduced r.M^-1 r
  Tree tree;
  ColState cs;
  const double* mega_dots;
  int nmega;
  int mode;              // 0: stopping test of the pending update, then alpha/beta; 1: test
                         // only; 2: test only, and only when the previous mode-0 launch
                         // predicted that every active column stops
};

// The per-iteration finishing step, in two launches without device-scope fences:
//  k_fin_sum  (ceil(parts/32) x ceil(values/64) blocks) level-1 sums of the block
//             partials of the previous update (r.r, and r.M^-1 r with the Jacobi
//             variant) and of this SpMM (p.q, r.q, q.q; M^-1-weighted r.q, q.q with
//             the Jacobi variant),
//             stored value-major so that the next launch reads them contiguously;
//             skipped when the partial sets are short (k_fin_col then reads them);
//  k_fin_col  (one block per column) the grid totals of its column in a fixed order,
//             then (1) the stopping test of the pending update, r.r <= tol^2 rho_0,
//             and rho = r.r (or r.M^-1 r), and (2) alpha = rho / p.q and, for the
//             direction update, rho' = rho - 2 alpha r.q + alpha^2 q.q, i.e. the new rho
//             expanded in double-double.  One integer atomic per block collects the
//             active-column count; the last block to finish publishes it.
// mode 0: both steps; 1: the stopping test only; 2: the stopping test only, and only
// when the previous mode-0 step predicted that every active column stops.
constexpr int kFinDirectMax = 2048;  // longest partial set k_fin_col sums by itself
constexpr unsigned long long kFinField = (1ull << 20) - 1;  // one field of the counter word

// k_fin_sum's grid is (groups of kTreeFan partials) x (64-value slices): each wavefront
// of a block adds one quarter of its group's partials for 64 consecutive values, all of
// its loads issued before they are added, and wavefront 0 then adds the quarters in
// order, so every level-1 sum waits on one round of loads.
constexpr int kFinWaves = kBlock / 64;
constexpr int kFinPer = kTreeFan / kFinWaves;  // partials per wavefront and value
static_assert(kTreeFan % kFinWaves == 0, "a partial group must split over the wavefronts");

template <int KB>
__global__ __launch_bounds__(kBlock) void k_fin_sum(IterArgs a) {
  if (*a.cs.n_active == 0) return;
  if (a.mode == 2 && *a.cs.pred_done == 0) return;
  __shared__ DDv s_q[kFinWaves][64];
  const bool upd = *a.cs.upd_pending != 0;
  const bool dots = a.mode == 0;
  const int su = (a.pc ? 2 : 1) * KB;  // update values first, then the SpMM's three
  const int nval = su + 3 * KB;
  const int lane = threadIdx.x & 63;
  const int wq = threadIdx.x >> 6;
  const int v = blockIdx.y * 64 + lane;
  DDv acc = DDv{0.0, 0.0};
  if (v < nval) {
    const bool isu = v < su;
    const DDv* part = reinterpret_cast<const DDv*>(isu ? a.part_u : a.part_s);
    const int np = isu ? a.nparts_u : a.nparts_s;
    const int pv = isu ? su : 3 * KB;
    const int vv = isu ? v : v - su;
    const int k0 = blockIdx.x * kTreeFan + wq * kFinPer;
    const int cnt = min(kFinPer, np - k0);
    if ((isu ? upd : dots) && cnt > 0) {
      // this wavefront's partials in block order
      const DDv* src = part + static_cast<int64_t>(k0) * pv + vv;
      DDv x[kFinPer];
#pragma unroll
      for (int u = 0; u < kFinPer; ++u)
        x[u] = u < cnt ? src[static_cast<int64_t>(u) * pv] : DDv{0.0, 0.0};
      acc = x[0];
#pragma unroll
      for (int u = 1; u < kFinPer; ++u)
        if (u < cnt) acc = dd_add(acc, x[u]);
    }
  }
  s_q[wq][lane] = acc;
  __syncthreads();
  if (wq == 0 && v < nval) {
#pragma unroll
    for (int q = 1; q < kFinWaves; ++q) acc = dd_add(acc, s_q[q][lane]);
    reinterpret_cast<DDv*>(a.tree.lvl0)[static_cast<int64_t>(v) * gridDim.x + blockIdx.x] = acc;
  }
}

// nsum > 0: k_fin_sum wrote nsum level-1 sums per value; nsum == 0: read the block
// partials themselves.
template <int KB>
__global__ __launch_bounds__(kBlock) void k_fin_col(IterArgs a, int nsum) {
  if (*a.cs.n_active == 0) return;
  if (a.mode == 2 && *a.cs.pred_done == 0) return;
  __shared__ DDv s_red[5][kBlock / 64];
  __shared__ int s_last;
  const bool upd = *a.cs.upd_pending != 0;
  const bool dots = a.mode == 0;
  const int su = (a.pc ? 2 : 1) * KB;
  const int c = blockIdx.x;
  const int tid = threadIdx.x;
  // value slots of this column: r.r, r.M^-1 r, p.q, r.q, q.q
  const int idx[5] = {c, KB + c, su + c, su + KB + c, su + 2 * KB + c};
#pragma unroll
  for (int k = 0; k < 5; ++k) {
    const bool need = (k == 0 && upd) || (k == 1 && upd && a.pc) || (k >= 2 && dots);
    // element t of this value's list: a level-1 sum, or one block's partial
    const DDv* src;
    int64_t stride;
    int cnt;
    if (nsum > 0) {
      src = reinterpret_cast<const DDv*>(a.tree.lvl0) + static_cast<int64_t>(idx[k]) * nsum;
      stride = 1;
      cnt = nsum;
    } else if (k < 2) {
      src = reinterpret_cast<const DDv*>(a.part_u) + idx[k];
      stride = su;
      cnt = a.nparts_u;
    } else {
      src = reinterpret_cast<const DDv*>(a.part_s) + (idx[k] - su);
      stride = 3 * KB;
      cnt = a.nparts_s;
    }
    DDv acc = DDv{0.0, 0.0};
    if (need) {
      // this thread's elements t = tid, tid + kBlock, ... added in that order; eight
      // loads are issued before they are added, which leaves the sum unchanged
      int t = tid;
      for (; t + 7 * kBlock < cnt; t += 8 * kBlock) {
        DDv x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] = src[static_cast<int64_t>(t + u * kBlock) * stride];
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = (t + u * kBlock == tid) ? x[u] : dd_add(acc, x[u]);
      }
      for (; t < cnt; t += kBlock) {
        const DDv x = src[static_cast<int64_t>(t) * stride];
        acc = (t == tid) ? x : dd_add(acc, x);
      }
      // the SpMM dots of rows split over several blocks (one triple of pairs per row)
      if (k >= 2) {
        const DDv* md = reinterpret_cast<const DDv*>(a.mega_dots) + (k - 2) * KB + c;
        for (int mh = tid; mh < a.nmega; mh += kBlock)
          acc = dd_add(acc, md[static_cast<int64_t>(mh) * 3 * KB]);
      }
    }
    // fold the wavefront's 64 sums (xor butterfly: every lane ends with the same,
    // order-fixed total); the block's four wavefront totals are added below in order
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      DDv y;
      y.s = __shfl_xor(acc.s, off);
      y.c = __shfl_xor(acc.c, off);
      acc = dd_add(acc, y);
    }
    if ((tid & 63) == 0) s_red[k][tid >> 6] = acc;
  }
  __syncthreads();
  if (tid == 0) {
#pragma unroll
    for (int k = 0; k < 5; ++k) {
      DDv t = s_red[k][0];
      for (int w = 1; w < kBlock / 64; ++w) t = dd_add(t, s_red[k][w]);
      s_red[k][0] = t;
    }
    int live = 0;
    if (upd && a.cs.active[c]) {
      const double rn = dd_value(s_red[0][0]);
      const double rs = a.pc ? dd_value(s_red[1][0]) : rn;
      a.cs.iters[c] += 1;
      a.cs.rr[c] = rn;
      a.cs.rho[c] = rs;
      if (!(rn > a.cs.thr[c])) {
        a.cs.active[c] = 0;
        if (!isfinite(rn)) a.cs.status[c] = 1;
      } else if (!(rs > 0.0) || !isfinite(rs)) {
        a.cs.active[c] = 0;
        a.cs.status[c] = 1;
      }
    }
    if (dots && a.cs.active[c]) {
      const DDv pqd = s_red[2][0], rq = s_red[3][0], qq = s_red[4][0];
      const double pq = dd_value(pqd);
      const double rho = a.cs.rho[c];
      if (!(pq > 0.0) || !isfinite(pq) || !isfinite(dd_value(rq)) || !isfinite(dd_value(qq))) {
        a.cs.active[c] = 0;
        a.cs.status[c] = 1;
        a.cs.alpha[c] = 0.0;
        a.cs.beta[c] = 0.0;
      } else {
        // rho' = ||r - alpha q||^2 = rho - 2 alpha r.q + alpha^2 q.q (M^-1-weighted with
        // the Jacobi variant), evaluated in double-double; the exact value for the
        // updated r is reduced by the next finishing step and drives the stopping test
        // and the next alpha.
        const double al = rho / pq;
        const DDv t1 = dd_mul_d(rq, -2.0 * al);
        const DDv t2 = dd_mul_d(dd_mul_d(qq, al), al);
        const double rf = dd_value(dd_add(dd_add(DDv{rho, 0.0}, t1), t2));
        a.cs.alpha[c] = al;
        a.cs.beta[c] = (rf > 0.0 ? rf : 0.0) / rho;
        // plain CG: rf predicts the r.r of the stopping test; with the Jacobi variant
        // it is r.M^-1 r, so every column counts as possibly stopping
        live = (!a.pc && rf > a.cs.thr[c]) ? 1 : 0;
      }
    } else {
      a.cs.alpha[c] = 0.0;
      a.cs.beta[c] = 0.0;
    }
    // one atomic per block on one word: active columns (bits 40-59), columns predicted
    // to go on (bits 20-39) and blocks done (bits 0-19); the block that adds last reads
    // the totals from the sum and clears the word for the next launch
    const unsigned long long add = (static_cast<unsigned long long>(a.cs.active[c] ? 1 : 0) << 40) |
                                   (static_cast<unsigned long long>(live) << 20) | 1ull;
    const unsigned long long old = atomicAdd(a.cs.fin_word, add);
    s_last = (old & kFinField) == static_cast<unsigned long long>(gridDim.x - 1);
    if (s_last) {
      // every other block has added its column: publish the totals, reset the word
      const unsigned long long tot = old + add;
      const int cnt = static_cast<int>((tot >> 40) & kFinField);
      const bool any_live = ((tot >> 20) & kFinField) != 0;
      atomicExch(a.cs.fin_word, 0ull);
      *a.cs.n_active = cnt;
      *a.cs.upd_pending = (dots && cnt > 0) ? 1 : 0;
      *a.cs.pred_done = (dots && cnt > 0 && !any_live) ? 1 : 0;
      if (dots) *a.cs.nspmm += 1;
    }
  }
}

#ifndef ERC_UPD_UNROLL
#define ERC_UPD_UNROLL 2
#endif
constexpr int kUpdUnroll = ERC_UPD_UNROLL;

struct UpdArgs {
  void* z;
  void* r;
  void* p;
  const void* q;
  const void* minv;  // Jacobi variant: 1/(d_i + delta) per row
  int64_t nvec;  // n * kb / VEC
  double* part;  // grid x kb pairs (grid x 2 kb with the Jacobi variant)
  ColState cs;
};

// z += alpha p; r -= alpha q; p = r + beta p (active columns); rho' = r.r in at least
// twice the working precision.  With the Jacobi variant (PC): s = m_i r, p = s + beta p
// and the partials hold r.r then r.s.  Thread x of the grid-stride loop always covers
// column group x % CG (and row x / CG), so each thread keeps fixed-column partials.
template <typename T, int CG, bool PC>
__global__ __launch_bounds__(kBlock) void k_update(UpdArgs a) {
  constexpr int VEC = V<T>::N;
  constexpr int KB = CG * VEC;
  constexpr int NP = PC ? 2 : 1;
  static_assert(kBlock % CG == 0, "column groups must divide the block");
  if (*a.cs.n_active == 0) return;
  __shared__ DDv s_part[kBlock][NP * VEC];
  const T* __restrict__ minv = static_cast<const T*>(a.minv);
  const int cg = threadIdx.x % CG;
  T al[VEC], be[VEC];
  bool act[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) {
    const int c = cg * VEC + v;
    al[v] = static_cast<T>(a.cs.alpha[c]);
    be[v] = static_cast<T>(a.cs.beta[c]);
    act[v] = a.cs.active[c] != 0;
  }
  Dot<T> part[VEC];
  Dot<T> part_s[PC ? VEC : 1];
  T* __restrict__ Z = static_cast<T*>(a.z);
  T* __restrict__ R = static_cast<T*>(a.r);
  T* __restrict__ P = static_cast<T*>(a.p);
  const T* __restrict__ Qv = static_cast<const T*>(a.q);
  // kUpdUnroll vectors per thread per step, loads of all of them issued first
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t x0 = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; x0 < a.nvec;
       x0 += stride * kUpdUnroll) {
    V<T> z[kUpdUnroll], r[kUpdUnroll], p[kUpdUnroll], q[kUpdUnroll];
#pragma unroll
    for (int u = 0; u < kUpdUnroll; ++u) {
      const int64_t x = x0 + u * stride;
      if (x < a.nvec) {
        const int64_t o = x * VEC;
        z[u] = ldv_nt(Z + o);
        r[u] = ldv_nt(R + o);
        p[u] = ldv_nt(P + o);
        q[u] = ldv_nt(Qv + o);
      }
    }
#pragma unroll
    for (int u = 0; u < kUpdUnroll; ++u) {
      const int64_t x = x0 + u * stride;
      if (x < a.nvec) {
        const int64_t o = x * VEC;
        const T mi = PC ? minv[x / CG] : T(1);
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
          z[u].x[v] += al[v] * p[u].x[v];
          r[u].x[v] -= al[v] * q[u].x[v];
          part[v].add(r[u].x[v], r[u].x[v]);
          if constexpr (PC) {
            const T sv = mi * r[u].x[v];
            part_s[v].add(r[u].x[v], sv);
            if (act[v]) p[u].x[v] = sv + be[v] * p[u].x[v];
          } else {
            if (act[v]) p[u].x[v] = r[u].x[v] + be[v] * p[u].x[v];
          }
        }
        stv_nt(Z + o, z[u]);
        stv_nt(R + o, r[u]);
        stv(P + o, p[u]);  // p is gathered by the next SpMM
      }
    }
  }
#pragma unroll
  for (int v = 0; v < VEC; ++v) {
    s_part[threadIdx.x][v] = part[v].get();
    if constexpr (PC) s_part[threadIdx.x][VEC + v] = part_s[v].get();
  }
  __syncthreads();
  DDv* bp = reinterpret_cast<DDv*>(a.part) + static_cast<int64_t>(blockIdx.x) * NP * KB;
  for (int c = threadIdx.x; c < NP * KB; c += kBlock) {
    const int k = c / KB, cc = c % KB;
    const int g = cc / VEC, v = k * VEC + cc % VEC;
    DDv acc = s_part[g][v];
    for (int t = g + CG; t < kBlock; t += CG) acc = dd_add(acc, s_part[t][v]);
    bp[c] = acc;
  }
}

struct RhsArgs {
  DevGraph g;
  void* z;
  void* r;
  void* p;
  int col0;
  int ncols;
  uint64_t words;  // 64-bit sign words per edge, ceil(K/64)
  uint64_t base;   // SplitMix64 state the sign stream starts from
  double inv_sqrt_k;
  double* part;    // grid x kb pairs (grid x 2 kb with the Jacobi variant)
  const void* minv;  // Jacobi variant: 1/(d_i + delta) per row
};

// One wavefront per row; lane l holds columns l, l+64, ... of the block.  The sum over
// the row's neighbours runs in ascending CSR order in fp64 and is rounded once, so Y is
// reproducible bit for bit.  Neighbours, edge ids and sqrt(w) are loaded 64 at a time;
// each lane hashes the sign words of its own entry once, and the per-entry loop reads
// them back with readlane (one hash per entry instead of one per entry and lane).  The CG
// state starts as z = 0, r = y and p = y (p = m_i y with the Jacobi variant, PC).
template <typename T, int KB, bool PC>
__global__ __launch_bounds__(kBlock) void k_rhs(RhsArgs a) {
  constexpr int CPL = (KB + 63) / 64;
  constexpr int NP = PC ? 2 : 1;
  __shared__ DDv s_part[kWavesPerBlock][NP * KB];
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  T* __restrict__ Z = static_cast<T*>(a.z);
  T* __restrict__ R = static_cast<T*>(a.r);
  T* __restrict__ Pp = static_cast<T*>(a.p);
  const bool aligned = (a.col0 & 63) == 0;
  Dot<T> r0[CPL];
  Dot<T> s0[PC ? CPL : 1];
  const int nw = gridDim.x * kWavesPerBlock;
  for (int i = blockIdx.x * kWavesPerBlock + wv; i < a.g.n; i += nw) {
    double acc[CPL];
#pragma unroll
    for (int cl = 0; cl < CPL; ++cl) acc[cl] = 0.0;
    const int64_t b = a.g.rowptr[i];
    const int64_t e = a.g.rowptr[i + 1];
    for (int64_t base = b; base < e; base += 64) {
      const int cnt = static_cast<int>(min(static_cast<int64_t>(64), e - base));
      int myj = 0, mye = 0;
      double mysw = 0.0;
      if (lane < cnt) {
        myj = a.g.col[base + lane];
        mye = a.g.eid[base + lane];
        // sqrt(w_e): from the entry's own weight when it holds the input value exactly
        // (a correctly rounded fp64 sqrt, the same value the host stores per edge), else
        // from the per-edge table
        if (!a.g.weighted)
          mysw = 1.0;
        else if (a.g.sw_from_w)
          mysw = sqrt(static_cast<double>(static_cast<const T*>(a.g.w)[base + lane]));
        else
          mysw = a.g.sw[mye];
      }
      // lane l hashes the sign words of entry base + l that the block's columns need:
      // words w0 .. w0 + NW - 1 of its edge (one more when col0 is not word-aligned)
      uint64_t myw[CPL + 1];
      {
        const uint64_t ctr0 = static_cast<uint64_t>(mye) * a.words + static_cast<uint64_t>(a.col0 >> 6);
#pragma unroll
        for (int u = 0; u < CPL + 1; ++u)
          myw[u] = (u < CPL || !aligned) ? splitmix_at(a.base, ctr0 + u) : 0ull;
      }
      for (int k = 0; k < cnt; ++k) {
        const int j = __builtin_amdgcn_readlane(myj, k);
        const double s = readlane_f64(mysw, k);
        const double t = (i < j) ? s : -s;  // B_{e,i}: +1 at the smaller endpoint
#pragma unroll
        for (int cl = 0; cl < CPL; ++cl) {
          const int c = a.col0 + cl * 64 + lane;  // global column of this lane
          uint64_t word = readlane_u64(myw[cl], k);
          if (!aligned) {
            const uint64_t whi = readlane_u64(myw[cl + 1], k);
            word = ((c >> 6) == ((a.col0 + cl * 64) >> 6)) ? word : whi;
          }
          const bool neg = (word >> (c & 63)) & 1ull;
          acc[cl] += neg ? -t : t;
        }
      }
    }
    const T mi = PC ? static_cast<const T*>(a.minv)[i] : T(1);
#pragma unroll
    for (int cl = 0; cl < CPL; ++cl) {
      const int cc = cl * 64 + lane;
      if (cc < KB) {
        const T y = (cc < a.ncols) ? static_cast<T>(acc[cl] * a.inv_sqrt_k) : T(0);
        const int64_t o = static_cast<int64_t>(i) * KB + cc;
        R[o] = y;
        Z[o] = T(0);
        r0[cl].add(y, y);
        if constexpr (PC) {
          const T sv = mi * y;
          Pp[o] = sv;
          s0[cl].add(y, sv);
        } else {
          Pp[o] = y;
        }
      }
    }
  }
#pragma unroll
  for (int cl = 0; cl < CPL; ++cl) {
    const int cc = cl * 64 + lane;
    if (cc < KB) {
      s_part[wv][cc] = r0[cl].get();
      if constexpr (PC) s_part[wv][KB + cc] = s0[cl].get();
    }
  }
  __syncthreads();
  for (int c = threadIdx.x; c < NP * KB; c += kBlock) {
    DDv acc = s_part[0][c];
#pragma unroll
    for (int w = 1; w < kWavesPerBlock; ++w) acc = dd_add(acc, s_part[w][c]);
    s_part[0][c] = acc;
  }
  __syncthreads();
  DDv* part = reinterpret_cast<DDv*>(a.part) + static_cast<int64_t>(blockIdx.x) * NP * KB;
  for (int c = threadIdx.x; c < NP * KB; c += kBlock) part[c] = s_part[0][c];
}

// Unit weights, blocks of at most 64 columns: every term of a row's sum is +-1, so the
// sum is an exact integer whatever the order of its terms, and the wavefront forms it
// from ballots instead of a per-entry loop.  Lane l takes entry l of each 64-entry chunk
// (orientation o_l = +1 when i < j, else -1; sign bits b_lc of the block's columns);
// column c gains sum_l o_l (1 - 2 b_lc) = (|P| - |N|) - 2 (|P & B_c| - |N & B_c|) with
// P, N the lanes of positive and negative orientation and B_c the lanes whose bit c is
// set.  The integer times 1/sqrt(K), rounded once, is the same Y as the fp64 sum of
// k_rhs; z, r, p and the y.y partials are written as there.
template <typename T, int KB>
__global__ __launch_bounds__(kBlock) void k_rhs_unit(RhsArgs a) {
  static_assert(KB <= 64, "a block's columns span at most two sign words");
  __shared__ DDv s_part[kWavesPerBlock][KB];
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  T* __restrict__ Z = static_cast<T*>(a.z);
  T* __restrict__ R = static_cast<T*>(a.r);
  T* __restrict__ Pp = static_cast<T*>(a.p);
  const int sh = a.col0 & 63;  // bit of the block's first column in its sign word
  const bool two = sh + KB > 64;
  Dot<T> r0;
  const int nw = gridDim.x * kWavesPerBlock;
  for (int i = blockIdx.x * kWavesPerBlock + wv; i < a.g.n; i += nw) {
    int acc = 0;  // lane c < KB: column col0 + c of row i
    const int64_t b = a.g.rowptr[i];
    const int64_t e = a.g.rowptr[i + 1];
    for (int64_t base = b; base < e; base += 64) {
      const int cnt = static_cast<int>(min(static_cast<int64_t>(64), e - base));
      const bool live = lane < cnt;
      int myj = i, mye = 0;
      if (live) {
        myj = a.g.col[base + lane];
        mye = a.g.eid[base + lane];
      }
      const uint64_t ctr0 = static_cast<uint64_t>(mye) * a.words + static_cast<uint64_t>(a.col0 >> 6);
      const uint64_t w0 = splitmix_at(a.base, ctr0);
      const uint64_t w1 = two ? splitmix_at(a.base, ctr0 + 1) : 0ull;
      // bit c: the sign bit of global column col0 + c of this entry's edge
      const uint64_t bits = sh == 0 ? w0 : ((w0 >> sh) | (w1 << (64 - sh)));
      const uint64_t pos = __ballot(live && i < myj);
      const uint64_t neg = __ballot(live && i > myj);
      const int base_c = __popcll(pos) - __popcll(neg);
#pragma unroll
      for (int c = 0; c < KB; ++c) {
        const uint64_t m = __ballot(live && ((bits >> c) & 1ull));
        const int v = base_c - 2 * (__popcll(pos & m) - __popcll(neg & m));
        acc += (lane == c) ? v : 0;
      }
    }
    if (lane < KB) {
      const T y = (lane < a.ncols) ? static_cast<T>(static_cast<double>(acc) * a.inv_sqrt_k) : T(0);
      const int64_t o = static_cast<int64_t>(i) * KB + lane;
      R[o] = y;
      Z[o] = T(0);
      Pp[o] = y;
      r0.add(y, y);
    }
  }
  if (lane < KB) s_part[wv][lane] = r0.get();
  __syncthreads();
  for (int c = threadIdx.x; c < KB; c += kBlock) {
    DDv acc = s_part[0][c];
#pragma unroll
    for (int w = 1; w < kWavesPerBlock; ++w) acc = dd_add(acc, s_part[w][c]);
    s_part[0][c] = acc;
  }
  __syncthreads();
  DDv* part = reinterpret_cast<DDv*>(a.part) + static_cast<int64_t>(blockIdx.x) * KB;
  for (int c = threadIdx.x; c < KB; c += kBlock) part[c] = s_part[0][c];
}

// rho_0 = y.y per column; initial CG state of the block (rho = y.M^-1 y with the
// Jacobi variant).
template <int KB>
__global__ __launch_bounds__(kBlock) void k_fin_rhs(FinArgs a) {
  __shared__ DDv s_in[2 * KB];
  __shared__ DDv s_out[2 * KB];
  const int nval = (a.pc ? 2 : 1) * KB;
  if (!reduce_partials(reinterpret_cast<const DDv*>(a.part), a.nparts, nval, a.tree, s_in, s_out))
    return;
  if (threadIdx.x == 0) {
    *a.cs.upd_pending = 0;
    *a.cs.pred_done = 0;
    *a.cs.nspmm = 0;
  }
  for (int c = threadIdx.x; c < KB; c += kBlock) {
    const double rr = dd_value(s_out[c]);
    a.cs.rho[c] = a.pc ? dd_value(s_out[KB + c]) : rr;
    a.cs.rr[c] = rr;
    a.cs.rho0[c] = rr;
    a.cs.thr[c] = a.tol2 * rr;
    a.cs.active[c] = (c < a.ncols && rr > 0.0) ? 1 : 0;
    a.cs.iters[c] = 0;
    a.cs.status[c] = 0;
    a.cs.alpha[c] = 0.0;
    a.cs.beta[c] = 0.0;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int cnt = 0;
    for (int c = 0; c < KB; ++c) cnt += a.cs.active[c] != 0;
    *a.cs.n_active = cnt;
  }
}

// R_e (+)= sum_c (z_uc - z_vc)^2 over the upper entries (v > u) of each piece.  The
// squared difference is formed in fp64; LPN lanes sum one edge's columns.
template <typename T, int LPN>
__global__ __launch_bounds__(kBlock) void k_edge_dist(DevGraph g, const T* __restrict__ Z,
                                                      double* __restrict__ R, int accumulate) {
  constexpr int VEC = V<T>::N;
  constexpr int KB = LPN * VEC;
  constexpr int NPW = 64 / LPN;
  const int lane = threadIdx.x & 63;
  const int grp = lane / LPN;
  const int sub = lane % LPN;
  const int64_t nw = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
       t < g.npiece; t += nw) {
    const int u = g.piece_row[t];
    const int64_t pb = g.piece_beg[t];
    const int64_t pe = g.piece_end[t];
    const int64_t upos = g.rowptr[u + 1] - (g.ubase[u + 1] - g.ubase[u]);
    const int64_t ebase = g.ubase[u] + (pb - upos);
    const V<T> zu = ldv(Z + static_cast<int64_t>(u) * KB + sub * VEC);
    for (int64_t base = pb; base < pe; base += 64) {
      const int cnt = static_cast<int>(min(static_cast<int64_t>(64), pe - base));
      const int64_t e0 = ebase + (base - pb);
      // this window's neighbours and (when accumulating) their previous R, one
      // coalesced load each; then kInflight neighbour rows of z in flight per lane
      const int myj = (lane < cnt) ? g.col[base + lane] : u;
      const double myr = (accumulate && lane < cnt) ? R[e0 + lane] : 0.0;
      const int steps = (cnt + NPW - 1) / NPW;
      for (int st0 = 0; st0 < steps; st0 += kInflight) {
        V<T> zv[kInflight];
#pragma unroll
        for (int q = 0; q < kInflight; ++q) {
          const int k = (st0 + q) * NPW + grp;
          int j = __shfl(myj, k & 63);
          if (k >= cnt) j = u;
          zv[q] = ldv(Z + static_cast<int64_t>(j) * KB + sub * VEC);
        }
#pragma unroll
        for (int q = 0; q < kInflight; ++q) {
          const int k = (st0 + q) * NPW + grp;
          double d = 0.0;
#pragma unroll
          for (int v = 0; v < VEC; ++v) {
            const double df = static_cast<double>(zu.x[v]) - static_cast<double>(zv[q].x[v]);
            d += df * df;
          }
#pragma unroll
          for (int off = 1; off < LPN; off <<= 1) d += __shfl_xor(d, off);
          const double r0 = __shfl(myr, k & 63);
          if (sub == 0 && k < cnt) R[e0 + k] = accumulate ? r0 + d : d;
        }
      }
    }
  }
}

// p_u = 1 - 1/2 sum_v w_uv R_e(u,v): one wavefront per row, lanes striding the row.
template <typename T>
__global__ __launch_bounds__(kBlock) void k_node_p(DevGraph g, const double* __restrict__ R,
                                                   double* __restrict__ p) {
  const int lane = threadIdx.x & 63;
  const int nw = gridDim.x * kWavesPerBlock;
  const T* __restrict__ w = static_cast<const T*>(g.w);
  for (int i = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6); i < g.n; i += nw) {
    const int64_t b = g.rowptr[i], e = g.rowptr[i + 1];
    double s = 0.0;
    for (int64_t pos = b + lane; pos < e; pos += 64) {
      const double wt = g.weighted ? static_cast<double>(w[pos]) : 1.0;
      s += wt * R[g.eid[pos]];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if (lane == 0) p[i] = 1.0 - 0.5 * s;
  }
}

// kappa_e = 2 (p_u + p_v) / R_e over the edge pieces, one lane per edge.
__global__ __launch_bounds__(kBlock) void k_edge_kappa(DevGraph g, const double* __restrict__ R,
                                                       const double* __restrict__ p,
                                                       double* __restrict__ kappa) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
       t < g.npiece; t += nw) {
    const int u = g.piece_row[t];
    const int64_t pb = g.piece_beg[t], pe = g.piece_end[t];
    const int64_t upos = g.rowptr[u + 1] - (g.ubase[u + 1] - g.ubase[u]);
    const int64_t ebase = g.ubase[u] + (pb - upos);
    const double pu = p[u];
    for (int64_t pos = pb + lane; pos < pe; pos += 64) {
      const int64_t e = ebase + (pos - pb);
      kappa[e] = 2.0 * (pu + p[g.col[pos]]) / R[e];
    }
  }
}

__global__ __launch_bounds__(kBlock) void k_endpoints(DevGraph g, int32_t* __restrict__ eu,
                                                      int32_t* __restrict__ ev) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
       t < g.npiece; t += nw) {
    const int u = g.piece_row[t];
    const int64_t pb = g.piece_beg[t], pe = g.piece_end[t];
    const int64_t upos = g.rowptr[u + 1] - (g.ubase[u + 1] - g.ubase[u]);
    const int64_t ebase = g.ubase[u] + (pb - upos);
    for (int64_t pos = pb + lane; pos < pe; pos += 64) {
      const int64_t e = ebase + (pos - pb);
      eu[e] = u;
      ev[e] = g.col[pos];
    }
  }
}

__global__ __launch_bounds__(kBlock) void k_fill_u32(uint32_t* p, uint32_t v, int64_t count) {
  for (int64_t x = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; x < count;
       x += static_cast<int64_t>(gridDim.x) * kBlock)
    p[x] = v;
}
__global__ __launch_bounds__(kBlock) void k_fill_f64(double* p, double v, int64_t count) {
  for (int64_t x = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; x < count;
       x += static_cast<int64_t>(gridDim.x) * kBlock)
    p[x] = v;
}

// count of entries that are <= 0 or not finite -> out[0]
__global__ __launch_bounds__(kBlock) void k_count_bad(const double* __restrict__ x, int64_t count,
                                                      Tree tree, double* out) {
  __shared__ double s_w[kWavesPerBlock];
  __shared__ double s_in[1], s_out[1];
  double c = 0.0;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    const double v = x[i];
    c += (!(v > 0.0) || !isfinite(v)) ? 1.0 : 0.0;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
  if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = s_w[0];
    for (int w = 1; w < kWavesPerBlock; ++w) s += s_w[w];
    s_in[0] = s;
  }
  __syncthreads();
  if (!tree_reduce<OpSum>(tree, 1, s_in, s_out)) return;
  if (threadIdx.x == 0) out[0] = s_out[0];
}

// dst (n x ncols, row-major) = the first ncols columns of src (n x kb)
template <typename T>
__global__ __launch_bounds__(kBlock) void k_copy_cols(const T* __restrict__ src, int kb,
                                                      T* __restrict__ dst, int ncols, int64_t n) {
  const int64_t total = n * ncols;
  for (int64_t x = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; x < total;
       x += static_cast<int64_t>(gridDim.x) * kBlock) {
    const int64_t i = x / ncols;
    const int c = static_cast<int>(x - i * ncols);
    dst[x] = src[i * kb + c];
  }
}

// ---- sampling (Eqs. 7, 8) --------------------------------------------------------
// Four launches and no device-scope fence: each launch stores one partial per block and
// the next launch reduces the previous one's partials itself.  That reduction is done
// redundantly by every block that needs the total, in the same fixed order in each
// (thread t adds partials t, t + kBlock, ... in turn, then the block adds the threads'
// sums in a fixed tree), so every block sees the same bits.

// Block-wide reduction: every thread passes its value; every thread gets the total.
// Sums (Max = false) are added in a fixed order: wavefronts by xor butterfly, then the
// waves in order.
template <bool Max>
__device__ __forceinline__ double block_total(double v) {
  __shared__ double s_w[kWavesPerBlock];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const double o = __shfl_xor(v, off);
    v = Max ? fmax(v, o) : v + o;
  }
  __syncthreads();  // s_w may still be read by a previous call
  if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = v;
  __syncthreads();
  double t = s_w[0];
#pragma unroll
  for (int w = 1; w < kWavesPerBlock; ++w) t = Max ? fmax(t, s_w[w]) : t + s_w[w];
  return t;
}

// Total of value k of nparts partials of `stride` doubles each, in every thread.
template <bool Max>
__device__ __forceinline__ double reduce_block_parts(const double* __restrict__ part, int nparts,
                                                     int stride, int k) {
  double v = Max ? -INFINITY : 0.0;
  for (int b = threadIdx.x; b < nparts; b += kBlock) {
    const double x = part[static_cast<int64_t>(b) * stride + k];
    v = Max ? fmax(v, x) : v + x;
  }
  return block_total<Max>(v);
}

// Block partials (-kappa_min, kappa_max, 1 if a kappa is not finite) -> part[3 b + 0..2]
__global__ __launch_bounds__(kBlock) void k_minmax(const double* __restrict__ kappa, int64_t m,
                                                   double* __restrict__ part) {
  double nmn = -INFINITY, mx = -INFINITY, bad = 0.0;
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; e < m;
       e += static_cast<int64_t>(gridDim.x) * kBlock) {
    const double k = kappa[e];
    if (isfinite(k)) {
      nmn = fmax(nmn, -k);
      mx = fmax(mx, k);
    } else {
      bad = 1.0;
    }
  }
  nmn = block_total<true>(nmn);
  mx = block_total<true>(mx);
  bad = block_total<true>(bad);
  if (threadIdx.x == 0) {
    double* o = part + 3 * static_cast<int64_t>(blockIdx.x);
    o[0] = nmn;
    o[1] = mx;
    o[2] = bad;
  }
}

// q_u = sum_v (kappa_uv - kappa_min) / (kappa_max - kappa_min + eta) -> pn[u]; block
// partial sums -> part_n[b].  Block 0 also publishes totals[0] = -kappa_min,
// totals[1] = kappa_max and totals[4] = the non-finite flag for the launches after it.
__global__ __launch_bounds__(kBlock) void k_node_w(DevGraph g, const double* __restrict__ kappa,
                                                   double eta, const double* __restrict__ part_mm,
                                                   int nmm, double* totals,
                                                   double* __restrict__ part_n,
                                                   double* __restrict__ pn) {
  const double kmin = -reduce_block_parts<true>(part_mm, nmm, 3, 0);
  const double kmax = reduce_block_parts<true>(part_mm, nmm, 3, 1);
  const double bad = reduce_block_parts<true>(part_mm, nmm, 3, 2);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    totals[0] = -kmin;
    totals[1] = kmax;
    totals[4] = bad;
  }
  const double den = kmax - kmin + eta;
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int nw = gridDim.x * kWavesPerBlock;
  double acc = 0.0;
  for (int i = blockIdx.x * kWavesPerBlock + wv; i < g.n; i += nw) {
    const int64_t b = g.rowptr[i], e = g.rowptr[i + 1];
    double s = 0.0;
    for (int64_t pos = b + lane; pos < e; pos += 64) s += (kappa[g.eid[pos]] - kmin) / den;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if (lane == 0) pn[i] = s;
    acc += s;  // identical in every lane
  }
  // one lane per wave carries the wave's sum into the block total
  acc = block_total<false>(lane == 0 ? acc : 0.0);
  if (threadIdx.x == 0) part_n[blockIdx.x] = acc;
}

// q_e = sqrt(max(2 kappa_max - kappa_e, 0)) + 1 -> pe[e]; block partial sums -> part_e[b]
__global__ __launch_bounds__(kBlock) void k_edge_w(const double* __restrict__ kappa, int64_t m,
                                                   const double* totals,
                                                   double* __restrict__ part_e,
                                                   double* __restrict__ pe) {
  const double kmax = totals[1];
  double acc = 0.0;
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; e < m;
       e += static_cast<int64_t>(gridDim.x) * kBlock) {
    const double q = sqrt(fmax(2.0 * kmax - kappa[e], 0.0)) + 1.0;
    pe[e] = q;
    acc += q;
  }
  acc = block_total<false>(acc);
  if (threadIdx.x == 0) part_e[blockIdx.x] = acc;
}

// P_u = q_u / sum q, P_e = q_e / sum q_e (the sums reduced from the block partials of the
// two previous launches); block 0 publishes them as totals[2] and totals[3].
__global__ __launch_bounds__(kBlock) void k_normalise(DevGraph g, double* totals,
                                                      const double* __restrict__ part_n, int nn,
                                                      const double* __restrict__ part_e, int ne,
                                                      double inv_nonisolated,
                                                      double* __restrict__ pn,
                                                      double* __restrict__ pe) {
  const double tn = reduce_block_parts<false>(part_n, nn, 1, 0);
  const double te = reduce_block_parts<false>(part_e, ne, 1, 0);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    totals[2] = tn;
    totals[3] = te;
  }
  // a NaN or infinite kappa (flagged by k_minmax) makes every probability NaN, rather
  // than letting the NaN weight fall back to the uniform distribution
  const bool bad = totals[4] != 0.0;
  const double nan = __longlong_as_double(0x7ff8000000000000ll);
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < g.n; i += stride) {
    if (bad) {
      pn[i] = nan;
    } else if (tn > 0.0) {
      pn[i] = pn[i] / tn;
    } else {
      pn[i] = (g.rowptr[i + 1] > g.rowptr[i]) ? inv_nonisolated : 0.0;
    }
  }
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; e < g.m; e += stride)
    pe[e] = bad ? nan : pe[e] / te;
}

// ---------------------------------------------------------------------------------
int grid_for(int64_t items, int64_t per_block, int cap) {
  int64_t g = (items + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return static_cast<int>(g);
}

}  // namespace

// ---- launchers --------------------------------------------------------------------
// The stream argument of hipLaunchKernelGGL is passed through a small wrapper so every
// launch lands on the caller's stream.
#define ERC_LAUNCH(kernel, grid, stream, ...) \
  hipLaunchKernelGGL(kernel, dim3(grid), dim3(kBlock), 0, stream, __VA_ARGS__)

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  ERC_LAUNCH(k_fill_u32, grid_for(count, kBlock, 4096), s, p, v, count);
  return hipGetLastError();
}
hipError_t launch_fill_f64(double* p, double v, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  ERC_LAUNCH(k_fill_f64, grid_for(count, kBlock, 4096), s, p, v, count);
  return hipGetLastError();
}

template <int KB>
static hipError_t fin_rhs_launch(const FinArgs& f, hipStream_t s) {
  ERC_LAUNCH((k_fin_rhs<KB>), (f.nparts + kTreeFan - 1) / kTreeFan, s, f);
  return hipGetLastError();
}

template <int KB>
static hipError_t fin_iter_launch(const IterArgs& f, hipStream_t s) {
  const int np = f.nparts_s > f.nparts_u ? f.nparts_s : f.nparts_u;
  // short partial sets are summed by k_fin_col directly (one launch instead of two)
  const int nsum = np > kFinDirectMax ? (np + kTreeFan - 1) / kTreeFan : 0;
  if (nsum > 0) {
    const int nval = (f.pc ? 2 : 1) * KB + 3 * KB;
    ERC_LAUNCH((k_fin_sum<KB>), dim3(nsum, (nval + 63) / 64), s, f);
  }
  ERC_LAUNCH((k_fin_col<KB>), KB, s, f, nsum);
  return hipGetLastError();
}

static hipError_t fin_rhs_dispatch(int kb, const FinArgs& f, hipStream_t s) {
  switch (kb) {
    case 8: return fin_rhs_launch<8>(f, s);
    case 16: return fin_rhs_launch<16>(f, s);
    case 32: return fin_rhs_launch<32>(f, s);
    case 64: return fin_rhs_launch<64>(f, s);
    case 128: return fin_rhs_launch<128>(f, s);
    case 256: return fin_rhs_launch<256>(f, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_fin_iter(const DevGraph& g, const Work& w, int mode, hipStream_t s) {
  IterArgs f;
  f.part_s = w.part;
  f.nparts_s = g.grid;
  f.part_u = w.part_u;
  f.nparts_u = w.grid_upd;
  f.tree = w.tree;
  f.cs = w.cs;
  f.mega_dots = w.mega_dots;
  f.nmega = g.nmega;
  f.mode = mode;
  f.pc = w.pc;
  switch (w.kb) {
    case 8: return fin_iter_launch<8>(f, s);
    case 16: return fin_iter_launch<16>(f, s);
    case 32: return fin_iter_launch<32>(f, s);
    case 64: return fin_iter_launch<64>(f, s);
    case 128: return fin_iter_launch<128>(f, s);
    case 256: return fin_iter_launch<256>(f, s);
  }
  return hipErrorInvalidValue;
}

template <typename T, int KB>
static hipError_t rhs_t(const RhsArgs& a, int grid, hipStream_t s) {
  if (a.minv != nullptr) {
    ERC_LAUNCH((k_rhs<T, KB, true>), grid, s, a);
  } else {
    if constexpr (KB <= 64) {
      if (!a.g.weighted) {
        ERC_LAUNCH((k_rhs_unit<T, KB>), grid, s, a);
        return hipGetLastError();
      }
    }
    ERC_LAUNCH((k_rhs<T, KB, false>), grid, s, a);
  }
  return hipGetLastError();
}

static hipError_t rhs_dispatch(erc_dtype dt, int kb, const RhsArgs& a, int grid, hipStream_t s) {
  if (dt == ERC_F32) {
    switch (kb) {
      case 16: return rhs_t<float, 16>(a, grid, s);
      case 32: return rhs_t<float, 32>(a, grid, s);
      case 64: return rhs_t<float, 64>(a, grid, s);
      case 128: return rhs_t<float, 128>(a, grid, s);
      case 256: return rhs_t<float, 256>(a, grid, s);
    }
  } else {
    switch (kb) {
      case 8: return rhs_t<double, 8>(a, grid, s);
      case 16: return rhs_t<double, 16>(a, grid, s);
      case 32: return rhs_t<double, 32>(a, grid, s);
      case 64: return rhs_t<double, 64>(a, grid, s);
      case 128: return rhs_t<double, 128>(a, grid, s);
    }
  }
  return hipErrorInvalidValue;
}

hipError_t launch_rhs(const DevGraph& g, const Work& w, erc_dtype dt, int K, int col0, int ncols,
                      uint64_t base, double inv_sqrt_k, double tol, hipStream_t s) {
  RhsArgs a;
  a.g = g;
  a.z = w.z;
  a.r = w.r;
  a.p = w.p;
  a.col0 = col0;
  a.ncols = ncols;
  a.words = static_cast<uint64_t>((K + 63) / 64);
  a.base = base;
  a.inv_sqrt_k = inv_sqrt_k;
  a.part = w.part;
  a.minv = w.pc ? w.minv : nullptr;
  hipError_t e = rhs_dispatch(dt, w.kb, a, w.grid_rhs, s);
  if (e != hipSuccess) return e;
  FinArgs f;
  f.part = w.part;
  f.nparts = w.grid_rhs;
  f.tree = w.tree;
  f.cs = w.cs;
  f.tol2 = tol * tol;
  f.ncols = ncols;
  f.pc = w.pc;
  return fin_rhs_dispatch(w.kb, f, s);
}

template <typename T, int LPN>
static hipError_t spmm_launch(const SpmmArgs& a, hipStream_t s) {
  if (a.g.weighted)
    ERC_LAUNCH((k_spmm<T, LPN, true>), a.g.grid, s, a);
  else
    ERC_LAUNCH((k_spmm<T, LPN, false>), a.g.grid, s, a);
  if (a.g.nmega > 0) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_mega_fin<T, LPN>), dim3(a.g.nmega), dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_spmm(const DevGraph& g, const Work& w, erc_dtype dt, double delta, const void* p,
                       const void* r, void* q, const int32_t* gate, hipStream_t s) {
  SpmmArgs a;
  a.g = g;
  a.p = p;
  a.r = r;
  a.q = q;
  a.chunkbuf = w.chunkbuf;
  a.mega_dots = w.mega_dots;
  a.part = w.part;
  a.gate = gate;
  a.delta = delta;
  a.minv = w.pc ? w.minv : nullptr;
  const int lpn = (dt == ERC_F32) ? w.kb / 4 : w.kb / 2;
  if (dt == ERC_F32) {
    switch (lpn) {
      case 4: return spmm_launch<float, 4>(a, s);
      case 8: return spmm_launch<float, 8>(a, s);
      case 16: return spmm_launch<float, 16>(a, s);
      case 32: return spmm_launch<float, 32>(a, s);
      case 64: return spmm_launch<float, 64>(a, s);
    }
  } else {
    switch (lpn) {
      case 4: return spmm_launch<double, 4>(a, s);
      case 8: return spmm_launch<double, 8>(a, s);
      case 16: return spmm_launch<double, 16>(a, s);
      case 32: return spmm_launch<double, 32>(a, s);
      case 64: return spmm_launch<double, 64>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

template <typename T, int CG>
static hipError_t upd_launch(const UpdArgs& a, int grid, hipStream_t s) {
  if (a.minv != nullptr)
    ERC_LAUNCH((k_update<T, CG, true>), grid, s, a);
  else
    ERC_LAUNCH((k_update<T, CG, false>), grid, s, a);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_minv(const double* __restrict__ deg, double delta,
                                                 T* __restrict__ minv, int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n; i += stride)
    minv[i] = static_cast<T>(1.0 / (deg[i] + delta));
}

hipError_t launch_minv(const DevGraph& g, const Work& w, erc_dtype dt, double delta, hipStream_t s) {
  const int grid = grid_for(g.n, kBlock, 4096);
  if (dt == ERC_F32)
    ERC_LAUNCH(k_minv<float>, grid, s, g.deg, delta, static_cast<float*>(w.minv),
               static_cast<int64_t>(g.n));
  else
    ERC_LAUNCH(k_minv<double>, grid, s, g.deg, delta, static_cast<double*>(w.minv),
               static_cast<int64_t>(g.n));
  return hipGetLastError();
}

hipError_t launch_update(const DevGraph& g, const Work& w, erc_dtype dt, hipStream_t s) {
  UpdArgs a;
  a.z = w.z;
  a.r = w.r;
  a.p = w.p;
  a.q = w.q;
  a.minv = w.pc ? w.minv : nullptr;
  const int vec = (dt == ERC_F32) ? 4 : 2;
  a.nvec = static_cast<int64_t>(g.n) * w.kb / vec;
  a.part = w.part_u;
  a.cs = w.cs;
  const int cg = w.kb / vec;
  const int grid = w.grid_upd;
  hipError_t e = hipErrorInvalidValue;
  if (dt == ERC_F32) {
    switch (cg) {
      case 4: e = upd_launch<float, 4>(a, grid, s); break;
      case 8: e = upd_launch<float, 8>(a, grid, s); break;
      case 16: e = upd_launch<float, 16>(a, grid, s); break;
      case 32: e = upd_launch<float, 32>(a, grid, s); break;
      case 64: e = upd_launch<float, 64>(a, grid, s); break;
    }
  } else {
    switch (cg) {
      case 4: e = upd_launch<double, 4>(a, grid, s); break;
      case 8: e = upd_launch<double, 8>(a, grid, s); break;
      case 16: e = upd_launch<double, 16>(a, grid, s); break;
      case 32: e = upd_launch<double, 32>(a, grid, s); break;
      case 64: e = upd_launch<double, 64>(a, grid, s); break;
    }
  }
  return e;
}

template <typename T, int LPN>
static hipError_t ed_launch(const DevGraph& g, const void* z, double* R, int acc, int grid,
                            hipStream_t s) {
  ERC_LAUNCH((k_edge_dist<T, LPN>), grid, s, g, static_cast<const T*>(z), R, acc);
  return hipGetLastError();
}

hipError_t launch_edge_dist(const DevGraph& g, const Work& w, erc_dtype dt, double* R,
                            int accumulate, hipStream_t s) {
  if (g.npiece == 0) return hipSuccess;
  const int lpn = (dt == ERC_F32) ? w.kb / 4 : w.kb / 2;
  const int grid = w.grid_ed;
  if (dt == ERC_F32) {
    switch (lpn) {
      case 4: return ed_launch<float, 4>(g, w.z, R, accumulate, grid, s);
      case 8: return ed_launch<float, 8>(g, w.z, R, accumulate, grid, s);
      case 16: return ed_launch<float, 16>(g, w.z, R, accumulate, grid, s);
      case 32: return ed_launch<float, 32>(g, w.z, R, accumulate, grid, s);
      case 64: return ed_launch<float, 64>(g, w.z, R, accumulate, grid, s);
    }
  } else {
    switch (lpn) {
      case 4: return ed_launch<double, 4>(g, w.z, R, accumulate, grid, s);
      case 8: return ed_launch<double, 8>(g, w.z, R, accumulate, grid, s);
      case 16: return ed_launch<double, 16>(g, w.z, R, accumulate, grid, s);
      case 32: return ed_launch<double, 32>(g, w.z, R, accumulate, grid, s);
      case 64: return ed_launch<double, 64>(g, w.z, R, accumulate, grid, s);
    }
  }
  return hipErrorInvalidValue;
}

hipError_t launch_count_bad(const double* x, int64_t count, const Work& w, hipStream_t s) {
  const int grid = grid_for(count, kBlock * 16, 2048);
  ERC_LAUNCH(k_count_bad, grid, s, x, count, w.tree, w.out);
  return hipGetLastError();
}

hipError_t launch_copy_cols(const DevGraph& g, const void* src, int kb, erc_dtype dt, int ncols,
                            void* dst, hipStream_t s) {
  const int64_t total = static_cast<int64_t>(g.n) * ncols;
  if (total == 0) return hipSuccess;
  const int grid = grid_for(total, kBlock * 4, 8192);
  if (dt == ERC_F32)
    ERC_LAUNCH((k_copy_cols<float>), grid, s, static_cast<const float*>(src), kb,
               static_cast<float*>(dst), ncols, static_cast<int64_t>(g.n));
  else
    ERC_LAUNCH((k_copy_cols<double>), grid, s, static_cast<const double*>(src), kb,
               static_cast<double*>(dst), ncols, static_cast<int64_t>(g.n));
  return hipGetLastError();
}

hipError_t launch_node_p(const DevGraph& g, erc_dtype dt, const double* R, double* p,
                         hipStream_t s) {
  const int grid = grid_for(g.n, kWavesPerBlock, 8192);
  if (dt == ERC_F32)
    ERC_LAUNCH(k_node_p<float>, grid, s, g, R, p);
  else
    ERC_LAUNCH(k_node_p<double>, grid, s, g, R, p);
  return hipGetLastError();
}

hipError_t launch_edge_kappa(const DevGraph& g, const double* R, const double* p, double* kappa,
                             hipStream_t s) {
  if (g.npiece == 0) return hipSuccess;
  const int grid = grid_for(g.npiece, kWavesPerBlock, 8192);
  ERC_LAUNCH(k_edge_kappa, grid, s, g, R, p, kappa);
  return hipGetLastError();
}

hipError_t launch_endpoints(const DevGraph& g, int32_t* u, int32_t* v, hipStream_t s) {
  if (g.npiece == 0) return hipSuccess;
  const int grid = grid_for(g.npiece, kWavesPerBlock, 8192);
  ERC_LAUNCH(k_endpoints, grid, s, g, u, v);
  return hipGetLastError();
}

hipError_t launch_eids(const DevGraph& g, int32_t* out, hipStream_t s) {
  if (g.nnz == 0) return hipSuccess;
  return hipMemcpyAsync(out, g.eid, g.nnz * sizeof(int32_t), hipMemcpyDeviceToDevice, s);
}

hipError_t launch_sampling(const DevGraph& g, const double* kappa, double eta, int64_t nonisolated,
                           const SampleWork& sw, double* pn, double* pe, hipStream_t s) {
  // k_minmax and k_edge_w on sw.grid blocks, k_node_w on up to sw.grid blocks of 32 rows;
  // the edge partials reuse the min/max partials' space (k_node_w has read them by then)
  const int grid = sw.grid;
  ERC_LAUNCH(k_minmax, grid, s, kappa, g.m, sw.part_mm);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int gn = grid_for(g.n, kWavesPerBlock * 8, sw.grid);
  ERC_LAUNCH(k_node_w, gn, s, g, kappa, eta, sw.part_mm, grid, sw.totals, sw.part_n, pn);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  ERC_LAUNCH(k_edge_w, grid, s, kappa, g.m, sw.totals, sw.part_mm, pe);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  const double inv = nonisolated > 0 ? 1.0 / static_cast<double>(nonisolated) : 0.0;
  const int gz = grid_for(g.n > g.m ? g.n : g.m, kBlock * 4, 4096);
  ERC_LAUNCH(k_normalise, gz, s, g, sw.totals, sw.part_n, gn, sw.part_mm, grid, inv, pn, pe);
  return hipGetLastError();
}

}  // namespace erc
