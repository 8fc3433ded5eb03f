// Host side of the resistance-curvature library: graph validation and canonical edge
// numbering, the device work plan, buffer layouts, and the column-block CG driver of
// Algorithm 1 (streamed right-hand sides, batched CG, edge-block accumulation).
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <exception>
#include <new>
#include <numeric>
#include <string>
#include <thread>
#include <vector>

#include "erc_common.h"

using namespace erc;

namespace {

thread_local std::string g_last_error;

erc_status fail(erc_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

// The C ABI throws nothing: a failed host allocation or thread start inside a call
// becomes ERC_E_HOST with a message.
template <typename F>
erc_status guarded(F&& f) {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    return fail(ERC_E_HOST, "host memory allocation failed");
  } catch (const std::exception& e) {
    return fail(ERC_E_HOST, std::string("host error: ") + e.what());
  } catch (...) {
    return fail(ERC_E_HOST, "host error");
  }
}

#define ERC_HIP(call)                                                                  \
  do {                                                                                 \
    hipError_t e_ = (call);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(ERC_E_DEVICE, std::string(#call) + ": " + hipGetErrorString(e_));   \
  } while (0)

// Per-row cost of the SpMM plan, in units of one neighbour.
constexpr double kRowCost = 8.0;
// Cost per wave: at least 64 units; on small graphs up to 192 while that leaves 2048
// waves or more (two per SIMD), rather than spreading them over the whole grid cap
// (20k-node workload 2.17 -> 1.9 ms per step, 170k-node 337 -> 325 ms; the 2000-node
// one keeps 64, as a larger share leaves too few waves).
constexpr double kMinShare = 64.0;
constexpr double kSmallShare = 192.0;
constexpr double kMinWaves = 2048.0;
// SpMM grid (blocks of 4 waves): 8192 blocks, or up to 16384 on graphs with more than
// 32 rows per wave at 8192 (the 2.4M-node workload: 4.45 -> 4.38 ms per launch; the
// 170k- and 230k-node ones are slower on the larger grid).
constexpr int kBaseSpmmGrid = 8192;
constexpr int kMaxSpmmGrid = 16384;
constexpr int64_t kRowsPerWave = 32;
static_assert((kMaxSpmmGrid + kTreeFan - 1) / kTreeFan <= kMaxTreeGrid,
              "level-1 sums of the SpMM partials must fit the tree buffers");
// Longest edge piece of the per-edge kernels.
constexpr int64_t kPiece = 1024;
// Grid caps of the other kernels.
constexpr int kMaxGridRhs = 8192;
// The update streams seven n x kb arrays; 32768 blocks (about 4.6 vectors per thread
// and array on the 2.4M-node graph) ran it 5% faster than 8192 or 2048.  Its partial
// sets then hold up to 32768 entries, which the finishing step folds into at most
// 1024 level-1 sums (within kMaxTreeGrid).
constexpr int kMaxGridUpd = 32768;
static_assert((kMaxGridUpd + kTreeFan - 1) / kTreeFan <= kMaxTreeGrid,
              "level-1 sums of the update partials must fit the tree buffers");
constexpr int kMaxGridEd = 8192;
// Grid cap of the sampling passes: their scratch is 4 doubles per block plus 64 bytes,
// 33 KB at the cap, inside the fixed scratch of erc_sampling_probs_static.
constexpr int kSampleGrid = 1024;
static_assert(int64_t{kSampleGrid} * 4 * 8 + 3 * 256 <= static_cast<int64_t>(kStaticScratchBytes),
              "the sampling scratch at the grid cap must fit the fixed scratch");
constexpr int kDefaultCheck = 16;
// Neighbour-row bytes one SpMM gathers (nnz * kb * element size) above which each CG
// iteration also enqueues the early stopping test: 4 GB is about half a millisecond of
// gathers, against a few microseconds per extra launch and iteration.
constexpr double kFin2MinGather = 4e9;

size_t dsize(erc_dtype t) { return t == ERC_F32 ? 4 : 8; }
int64_t align_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

// Sizes that depend only on (n, nnz): the plan shape and upper bounds of its lists.
struct Shape {
  int64_t n, nnz, m;
  double share;      // target cost per wave
  int waves, grid;   // SpMM wavefronts and blocks
  int64_t heavy;     // rows with degree above this are block tasks
  int64_t chunk;     // block tasks are at most this long
  int64_t ntask_max, nmega_max, nslot_max, npiece_max;
};

Shape make_shape(int64_t n, int64_t nnz) {
  Shape s{};
  s.n = n;
  s.nnz = nnz;
  s.m = nnz / 2;
  const double total = static_cast<double>(nnz) + kRowCost * static_cast<double>(n);
  const int64_t grid_cap = std::min<int64_t>(
      kMaxSpmmGrid, std::max<int64_t>(kBaseSpmmGrid, n / (kRowsPerWave * kWavesPerBlock)));
  s.share = std::max({kMinShare, std::min(kSmallShare, total / kMinWaves),
                      total / static_cast<double>(grid_cap * kWavesPerBlock)});
  int64_t waves = static_cast<int64_t>(std::ceil(total / s.share));
  waves = std::max<int64_t>(kWavesPerBlock, align_up(waves, kWavesPerBlock));
  waves = std::min<int64_t>(waves, grid_cap * kWavesPerBlock);
  s.waves = static_cast<int>(waves);
  s.grid = s.waves / kWavesPerBlock;
  // Rows up to 1024 entries stay with the wavefronts (a block task costs a block-wide
  // reduction), and a block task covers up to 4096 entries: on graphs with a small
  // share (the 170k-node workload: 116 entries per wave) floors of 256 and 1024 made
  // the SpMM 0.269 ms against 0.181 ms with these.
  s.heavy = std::max<int64_t>(1024, static_cast<int64_t>(2.0 * s.share));
  s.chunk = std::max<int64_t>(4096, static_cast<int64_t>(8.0 * s.share));
  s.ntask_max = nnz / s.heavy + nnz / s.chunk + 1;
  s.nmega_max = nnz / s.chunk + 1;
  s.nslot_max = 2 * (nnz / s.chunk) + 1;
  s.npiece_max = n + s.m / kPiece + 1;
  return s;
}

// Byte layout of the graph buffer.
struct GraphLayout {
  int64_t rowptr, col, w, eid, sw, ubase, deg, light, wave_lo, task_row, task_mega, task_chunk,
      task_beg, task_end, mega_row, mega_nchunk, mega_chunk0, piece_row, piece_beg, piece_end, total;
};

GraphLayout graph_layout(const Shape& s, bool weighted, erc_dtype dt) {
  GraphLayout L{};
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    const int64_t at = off;
    off = align_up(off + std::max<int64_t>(bytes, 0), 256);
    return at;
  };
  L.rowptr = take((s.n + 1) * 8);
  L.col = take(s.nnz * 4);
  L.w = take(weighted ? s.nnz * static_cast<int64_t>(dsize(dt)) : 0);
  L.eid = take(s.nnz * 4);
  L.sw = take(s.m * 8);
  L.ubase = take((s.n + 1) * 8);
  L.deg = take(s.n * 8);
  L.light = take(s.n * static_cast<int64_t>(sizeof(LightRow)));
  L.wave_lo = take((static_cast<int64_t>(s.waves) + 1) * 4);
  L.task_row = take(s.ntask_max * 4);
  L.task_mega = take(s.ntask_max * 4);
  L.task_chunk = take(s.ntask_max * 4);
  L.task_beg = take(s.ntask_max * 8);
  L.task_end = take(s.ntask_max * 8);
  L.mega_row = take(s.nmega_max * 4);
  L.mega_nchunk = take(s.nmega_max * 4);
  L.mega_chunk0 = take(s.nmega_max * 4);
  L.piece_row = take(s.npiece_max * 4);
  L.piece_beg = take(s.npiece_max * 8);
  L.piece_end = take(s.npiece_max * 8);
  L.total = off;
  return L;
}

erc_status check_desc(const erc_graph_desc* d) {
  if (d == nullptr) return fail(ERC_E_INVALID_ARG, "graph description is NULL");
  if (d->n <= 0 || d->n >= (int64_t(1) << 31))
    return fail(ERC_E_INVALID_ARG, "n must be in [1, 2^31)");
  if (d->rowptr == nullptr) return fail(ERC_E_INVALID_ARG, "rowptr is NULL");
  if (d->solve_dtype != ERC_F32 && d->solve_dtype != ERC_F64)
    return fail(ERC_E_INVALID_ARG, "solve_dtype must be ERC_F32 or ERC_F64");
  if (d->w != nullptr && d->w_dtype != ERC_F32 && d->w_dtype != ERC_F64)
    return fail(ERC_E_INVALID_ARG, "w_dtype must be ERC_F32 or ERC_F64");
  const int64_t nnz = d->rowptr[d->n];
  if (d->rowptr[0] != 0) return fail(ERC_E_INVALID_GRAPH, "rowptr[0] must be 0");
  if (nnz < 0 || nnz >= (int64_t(1) << 31))
    return fail(ERC_E_INVALID_GRAPH, "nnz must be in [0, 2^31)");
  if (nnz > 0 && d->col == nullptr) return fail(ERC_E_INVALID_ARG, "col is NULL");
  return ERC_OK;
}

// Canonical form of a validated graph.
struct Canon {
  int64_t m = 0;
  std::vector<int32_t> eid;    // nnz
  std::vector<double> sw;      // m
  std::vector<int64_t> ubase;  // n+1
  std::vector<double> deg;     // n: sum_j w_ij in fp64, CSR order
  std::vector<unsigned char> wstore;  // nnz weights in the working precision
};

// Rows [0, n) split into `parts` contiguous ranges of about equal stored entries, each
// handled by its own thread (one thread for small graphs).
template <typename F>
void for_row_ranges(const int64_t* rp, int64_t n, F&& body) {
  const int64_t nnz = rp[n];
  int parts = 1;
  if (nnz >= (int64_t(1) << 20)) {
    const unsigned hc = std::thread::hardware_concurrency();
    parts = static_cast<int>(std::min<unsigned>(hc == 0 ? 1u : hc, 16u));
  }
  std::vector<int64_t> cut(parts + 1, n);
  cut[0] = 0;
  for (int t = 1; t < parts; ++t)
    cut[t] = std::upper_bound(rp, rp + n + 1, nnz * t / parts) - rp - 1;
  for (int t = 1; t <= parts; ++t) cut[t] = std::max(cut[t], cut[t - 1]);
  if (parts == 1) {
    body(0, int64_t(0), n);
    return;
  }
  // an exception in a worker (a failed allocation) is rethrown here, after all joined
  std::vector<std::exception_ptr> exc(parts);
  std::vector<std::thread> th;
  auto run = [&](int t) {
    try {
      body(t, cut[t], cut[t + 1]);
    } catch (...) {
      exc[t] = std::current_exception();
    }
  };
  try {
    for (int t = 0; t < parts; ++t) th.emplace_back(run, t);
  } catch (...) {
    for (auto& x : th) x.join();
    throw;
  }
  for (auto& x : th) x.join();
  for (auto& e : exc)
    if (e) std::rethrow_exception(e);
}

// The first problem a worker finds in its row range; the caller reports the one in
// the lowest row (workers never touch the thread-local error message).
struct RowError {
  int64_t row = INT64_MAX;
  std::string msg;
  void set(int64_t r, std::string m) {
    if (r < row) {
      row = r;
      msg = std::move(m);
    }
  }
};

template <typename WT>
erc_status sweep(const erc_graph_desc* d, const WT* w, Canon* out) {
  const int64_t n = d->n;
  const int64_t* rp = d->rowptr;
  const int32_t* col = d->col;
  const int64_t nnz = rp[n];
  for (int64_t i = 0; i < n; ++i)
    if (rp[i + 1] < rp[i]) return fail(ERC_E_INVALID_GRAPH, "rowptr decreases at row " + std::to_string(i));
  if (nnz % 2 != 0) return fail(ERC_E_INVALID_GRAPH, "odd number of stored entries: not symmetric");
  if (out) {
    out->eid.assign(nnz, -1);
    out->ubase.assign(n + 1, 0);
    out->deg.assign(n, 0.0);
  }
  // 1. per row: indices in range, no self-loop, strictly ascending, weights finite and
  //    positive; the number of upper entries (j > i) and d_i in CSR order
  std::vector<int64_t> nup(n, 0);
  std::vector<RowError> err1(16);
  for_row_ranges(rp, n, [&](int t, int64_t r0, int64_t r1) {
    RowError& e = err1[t];
    for (int64_t i = r0; i < r1 && e.row == INT64_MAX; ++i) {
      int64_t up = 0;
      double dsum = 0.0;
      for (int64_t pos = rp[i]; pos < rp[i + 1]; ++pos) {
        const int64_t j = col[pos];
        if (j < 0 || j >= n) {
          e.set(i, "column index out of range in row " + std::to_string(i));
          break;
        }
        if (j == i) {
          e.set(i, "self-loop at node " + std::to_string(i));
          break;
        }
        if (pos > rp[i] && col[pos - 1] >= j) {
          e.set(i, "columns not strictly ascending in row " + std::to_string(i));
          break;
        }
        if (w != nullptr) {
          const WT x = w[pos];
          if (!(std::isfinite(static_cast<double>(x)) && x > WT(0))) {
            e.set(i, "weight must be finite and > 0 at entry (" + std::to_string(i) + ", " +
                         std::to_string(j) + ")");
            break;
          }
        }
        dsum += (w != nullptr) ? static_cast<double>(w[pos]) : 1.0;
        up += (j > i) ? 1 : 0;
      }
      nup[i] = up;
      if (out) out->deg[i] = dsum;
    }
  });
  {
    RowError first;
    for (const RowError& e : err1) first.set(e.row, e.msg);
    if (first.row != INT64_MAX) return fail(ERC_E_INVALID_GRAPH, first.msg);
  }
  // 2. canonical edge ids: the upper entries in row-major order
  std::vector<int64_t> ub(n + 1, 0);
  for (int64_t i = 0; i < n; ++i) ub[i + 1] = ub[i] + nup[i];
  const int64_t m = ub[n];
  if (m * 2 != nnz) return fail(ERC_E_INVALID_GRAPH, "structure is not symmetric");
  if (out) {
    std::copy(ub.begin(), ub.end(), out->ubase.begin());
    out->sw.assign(m, 0.0);
  }
  // 3. every upper entry (i, j) has its mirror (j, i) with the same weight; as there are
  //    as many lower entries as upper ones, the mirrors are all of them.  Each edge id
  //    slot is written once, by the thread of the upper entry's row.
  std::vector<RowError> err3(16);
  for_row_ranges(rp, n, [&](int t, int64_t r0, int64_t r1) {
    RowError& e = err3[t];
    for (int64_t i = r0; i < r1 && e.row == INT64_MAX; ++i) {
      const int64_t first_up = rp[i + 1] - nup[i];
      for (int64_t pos = first_up; pos < rp[i + 1]; ++pos) {
        const int64_t j = col[pos];
        const int32_t* lo = col + rp[j];
        const int32_t* hi = col + rp[j + 1];
        const int32_t* it = std::lower_bound(lo, hi, static_cast<int32_t>(i));
        if (it == hi || *it != i) {
          e.set(i, "structure is not symmetric at entry (" + std::to_string(i) + ", " +
                       std::to_string(j) + ")");
          break;
        }
        const int64_t tpos = it - col;
        if (w != nullptr && !(w[tpos] == w[pos])) {
          e.set(i, "weights not symmetric at entry (" + std::to_string(i) + ", " +
                       std::to_string(j) + ")");
          break;
        }
        if (out) {
          const int64_t id = ub[i] + (pos - first_up);
          out->eid[pos] = static_cast<int32_t>(id);
          out->eid[tpos] = static_cast<int32_t>(id);
          out->sw[id] = (w != nullptr) ? std::sqrt(static_cast<double>(w[pos])) : 1.0;
        }
      }
    }
  });
  {
    RowError first;
    for (const RowError& e : err3) first.set(e.row, e.msg);
    if (first.row != INT64_MAX) return fail(ERC_E_INVALID_GRAPH, first.msg);
  }
  if (out) out->m = m;
  return ERC_OK;
}

erc_status canonicalise(const erc_graph_desc* d, Canon* out) {
  erc_status st = check_desc(d);
  if (st != ERC_OK) return st;
  if (d->w == nullptr) return sweep<float>(d, nullptr, out);
  if (d->w_dtype == ERC_F32) return sweep<float>(d, static_cast<const float*>(d->w), out);
  return sweep<double>(d, static_cast<const double*>(d->w), out);
}

// Host copy of the work plan.
struct Plan {
  std::vector<int32_t> light, wave_lo;
  std::vector<int32_t> task_row, task_mega, task_chunk;
  std::vector<int64_t> task_beg, task_end;
  std::vector<int32_t> mega_row, mega_nchunk, mega_chunk0;
  int32_t nslot = 0;
  std::vector<int32_t> piece_row;
  std::vector<int64_t> piece_beg, piece_end;
};

void build_plan(const erc_graph_desc* d, const Canon& c, const Shape& s, Plan* P) {
  const int64_t n = d->n;
  const int64_t* rp = d->rowptr;
  // long rows -> block tasks, longest first; very long rows are split into chunks
  std::vector<int32_t> heavy;
  for (int64_t i = 0; i < n; ++i)
    if (rp[i + 1] - rp[i] > s.heavy) heavy.push_back(static_cast<int32_t>(i));
  std::stable_sort(heavy.begin(), heavy.end(), [&](int32_t a, int32_t b) {
    return (rp[a + 1] - rp[a]) > (rp[b + 1] - rp[b]);
  });
  struct Task { int32_t row, mega, chunk; int64_t beg, end; };
  std::vector<Task> tasks;
  for (int32_t i : heavy) {
    const int64_t b = rp[i], e = rp[i + 1];
    const int64_t nch = (e - b + s.chunk - 1) / s.chunk;
    if (nch == 1) {
      tasks.push_back({i, -1, 0, b, e});
    } else {
      const int32_t mh = static_cast<int32_t>(P->mega_nchunk.size());
      P->mega_row.push_back(i);
      P->mega_nchunk.push_back(static_cast<int32_t>(nch));
      P->mega_chunk0.push_back(P->nslot);
      P->nslot += static_cast<int32_t>(nch);
      for (int64_t k = 0; k < nch; ++k)
        tasks.push_back({i, mh, static_cast<int32_t>(k), b + k * s.chunk, std::min(e, b + (k + 1) * s.chunk)});
    }
  }
  std::stable_sort(tasks.begin(), tasks.end(), [](const Task& a, const Task& b) {
    return (a.end - a.beg) > (b.end - b.beg);
  });
  std::vector<double> hcost(s.grid, 0.0);
  for (size_t t = 0; t < tasks.size(); ++t) {
    P->task_row.push_back(tasks[t].row);
    P->task_mega.push_back(tasks[t].mega);
    P->task_chunk.push_back(tasks[t].chunk);
    P->task_beg.push_back(tasks[t].beg);
    P->task_end.push_back(tasks[t].end);
    hcost[t % s.grid] += static_cast<double>(tasks[t].end - tasks[t].beg) + kRowCost;
  }
  // short rows -> contiguous per-wave ranges balanced by cost, leaving room for tasks
  double light_total = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t dg = rp[i + 1] - rp[i];
    if (dg <= s.heavy) {
      P->light.push_back(static_cast<int32_t>(i));
      light_total += static_cast<double>(dg) + kRowCost;
    }
  }
  const int W = s.waves;
  std::vector<double> budget(W);
  double bsum = 0.0;
  for (int w = 0; w < W; ++w) {
    budget[w] = std::max(0.0, s.share - hcost[w / kWavesPerBlock] / kWavesPerBlock);
    bsum += budget[w];
  }
  for (int w = 0; w < W; ++w)
    budget[w] = bsum > 0.0 ? budget[w] * (light_total / bsum) : light_total / W;
  P->wave_lo.assign(W + 1, 0);
  const int64_t nl = static_cast<int64_t>(P->light.size());
  int w = 0;
  double cum = 0.0, tnext = budget[0];
  for (int64_t k = 0; k < nl; ++k) {
    const int32_t i = P->light[k];
    const double cost = static_cast<double>(rp[i + 1] - rp[i]) + kRowCost;
    const double mid = cum + 0.5 * cost;
    while (w < W - 1 && mid >= tnext) {
      ++w;
      P->wave_lo[w] = static_cast<int32_t>(k);
      tnext += budget[w];
    }
    cum += cost;
  }
  while (w < W - 1) P->wave_lo[++w] = static_cast<int32_t>(nl);
  P->wave_lo[W] = static_cast<int32_t>(nl);
  // edge pieces over the upper entries of each row
  for (int64_t u = 0; u < n; ++u) {
    const int64_t up = c.ubase[u + 1] - c.ubase[u];
    const int64_t upos = rp[u + 1] - up;
    for (int64_t b = upos; b < rp[u + 1]; b += kPiece) {
      P->piece_row.push_back(static_cast<int32_t>(u));
      P->piece_beg.push_back(b);
      P->piece_end.push_back(std::min(rp[u + 1], b + kPiece));
    }
  }
}

// Workspace layout for a padded block width.
struct WorkLayout {
  int64_t z, r, p, q, chunkbuf, mega_dots, rho, rr, rho0, thr, alpha, beta, active,
      iters, status, n_active, upd_pending, pred_done, nspmm, fin_ctr, one, part, part_u, lvl0, lvl1, lvl2, tick, out, minv,
      total;
  int grid_rhs, grid_upd, grid_ed, grid_tree;
};

int padded_width(erc_dtype dt, int k) {
  int kb = (dt == ERC_F32) ? 16 : 8;
  while (kb < k) kb <<= 1;
  return kb;
}
int max_width(erc_dtype dt) { return dt == ERC_F32 ? 256 : 128; }

}  // namespace

struct erc_graph_s {
  int64_t n = 0, nnz = 0, m = 0;
  erc_dtype dt = ERC_F32;
  bool weighted = false;
  int device = 0;
  int64_t nonisolated = 0;
  Shape shape{};
  DevGraph dg{};
  int32_t* pinned = nullptr;  // host poll slots and per-column readback
  // [0..3] block phases, [4..5] poll groups, [6..7] whole erc_resistance call
  hipEvent_t ev[8] = {};
  std::vector<hipEvent_t> prof;  // SpMM timing pairs: [slot][launch][begin/end]
  int prof_check = 0;
  // one group of CG iterations captured as a HIP graph, replayed on the caller's stream;
  // the key names everything the captured kernel arguments depend on
  hipStream_t cap = nullptr;
  hipGraphExec_t gexec = nullptr;
  struct GroupKey {
    const void* ws = nullptr;
    int kb = 0, pc = 0, nb = 0, fin2 = 0;
    double delta = 0.0;
  } gkey;
};

namespace {

constexpr int kPinnedInts = 4096;
// pinned slot (8-byte aligned) of the sampling call's non-finite-curvature flag, past the
// per-column readback of the widest block (8 + 4 * 256 + 4 * 256 ints)
constexpr int kPinSampleFlag = 4064;

WorkLayout work_layout(const erc_graph_s* h, int kb) {
  WorkLayout L{};
  const int64_t s = static_cast<int64_t>(dsize(h->dt));
  const int vec = h->dt == ERC_F32 ? 4 : 2;
  L.grid_rhs = static_cast<int>(std::min<int64_t>(kMaxGridRhs, std::max<int64_t>(1, ceil_div(h->n, kWavesPerBlock))));
  const int64_t nvec = h->n * kb / vec;
  L.grid_upd = static_cast<int>(std::min<int64_t>(kMaxGridUpd, std::max<int64_t>(1, ceil_div(nvec, kBlock * 4))));
  L.grid_ed = static_cast<int>(std::min<int64_t>(kMaxGridEd, std::max<int64_t>(1, ceil_div(h->dg.npiece, kWavesPerBlock))));
  L.grid_tree = std::max({h->dg.grid, L.grid_rhs, L.grid_upd});
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    const int64_t at = off;
    off = align_up(off + std::max<int64_t>(bytes, 0), 256);
    return at;
  };
  const int64_t vecb = h->n * kb * s;
  L.z = take(vecb);
  L.r = take(vecb);
  L.p = take(vecb);
  L.q = take(vecb);
  L.chunkbuf = take(static_cast<int64_t>(h->dg.nchunk_slots) * kb * 8);  // fp64 chunk sums
  L.mega_dots = take(static_cast<int64_t>(h->dg.nmega) * 3 * kb * 16);
  L.rho = take(kb * 8);
  L.rr = take(kb * 8);
  L.rho0 = take(kb * 8);
  L.thr = take(kb * 8);
  L.alpha = take(kb * 8);
  L.beta = take(kb * 8);
  L.active = take(kb * 4);
  L.iters = take(kb * 4);
  L.status = take(kb * 4);
  L.n_active = take(4);
  L.upd_pending = take(4);
  L.pred_done = take(4);
  L.nspmm = take(4);
  L.fin_ctr = take(8);
  L.one = take(4);
  const int64_t nval = 10 * kb;  // up to five compensated (s, c) pairs per column
  L.part = take(static_cast<int64_t>(L.grid_tree) * 6 * kb * 8);
  L.part_u = take(static_cast<int64_t>(L.grid_upd) * 4 * kb * 8);  // r.r and r.M^-1 r
  // the finishing launches run ceil(grid/32) <= 256 blocks; k_count_bad runs <= 2048
  L.lvl0 = take(static_cast<int64_t>(kMaxTreeGrid) * nval * 8);
  L.lvl1 = take(ceil_div(kMaxTreeGrid, kTreeFan) * nval * 8);
  L.lvl2 = take(ceil_div(kMaxTreeGrid, kTreeFan * kTreeFan) * nval * 8);
  L.tick = take(tree_ticks(kMaxTreeGrid) * 4);
  L.out = take(8 * 8);
  L.minv = take(h->n * s);
  L.total = off;
  return L;
}

Work carve_work(const erc_graph_s* h, int kb, void* ws, const WorkLayout& L, int pc = 0) {
  char* b = static_cast<char*>(ws);
  Work w{};
  w.kb = kb;
  w.z = b + L.z;
  w.r = b + L.r;
  w.p = b + L.p;
  w.q = b + L.q;
  w.chunkbuf = b + L.chunkbuf;
  w.mega_dots = reinterpret_cast<double*>(b + L.mega_dots);
  w.cs.rho = reinterpret_cast<double*>(b + L.rho);
  w.cs.rr = reinterpret_cast<double*>(b + L.rr);
  w.cs.rho0 = reinterpret_cast<double*>(b + L.rho0);
  w.cs.thr = reinterpret_cast<double*>(b + L.thr);
  w.cs.alpha = reinterpret_cast<double*>(b + L.alpha);
  w.cs.beta = reinterpret_cast<double*>(b + L.beta);
  w.cs.active = reinterpret_cast<int32_t*>(b + L.active);
  w.cs.iters = reinterpret_cast<int32_t*>(b + L.iters);
  w.cs.status = reinterpret_cast<int32_t*>(b + L.status);
  w.cs.n_active = reinterpret_cast<int32_t*>(b + L.n_active);
  w.cs.upd_pending = reinterpret_cast<int32_t*>(b + L.upd_pending);
  w.cs.pred_done = reinterpret_cast<int32_t*>(b + L.pred_done);
  w.cs.nspmm = reinterpret_cast<int32_t*>(b + L.nspmm);
  w.cs.fin_word = reinterpret_cast<unsigned long long*>(b + L.fin_ctr);
  w.cs.one = reinterpret_cast<int32_t*>(b + L.one);
  w.part = reinterpret_cast<double*>(b + L.part);
  w.part_u = reinterpret_cast<double*>(b + L.part_u);
  w.tree.lvl0 = reinterpret_cast<double*>(b + L.lvl0);
  w.tree.lvl1 = reinterpret_cast<double*>(b + L.lvl1);
  w.tree.lvl2 = reinterpret_cast<double*>(b + L.lvl2);
  w.tree.tick = reinterpret_cast<uint32_t*>(b + L.tick);
  w.out = reinterpret_cast<double*>(b + L.out);
  w.minv = b + L.minv;
  w.pc = pc;
  // The early stopping test after each update (a third finishing launch, which exits at
  // once unless every active column is predicted to stop) saves the one SpMM that would
  // otherwise run after a block's last update, and costs a launch in every iteration.
  // It pays only where an SpMM is long: gathers of at least kFin2MinGather bytes.
  w.fin2 = static_cast<double>(h->nnz) * kb * static_cast<double>(dsize(h->dt)) >= kFin2MinGather;
  w.grid_rhs = L.grid_rhs;
  w.grid_upd = L.grid_upd;
  w.grid_ed = L.grid_ed;
  return w;
}

// Zero the tickets and set the constant-one gate (fill kernels, so a captured stream
// records no memset node).
erc_status prepare_work(const erc_graph_s* h, const Work& w, const WorkLayout& L, hipStream_t s) {
  ERC_HIP(launch_fill_u32(w.tree.tick, 0u, tree_ticks(kMaxTreeGrid), s));
  ERC_HIP(launch_fill_u32(reinterpret_cast<uint32_t*>(w.cs.fin_word), 0u, 2, s));
  ERC_HIP(launch_fill_u32(reinterpret_cast<uint32_t*>(w.cs.one), 1u, 1, s));
  return ERC_OK;
}

uint64_t splitmix_first(uint64_t seed) {
  uint64_t z = seed + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

erc_status check_params(const erc_graph_s* h, const erc_solve_params* p) {
  if (p == nullptr) return fail(ERC_E_INVALID_ARG, "params is NULL");
  if (p->K_total < 1) return fail(ERC_E_INVALID_ARG, "K_total must be >= 1");
  if (p->k_block < 1 || p->k_block > max_width(h->dt))
    return fail(ERC_E_INVALID_ARG, "k_block out of range for the working precision");
  if (p->col_begin < 0 || p->col_begin >= p->col_end || p->col_end > p->K_total)
    return fail(ERC_E_INVALID_ARG, "column range must satisfy 0 <= begin < end <= K_total");
  if (!(p->delta > 0.0) || !std::isfinite(p->delta))
    return fail(ERC_E_INVALID_ARG, "delta must be finite and > 0");
  if (!(p->tol > 0.0 && p->tol < 1.0)) return fail(ERC_E_INVALID_ARG, "tol must be in (0, 1)");
  if (p->max_iter < 1) return fail(ERC_E_INVALID_ARG, "max_iter must be >= 1");
  if (p->check_every < 0) return fail(ERC_E_INVALID_ARG, "check_every must be >= 0");
  if ((p->flags & ~(ERC_ACCUMULATE | ERC_PROFILE_SPMM | ERC_JACOBI | ERC_NO_GRAPH |
                     ERC_EARLY_STOP)) != 0u)
    return fail(ERC_E_INVALID_ARG, "unknown flag");
  return ERC_OK;
}

struct BlockStats {
  int32_t iters_max = 0, unconverged = 0, breakdowns = 0;
  int64_t iters_total = 0, launches = 0, spmm_full = 0;
  double max_relres = 0.0;
  float ms_rhs = 0, ms_cg = 0, ms_accum = 0, ms_spmm = 0;
  int64_t spmm_timed = 0;
};

erc_status ensure_prof_events(erc_graph_s* h, int check) {
  if (h->prof_check >= check) return ERC_OK;
  for (auto& e : h->prof)
    if (e) (void)hipEventDestroy(e);
  h->prof.assign(static_cast<size_t>(4) * check, nullptr);
  for (auto& e : h->prof) ERC_HIP(hipEventCreate(&e));
  h->prof_check = check;
  return ERC_OK;
}

// Sum the SpMM event pairs of one poll group.
erc_status read_prof(erc_graph_s* h, int slot, int count, BlockStats* st) {
  for (int j = 0; j < count; ++j) {
    float ms = 0.0f;
    hipEvent_t* pr = &h->prof[(static_cast<size_t>(slot) * h->prof_check + j) * 2];
    ERC_HIP(hipEventElapsedTime(&ms, pr[0], pr[1]));
    st->ms_spmm += ms;
    st->spmm_timed += 1;
  }
  return ERC_OK;
}

// One CG iteration: SpMM (+ split-row finish), finishing step, update, and the early
// stopping test that runs only when every column is predicted to stop.
hipError_t enqueue_iteration(const erc_graph_s* h, const Work& w, double delta, hipStream_t s) {
  hipError_t e = launch_spmm(h->dg, w, h->dt, delta, w.p, w.r, w.q, w.cs.n_active, s);
  if (e == hipSuccess) e = launch_fin_iter(h->dg, w, 0, s);
  if (e == hipSuccess) e = launch_update(h->dg, w, h->dt, s);
  // the exact stopping test, only when every column is predicted to stop: saves the
  // SpMM that would otherwise run after the last update (on graphs where it pays)
  if (e == hipSuccess && w.fin2) e = launch_fin_iter(h->dg, w, 2, s);
  return e;
}

// Capture nb iterations into the handle's graph unless the cached one has the same
// kernel arguments (same workspace, width, variant and shift).
erc_status ensure_group_graph(erc_graph_s* h, const Work& w, double delta, int nb) {
  erc_graph_s::GroupKey k;
  k.ws = w.z;
  k.kb = w.kb;
  k.pc = w.pc;
  k.nb = nb;
  k.fin2 = w.fin2;
  k.delta = delta;
  const erc_graph_s::GroupKey& o = h->gkey;
  if (h->gexec != nullptr && o.ws == k.ws && o.kb == k.kb && o.pc == k.pc && o.nb == k.nb &&
      o.fin2 == k.fin2 && o.delta == k.delta)
    return ERC_OK;
  if (h->gexec != nullptr) {
    (void)hipGraphExecDestroy(h->gexec);
    h->gexec = nullptr;
  }
  ERC_HIP(hipStreamBeginCapture(h->cap, hipStreamCaptureModeThreadLocal));
  hipError_t e = hipSuccess;
  for (int j = 0; j < nb && e == hipSuccess; ++j) e = enqueue_iteration(h, w, delta, h->cap);
  hipGraph_t g = nullptr;
  const hipError_t ee = hipStreamEndCapture(h->cap, &g);
  if (e == hipSuccess) e = ee;
  hipGraphExec_t x = nullptr;
  if (e == hipSuccess) e = hipGraphInstantiate(&x, g, nullptr, nullptr, 0);
  if (g != nullptr) (void)hipGraphDestroy(g);
  if (e != hipSuccess)
    return fail(ERC_E_DEVICE, std::string("CG group capture: ") + hipGetErrorString(e));
  h->gexec = x;
  h->gkey = k;
  return ERC_OK;
}

// One column block: right-hand sides, CG to tol or max_iter, then (if R != nullptr)
// the edge-distance accumulation.  Ends with the stream drained.
erc_status solve_block(erc_graph_s* h, const erc_solve_params* p, const Work& w, int col0, int nc,
                       double* R, int accumulate, int32_t* iters_out, BlockStats* st,
                       hipStream_t s) {
  const double inv_sqrt_k = 1.0 / std::sqrt(static_cast<double>(p->K_total));
  const uint64_t base = splitmix_first(p->seed);
  ERC_HIP(hipEventRecord(h->ev[0], s));
  if (w.pc) ERC_HIP(launch_minv(h->dg, w, h->dt, p->delta, s));
  ERC_HIP(launch_rhs(h->dg, w, h->dt, p->K_total, col0, nc, base, inv_sqrt_k, p->tol, s));
  ERC_HIP(hipEventRecord(h->ev[1], s));
  const int check = p->check_every > 0 ? p->check_every : kDefaultCheck;
  const bool prof = (p->flags & ERC_PROFILE_SPMM) != 0u;
  const bool graph = !prof && (p->flags & ERC_NO_GRAPH) == 0u;
  if (prof) {
    erc_status pst = ensure_prof_events(h, check);
    if (pst != ERC_OK) return pst;
  }
  volatile int32_t* poll = h->pinned;
  int done = 0, pending = -1, slot = 0;
  int group_count[2] = {0, 0};
  bool stop = false;
  while (!stop && done < p->max_iter) {
    const int nb = std::min(check, p->max_iter - done);
    slot ^= 1;
    if (graph && nb == check) {
      erc_status gst = ensure_group_graph(h, w, p->delta, nb);
      if (gst != ERC_OK) return gst;
      ERC_HIP(hipGraphLaunch(h->gexec, s));
    } else {
      for (int j = 0; j < nb; ++j) {
        hipEvent_t* pr = prof ? &h->prof[(static_cast<size_t>(slot) * h->prof_check + j) * 2] : nullptr;
        if (prof) {
          // the SpMM alone between the events (its split-row finish follows it)
          ERC_HIP(hipEventRecord(pr[0], s));
          ERC_HIP(launch_spmm(h->dg, w, h->dt, p->delta, w.p, w.r, w.q, w.cs.n_active, s));
          ERC_HIP(hipEventRecord(pr[1], s));
          ERC_HIP(launch_fin_iter(h->dg, w, 0, s));
          ERC_HIP(launch_update(h->dg, w, h->dt, s));
          if (w.fin2) ERC_HIP(launch_fin_iter(h->dg, w, 2, s));
        } else {
          ERC_HIP(enqueue_iteration(h, w, p->delta, s));
        }
      }
    }
    group_count[slot] = nb;
    done += nb;
    st->launches += nb;
    ERC_HIP(hipMemcpyAsync(const_cast<int32_t*>(poll) + slot, w.cs.n_active, sizeof(int32_t),
                           hipMemcpyDeviceToHost, s));
    ERC_HIP(hipEventRecord(h->ev[4 + slot], s));
    if (pending >= 0) {
      ERC_HIP(hipEventSynchronize(h->ev[4 + pending]));
      if (poll[pending] == 0) stop = true;
      if (prof) {
        erc_status pst = read_prof(h, pending, group_count[pending], st);
        if (pst != ERC_OK) return pst;
        group_count[pending] = 0;
      }
    }
    pending = slot;
  }
  // the last update's r.r: stopping test and iteration count of the final iteration
  ERC_HIP(launch_fin_iter(h->dg, w, 1, s));
  ERC_HIP(hipEventRecord(h->ev[2], s));
  if (R != nullptr) ERC_HIP(launch_edge_dist(h->dg, w, h->dt, R, accumulate, s));
  ERC_HIP(hipEventRecord(h->ev[3], s));
  // per-column state back to the host
  const int kb = w.kb;
  int32_t* hb = h->pinned + 8;
  ERC_HIP(hipMemcpyAsync(hb, w.cs.iters, kb * 4, hipMemcpyDeviceToHost, s));
  ERC_HIP(hipMemcpyAsync(hb + kb, w.cs.active, kb * 4, hipMemcpyDeviceToHost, s));
  ERC_HIP(hipMemcpyAsync(hb + 2 * kb, w.cs.status, kb * 4, hipMemcpyDeviceToHost, s));
  double* hd = reinterpret_cast<double*>(h->pinned + 8 + 4 * kb);
  ERC_HIP(hipMemcpyAsync(hd, w.cs.rr, kb * 8, hipMemcpyDeviceToHost, s));
  ERC_HIP(hipMemcpyAsync(hd + kb, w.cs.rho0, kb * 8, hipMemcpyDeviceToHost, s));
  ERC_HIP(hipMemcpyAsync(h->pinned + 2, w.cs.nspmm, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  ERC_HIP(hipStreamSynchronize(s));
  if (prof && pending >= 0 && group_count[pending] > 0) {
    erc_status pst = read_prof(h, pending, group_count[pending], st);
    if (pst != ERC_OK) return pst;
  }
  // SpMM launches that found an active column (counted on the device)
  st->spmm_full += h->pinned[2];
  for (int c = 0; c < nc; ++c) {
    const int32_t it = hb[c];
    st->iters_total += it;
    st->iters_max = std::max(st->iters_max, it);
    if (hb[2 * kb + c] != 0) st->breakdowns += 1;
    else if (hb[kb + c] != 0) st->unconverged += 1;
    if (hd[kb + c] > 0.0) st->max_relres = std::max(st->max_relres, std::sqrt(hd[c] / hd[kb + c]));
    if (iters_out) iters_out[c] = it;
  }
  float a = 0, b = 0, c = 0;
  ERC_HIP(hipEventElapsedTime(&a, h->ev[0], h->ev[1]));
  ERC_HIP(hipEventElapsedTime(&b, h->ev[1], h->ev[2]));
  ERC_HIP(hipEventElapsedTime(&c, h->ev[2], h->ev[3]));
  st->ms_rhs += a;
  st->ms_cg += b;
  st->ms_accum += c;
  return ERC_OK;
}

erc_status check_handle(const erc_graph_s* h) {
  if (h == nullptr) return fail(ERC_E_INVALID_ARG, "handle is NULL");
  return ERC_OK;
}

}  // namespace

extern "C" {

const char* erc_status_string(erc_status s) {
  switch (s) {
    case ERC_OK: return "ok";
    case ERC_E_INVALID_ARG: return "invalid argument";
    case ERC_E_INVALID_GRAPH: return "invalid graph";
    case ERC_E_WORKSPACE: return "workspace too small";
    case ERC_E_DEVICE: return "device error";
    case ERC_E_NOT_CONVERGED: return "not converged";
    case ERC_E_NUMERIC: return "numerical breakdown";
    case ERC_E_STATE: return "invalid state";
    case ERC_E_HOST: return "host allocation or thread failure";
  }
  return "unknown status";
}

const char* erc_last_error(void) { return g_last_error.c_str(); }

erc_status erc_validate(const erc_graph_desc* desc, int64_t* m_out) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    erc_status st = check_desc(desc);
    if (st != ERC_OK) return st;
    Canon c;
    if (desc->w == nullptr) st = sweep<float>(desc, nullptr, nullptr);
    else if (desc->w_dtype == ERC_F32) st = sweep<float>(desc, static_cast<const float*>(desc->w), nullptr);
    else st = sweep<double>(desc, static_cast<const double*>(desc->w), nullptr);
    if (st != ERC_OK) return st;
    if (m_out) *m_out = desc->rowptr[desc->n] / 2;
    return ERC_OK;
  });
}

erc_status erc_graph_bytes(const erc_graph_desc* desc, size_t* bytes) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    erc_status st = check_desc(desc);
    if (st != ERC_OK) return st;
    if (bytes == nullptr) return fail(ERC_E_INVALID_ARG, "bytes is NULL");
    const Shape s = make_shape(desc->n, desc->rowptr[desc->n]);
    *bytes = static_cast<size_t>(graph_layout(s, desc->w != nullptr, desc->solve_dtype).total);
    return ERC_OK;
  });
}

erc_status erc_create(const erc_graph_desc* desc, void* dev_mem, size_t bytes, void* stream,
                      erc_handle* out) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (out == nullptr) return fail(ERC_E_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (dev_mem == nullptr) return fail(ERC_E_INVALID_ARG, "dev_mem is NULL");
    if (reinterpret_cast<uintptr_t>(dev_mem) % 256 != 0)
      return fail(ERC_E_INVALID_ARG, "dev_mem must be 256-byte aligned");
    Canon c;
    erc_status st = canonicalise(desc, &c);
    if (st != ERC_OK) return st;
    const int64_t n = desc->n;
    const int64_t nnz = desc->rowptr[n];
    const Shape s = make_shape(n, nnz);
    const bool weighted = desc->w != nullptr;
    const GraphLayout L = graph_layout(s, weighted, desc->solve_dtype);
    if (static_cast<int64_t>(bytes) < L.total)
      return fail(ERC_E_WORKSPACE, "graph buffer smaller than erc_graph_bytes");
    Plan P;
    build_plan(desc, c, s, &P);
    if (static_cast<int64_t>(P.task_row.size()) > s.ntask_max ||
        static_cast<int64_t>(P.mega_nchunk.size()) > s.nmega_max ||
        static_cast<int64_t>(P.piece_row.size()) > s.npiece_max || P.nslot > s.nslot_max)
      return fail(ERC_E_STATE, "internal: work plan exceeds its size bound");
    // weights in the working precision
    std::vector<float> wf;
    std::vector<double> wd;
    const void* wsrc = nullptr;
    if (weighted) {
      if (desc->solve_dtype == ERC_F32) {
        if (desc->w_dtype == ERC_F32) {
          wsrc = desc->w;
        } else {
          wf.resize(nnz);
          const double* x = static_cast<const double*>(desc->w);
          for (int64_t k = 0; k < nnz; ++k) wf[k] = static_cast<float>(x[k]);
          wsrc = wf.data();
        }
      } else {
        if (desc->w_dtype == ERC_F64) {
          wsrc = desc->w;
        } else {
          wd.resize(nnz);
          const float* x = static_cast<const float*>(desc->w);
          for (int64_t k = 0; k < nnz; ++k) wd[k] = static_cast<double>(x[k]);
          wsrc = wd.data();
        }
      }
    }
    auto* h = new erc_graph_s();
    h->n = n;
    h->nnz = nnz;
    h->m = c.m;
    h->dt = desc->solve_dtype;
    h->weighted = weighted;
    h->shape = s;
    for (int64_t i = 0; i < n; ++i) h->nonisolated += desc->rowptr[i + 1] > desc->rowptr[i];
    auto cleanup = [&](erc_status e) {
      if (h->pinned) (void)hipHostFree(h->pinned);
      for (auto& ev : h->ev)
        if (ev) (void)hipEventDestroy(ev);
      if (h->cap) (void)hipStreamDestroy(h->cap);
      delete h;
      return e;
    };
    if (hipGetDevice(&h->device) != hipSuccess) return cleanup(fail(ERC_E_DEVICE, "hipGetDevice failed"));
    if (hipHostMalloc(reinterpret_cast<void**>(&h->pinned), kPinnedInts * sizeof(int32_t),
                      hipHostMallocDefault) != hipSuccess)
      return cleanup(fail(ERC_E_DEVICE, "hipHostMalloc failed"));
    for (auto& ev : h->ev)
      if (hipEventCreate(&ev) != hipSuccess) return cleanup(fail(ERC_E_DEVICE, "hipEventCreate failed"));
    // the fixed scratch of erc_sampling_probs_static on this device (that call retries
    // the lookup if it fails here, so a failure does not stop the handle)
    (void)static_scratch_setup(h->device);
    // default priority (no priority argument): the stream only records graph captures
    if (hipStreamCreateWithFlags(&h->cap, hipStreamNonBlocking) != hipSuccess)
      return cleanup(fail(ERC_E_DEVICE, "hipStreamCreateWithFlags failed"));
    char* base = static_cast<char*>(dev_mem);
    hipStream_t hs = static_cast<hipStream_t>(stream);
    auto up = [&](int64_t off, const void* src, int64_t nbytes) -> hipError_t {
      if (nbytes <= 0) return hipSuccess;
      return hipMemcpyAsync(base + off, src, nbytes, hipMemcpyHostToDevice, hs);
    };
    hipError_t e = hipSuccess;
    auto chk = [&](hipError_t x) { if (e == hipSuccess) e = x; };
    chk(up(L.rowptr, desc->rowptr, (n + 1) * 8));
    chk(up(L.col, desc->col, nnz * 4));
    if (weighted) chk(up(L.w, wsrc, nnz * static_cast<int64_t>(dsize(desc->solve_dtype))));
    chk(up(L.eid, c.eid.data(), nnz * 4));
    chk(up(L.sw, c.sw.data(), c.m * 8));
    chk(up(L.ubase, c.ubase.data(), (n + 1) * 8));
    chk(up(L.deg, c.deg.data(), n * 8));
    std::vector<LightRow> lrows(P.light.size());
    for (size_t k = 0; k < P.light.size(); ++k) {
      const int32_t i = P.light[k];
      lrows[k] = LightRow{desc->rowptr[i], i, static_cast<int32_t>(desc->rowptr[i + 1] - desc->rowptr[i])};
    }
    chk(up(L.light, lrows.data(), static_cast<int64_t>(lrows.size() * sizeof(LightRow))));
    chk(up(L.wave_lo, P.wave_lo.data(), static_cast<int64_t>(P.wave_lo.size()) * 4));
    const int64_t nt = static_cast<int64_t>(P.task_row.size());
    chk(up(L.task_row, P.task_row.data(), nt * 4));
    chk(up(L.task_mega, P.task_mega.data(), nt * 4));
    chk(up(L.task_chunk, P.task_chunk.data(), nt * 4));
    chk(up(L.task_beg, P.task_beg.data(), nt * 8));
    chk(up(L.task_end, P.task_end.data(), nt * 8));
    const int64_t nm = static_cast<int64_t>(P.mega_nchunk.size());
    chk(up(L.mega_row, P.mega_row.data(), nm * 4));
    chk(up(L.mega_nchunk, P.mega_nchunk.data(), nm * 4));
    chk(up(L.mega_chunk0, P.mega_chunk0.data(), nm * 4));
    const int64_t np = static_cast<int64_t>(P.piece_row.size());
    chk(up(L.piece_row, P.piece_row.data(), np * 4));
    chk(up(L.piece_beg, P.piece_beg.data(), np * 8));
    chk(up(L.piece_end, P.piece_end.data(), np * 8));
    if (e == hipSuccess) e = hipStreamSynchronize(hs);
    if (e != hipSuccess) return cleanup(fail(ERC_E_DEVICE, std::string("graph upload: ") + hipGetErrorString(e)));
    DevGraph& g = h->dg;
    g.n = static_cast<int32_t>(n);
    g.nnz = nnz;
    g.m = c.m;
    g.weighted = weighted ? 1 : 0;
    // the stored weights equal the input ones unless fp64 input is rounded to fp32
    g.sw_from_w = (weighted && !(desc->w_dtype == ERC_F64 && desc->solve_dtype == ERC_F32)) ? 1 : 0;
    g.rowptr = reinterpret_cast<const int64_t*>(base + L.rowptr);
    g.col = reinterpret_cast<const int32_t*>(base + L.col);
    g.w = weighted ? base + L.w : nullptr;
    g.eid = reinterpret_cast<const int32_t*>(base + L.eid);
    g.sw = reinterpret_cast<const double*>(base + L.sw);
    g.ubase = reinterpret_cast<const int64_t*>(base + L.ubase);
    g.deg = reinterpret_cast<const double*>(base + L.deg);
    g.grid = s.grid;
    g.light = reinterpret_cast<const LightRow*>(base + L.light);
    g.wave_lo = reinterpret_cast<const int32_t*>(base + L.wave_lo);
    g.ntask = static_cast<int32_t>(nt);
    g.task_row = reinterpret_cast<const int32_t*>(base + L.task_row);
    g.task_mega = reinterpret_cast<const int32_t*>(base + L.task_mega);
    g.task_chunk = reinterpret_cast<const int32_t*>(base + L.task_chunk);
    g.task_beg = reinterpret_cast<const int64_t*>(base + L.task_beg);
    g.task_end = reinterpret_cast<const int64_t*>(base + L.task_end);
    g.nmega = static_cast<int32_t>(nm);
    g.mega_row = reinterpret_cast<const int32_t*>(base + L.mega_row);
    g.mega_nchunk = reinterpret_cast<const int32_t*>(base + L.mega_nchunk);
    g.mega_chunk0 = reinterpret_cast<const int32_t*>(base + L.mega_chunk0);
    g.nchunk_slots = P.nslot;
    g.npiece = np;
    g.piece_row = reinterpret_cast<const int32_t*>(base + L.piece_row);
    g.piece_beg = reinterpret_cast<const int64_t*>(base + L.piece_beg);
    g.piece_end = reinterpret_cast<const int64_t*>(base + L.piece_end);
    *out = h;
    return ERC_OK;
  });
}

erc_status erc_num_nodes(erc_handle h, int64_t* n) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (n == nullptr) return fail(ERC_E_INVALID_ARG, "n is NULL");
    *n = h->n;
    return ERC_OK;
  });
}

erc_status erc_num_edges(erc_handle h, int64_t* m) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (m == nullptr) return fail(ERC_E_INVALID_ARG, "m is NULL");
    *m = h->m;
    return ERC_OK;
  });
}

erc_status erc_edge_endpoints(erc_handle h, int32_t* u_dev, int32_t* v_dev, void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (h->m > 0 && (u_dev == nullptr || v_dev == nullptr)) return fail(ERC_E_INVALID_ARG, "output is NULL");
    ERC_HIP(launch_endpoints(h->dg, u_dev, v_dev, static_cast<hipStream_t>(stream)));
    return ERC_OK;
  });
}

erc_status erc_destroy(erc_handle h) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (h == nullptr) return ERC_OK;
    if (h->pinned) (void)hipHostFree(h->pinned);
    for (auto& ev : h->ev)
      if (ev) (void)hipEventDestroy(ev);
    for (auto& ev : h->prof)
      if (ev) (void)hipEventDestroy(ev);
    if (h->gexec) (void)hipGraphExecDestroy(h->gexec);
    if (h->cap) (void)hipStreamDestroy(h->cap);
    delete h;
    return ERC_OK;
  });
}

erc_status erc_workspace_bytes(erc_handle h, int32_t k_block, size_t* bytes) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (bytes == nullptr) return fail(ERC_E_INVALID_ARG, "bytes is NULL");
    if (k_block < 1 || k_block > max_width(h->dt))
      return fail(ERC_E_INVALID_ARG, "k_block out of range for the working precision");
    *bytes = static_cast<size_t>(work_layout(h, padded_width(h->dt, k_block)).total);
    return ERC_OK;
  });
}

erc_status erc_resistance(erc_handle h, const erc_solve_params* params, void* ws_dev, size_t ws_bytes,
                          double* R_dev, erc_solve_info* info, void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    erc_status st = check_params(h, params);
    if (st != ERC_OK) return st;
    if (h->m > 0 && R_dev == nullptr) return fail(ERC_E_INVALID_ARG, "R_dev is NULL");
    if (ws_dev == nullptr) return fail(ERC_E_INVALID_ARG, "ws_dev is NULL");
    const int kb = padded_width(h->dt, params->k_block);
    const WorkLayout L = work_layout(h, kb);
    if (static_cast<int64_t>(ws_bytes) < L.total)
      return fail(ERC_E_WORKSPACE, "workspace smaller than erc_workspace_bytes");
    hipStream_t s = static_cast<hipStream_t>(stream);
    Work w = carve_work(h, kb, ws_dev, L, (params->flags & ERC_JACOBI) ? 1 : 0);
    if (params->flags & ERC_EARLY_STOP) w.fin2 = 1;
    st = prepare_work(h, w, L, s);
    if (st != ERC_OK) return st;
    hipEvent_t t0 = h->ev[6], t1 = h->ev[7];
    ERC_HIP(hipEventRecord(t0, s));
    BlockStats bs;
    int blocks = 0;
    for (int c0 = params->col_begin; c0 < params->col_end; c0 += params->k_block) {
      const int nc = std::min(params->k_block, params->col_end - c0);
      const int acc = (c0 == params->col_begin && !(params->flags & ERC_ACCUMULATE)) ? 0 : 1;
      st = solve_block(h, params, w, c0, nc, h->m > 0 ? R_dev : nullptr, acc, nullptr, &bs, s);
      if (st != ERC_OK) return st;
      ++blocks;
    }
    int64_t bad = 0;
    if (h->m > 0) {
      ERC_HIP(launch_count_bad(R_dev, h->m, w, s));
      double hb = 0.0;
      ERC_HIP(hipMemcpyAsync(reinterpret_cast<double*>(h->pinned + 2), w.out, 8, hipMemcpyDeviceToHost, s));
      ERC_HIP(hipEventRecord(t1, s));
      ERC_HIP(hipStreamSynchronize(s));
      std::memcpy(&hb, h->pinned + 2, 8);
      bad = static_cast<int64_t>(hb);
    } else {
      ERC_HIP(hipEventRecord(t1, s));
      ERC_HIP(hipStreamSynchronize(s));
    }
    float total = 0.0f;
    (void)hipEventElapsedTime(&total, t0, t1);  // timing only: 0 if unavailable
    if (info) {
      info->blocks = blocks;
      info->iters_max = bs.iters_max;
      info->cols_unconverged = bs.unconverged;
      info->breakdowns = bs.breakdowns;
      info->iters_total = bs.iters_total;
      info->launches = bs.launches;
      info->nonpositive = bad;
      info->max_final_relres = bs.max_relres;
      info->ms_rhs = bs.ms_rhs;
      info->ms_cg = bs.ms_cg;
      info->ms_accum = bs.ms_accum;
      info->ms_total = total;
      info->ms_spmm = bs.ms_spmm;
      info->spmm_timed = bs.spmm_timed;
      info->spmm_full = bs.spmm_full;
      // algorithmic bytes (no neighbour-row gathers beyond one read of each vector): every
      // SpMM that found active columns reads col (+ w), rowptr, p and r and writes q; its
      // update reads z, r, p, q and writes z, r, p; per block the right-hand sides read
      // col, eid (+ w) and write z, r, p, and the edge distances read the upper col
      // entries and z and read-modify-write R
      {
        const double sz = static_cast<double>(dsize(h->dt));
        const double n = static_cast<double>(h->n), nnz = static_cast<double>(h->nnz);
        const double m = static_cast<double>(h->m);
        const double kb = static_cast<double>(padded_width(h->dt, params->k_block));
        const double wb = h->weighted ? sz : 0.0;
        const double spmm = (4.0 + wb) * nnz + 8.0 * (n + 1) + 3.0 * sz * n * kb;
        const double upd = 7.0 * sz * n * kb;
        const double rhs = (8.0 + wb) * nnz + 3.0 * sz * n * kb;
        const double ed = 2.0 * nnz + sz * n * kb + 16.0 * m;
        info->bytes_model = static_cast<double>(bs.spmm_full) * (spmm + upd) +
                            static_cast<double>(blocks) * (rhs + ed);
      }
    }
    if (bs.breakdowns > 0) return fail(ERC_E_NUMERIC, "CG breakdown in " + std::to_string(bs.breakdowns) + " column(s)");
    if (bad > 0) return fail(ERC_E_NUMERIC, std::to_string(bad) + " resistance(s) <= 0 or not finite");
    if (bs.unconverged > 0)
      return fail(ERC_E_NOT_CONVERGED, std::to_string(bs.unconverged) + " column(s) reached max_iter");
    return ERC_OK;
  });
}

erc_status erc_curvature(erc_handle h, const double* R_dev, double* p_dev, double* kappa_dev,
                         void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (p_dev == nullptr || (h->m > 0 && (R_dev == nullptr || kappa_dev == nullptr)))
      return fail(ERC_E_INVALID_ARG, "NULL buffer");
    hipStream_t s = static_cast<hipStream_t>(stream);
    ERC_HIP(launch_node_p(h->dg, h->dt, R_dev, p_dev, s));
    ERC_HIP(launch_edge_kappa(h->dg, R_dev, p_dev, kappa_dev, s));
    return ERC_OK;
  });
}

namespace {
struct SampleLayout {
  int64_t part_mm, part_n, totals, total;
  int grid;
};
SampleLayout sample_layout(const erc_graph_s* h) {
  SampleLayout L{};
  // eight items per thread for the per-edge passes, and at least one block per 32 rows
  // for the per-node pass (a wavefront per row: on small graphs a grid sized by items
  // alone left each wavefront a long chain of dependent row loads)
  const int64_t items = std::max(h->n, h->m);
  const int64_t want = std::max(ceil_div(items, kBlock * 8), ceil_div(h->n, kWavesPerBlock * 8));
  L.grid = static_cast<int>(std::min<int64_t>(kSampleGrid, std::max<int64_t>(1, want)));
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    const int64_t at = off;
    off = align_up(off + std::max<int64_t>(bytes, 0), 256);
    return at;
  };
  L.part_mm = take(static_cast<int64_t>(L.grid) * 3 * 8);
  L.part_n = take(static_cast<int64_t>(L.grid) * 8);
  L.totals = take(8 * 8);
  L.total = off;
  return L;
}
}  // namespace

erc_status erc_sampling_scratch_bytes(erc_handle h, size_t* bytes) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (bytes == nullptr) return fail(ERC_E_INVALID_ARG, "bytes is NULL");
    *bytes = static_cast<size_t>(sample_layout(h).total);
    return ERC_OK;
  });
}

namespace {
// Enqueue the sampling-probability kernels with their scratch at scratch_dev; with
// `wait`, bring the non-finite-curvature flag back and report it.
erc_status sampling_probs_into(erc_graph_s* h, const double* kappa_dev, double eta,
                               void* scratch_dev, size_t scratch_bytes, double* node_prob_dev,
                               double* edge_prob_dev, hipStream_t s, bool wait) {
  if (!(eta > 0.0) || !std::isfinite(eta)) return fail(ERC_E_INVALID_ARG, "eta must be finite and > 0");
  if (node_prob_dev == nullptr || scratch_dev == nullptr ||
      (h->m > 0 && (kappa_dev == nullptr || edge_prob_dev == nullptr)))
    return fail(ERC_E_INVALID_ARG, "NULL buffer");
  const SampleLayout L = sample_layout(h);
  if (static_cast<int64_t>(scratch_bytes) < L.total)
    return fail(ERC_E_WORKSPACE, "scratch smaller than erc_sampling_scratch_bytes (" +
                                     std::to_string(L.total) + " bytes)");
  char* b = static_cast<char*>(scratch_dev);
  SampleWork sw{};
  sw.part_mm = reinterpret_cast<double*>(b + L.part_mm);
  sw.part_n = reinterpret_cast<double*>(b + L.part_n);
  sw.totals = reinterpret_cast<double*>(b + L.totals);
  sw.grid = L.grid;
  // every partial and total is written before it is read, in stream order: nothing is
  // cleared and no ticket is kept between calls
  ERC_HIP(launch_sampling(h->dg, kappa_dev, eta, h->nonisolated, sw, node_prob_dev, edge_prob_dev, s));
  if (!wait) return ERC_OK;
  // the minimum/maximum pass flags a NaN or infinite kappa (the probabilities are then
  // written as NaN); the flag comes back to the host so the call can report it
  double* flag = reinterpret_cast<double*>(h->pinned + kPinSampleFlag);
  ERC_HIP(hipMemcpyAsync(flag, sw.totals + 4, sizeof(double), hipMemcpyDeviceToHost, s));
  ERC_HIP(hipStreamSynchronize(s));
  if (*flag != 0.0) return fail(ERC_E_NUMERIC, "curvature contains NaN or infinite values");
  return ERC_OK;
}
}  // namespace

erc_status erc_sampling_probs(erc_handle h, const double* kappa_dev, double eta, void* scratch_dev,
                              size_t scratch_bytes, double* node_prob_dev, double* edge_prob_dev,
                              void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    return sampling_probs_into(h, kappa_dev, eta, scratch_dev, scratch_bytes, node_prob_dev,
                               edge_prob_dev, static_cast<hipStream_t>(stream), true);
  });
}

erc_status erc_sampling_probs_static(erc_handle h, const double* kappa_dev, double eta,
                                     double* node_prob_dev, double* edge_prob_dev, void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    int cur = -1;
    ERC_HIP(hipGetDevice(&cur));
    if (cur != h->device)
      return fail(ERC_E_INVALID_ARG, "the handle's device (" + std::to_string(h->device) +
                                         ") is not the current device (" + std::to_string(cur) + ")");
    const int64_t need = sample_layout(h).total;
    if (need > static_cast<int64_t>(kStaticScratchBytes))
      return fail(ERC_E_WORKSPACE, "needs " + std::to_string(need) + " bytes of scratch; the static "
                                   "scratch holds " + std::to_string(kStaticScratchBytes));
    // looked up at erc_create; again here if that lookup failed
    ERC_HIP(static_scratch_setup(h->device));
    void* scratch = static_scratch_ptr(h->device);
    if (scratch == nullptr) return fail(ERC_E_DEVICE, "static scratch address unavailable");
    return sampling_probs_into(h, kappa_dev, eta, scratch, kStaticScratchBytes, node_prob_dev,
                               edge_prob_dev, static_cast<hipStream_t>(stream), false);
  });
}

namespace {
struct DrawLayout {
  int64_t cdf, bsum, psum, status, total;
};
DrawLayout draw_layout(int64_t N) {
  DrawLayout L{};
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    const int64_t at = off;
    off = align_up(off + std::max<int64_t>(bytes, 0), 256);
    return at;
  };
  const int64_t nb = std::max<int64_t>(1, scan_blocks(N));
  L.cdf = take((N + 1) * 8);
  L.bsum = take(nb * 8);
  L.psum = take(nb * 8);
  L.status = take(4);
  L.total = off;
  return L;
}
struct SubLayout {
  int64_t npos, epos, bsum, status, total;
};
SubLayout sub_layout(const erc_graph_s* h) {
  SubLayout L{};
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    const int64_t at = off;
    off = align_up(off + std::max<int64_t>(bytes, 0), 256);
    return at;
  };
  L.npos = take((h->n + 1) * 4);
  L.epos = take((h->m + 1) * 4);
  L.bsum = take(std::max<int64_t>(1, scan_blocks(std::max(h->n, h->m))) * 4);
  L.status = take(4);
  L.total = off;
  return L;
}
erc_status read_status(uint32_t* status_dev, hipStream_t s, uint32_t* out) {
  ERC_HIP(hipMemcpyAsync(out, status_dev, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
  ERC_HIP(hipStreamSynchronize(s));
  return ERC_OK;
}
}  // namespace

erc_status erc_draw_scratch_bytes(erc_handle h, erc_items items, size_t* bytes) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (bytes == nullptr) return fail(ERC_E_INVALID_ARG, "bytes is NULL");
    if (items != ERC_NODES && items != ERC_EDGES) return fail(ERC_E_INVALID_ARG, "items must be ERC_NODES or ERC_EDGES");
    *bytes = static_cast<size_t>(draw_layout(items == ERC_NODES ? h->n : h->m).total);
    return ERC_OK;
  });
}

erc_status erc_draw(erc_handle h, erc_items items, const double* prob_dev, int64_t draws,
                    uint64_t seed, void* scratch_dev, size_t scratch_bytes, int64_t* idx_dev,
                    void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (items != ERC_NODES && items != ERC_EDGES) return fail(ERC_E_INVALID_ARG, "items must be ERC_NODES or ERC_EDGES");
    const int64_t N = items == ERC_NODES ? h->n : h->m;
    if (N <= 0) return fail(ERC_E_INVALID_ARG, "no items to draw from");
    if (draws < 0) return fail(ERC_E_INVALID_ARG, "draws must be >= 0");
    if (prob_dev == nullptr || scratch_dev == nullptr || (draws > 0 && idx_dev == nullptr))
      return fail(ERC_E_INVALID_ARG, "NULL buffer");
    const DrawLayout L = draw_layout(N);
    if (static_cast<int64_t>(scratch_bytes) < L.total)
      return fail(ERC_E_WORKSPACE, "scratch smaller than erc_draw_scratch_bytes");
    char* b = static_cast<char*>(scratch_dev);
    DrawWork w{};
    w.cdf = reinterpret_cast<uint64_t*>(b + L.cdf);
    w.bsum = reinterpret_cast<uint64_t*>(b + L.bsum);
    w.psum = reinterpret_cast<double*>(b + L.psum);
    w.status = reinterpret_cast<uint32_t*>(b + L.status);
    hipStream_t s = static_cast<hipStream_t>(stream);
    ERC_HIP(launch_fill_u32(w.status, 0u, 1, s));
    ERC_HIP(launch_draw(prob_dev, N, draws, splitmix_first(seed), w, idx_dev, s));
    uint32_t st = 0;
    erc_status rs = read_status(w.status, s, &st);
    if (rs != ERC_OK) return rs;
    if (st & kDrawBadProb) return fail(ERC_E_NUMERIC, "a probability is NaN or outside [0, 1]");
    if (st & kDrawSumTooLarge) return fail(ERC_E_NUMERIC, "probabilities sum above 1.5");
    if (st & kDrawAllZero) return fail(ERC_E_NUMERIC, "every probability rounds to a zero weight");
    return ERC_OK;
  });
}

erc_status erc_subgraph_scratch_bytes(erc_handle h, size_t* bytes) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (bytes == nullptr) return fail(ERC_E_INVALID_ARG, "bytes is NULL");
    *bytes = static_cast<size_t>(sub_layout(h).total);
    return ERC_OK;
  });
}

erc_status erc_subgraph(erc_handle h, erc_items items, const int64_t* idx_dev, int64_t count,
                        void* scratch_dev, size_t scratch_bytes, int32_t* nodes_dev,
                        int64_t* edges_dev, int32_t* u_dev, int32_t* v_dev,
                        int64_t* counts_host, void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (items != ERC_NODES && items != ERC_EDGES) return fail(ERC_E_INVALID_ARG, "items must be ERC_NODES or ERC_EDGES");
    if (count < 0) return fail(ERC_E_INVALID_ARG, "count must be >= 0");
    if (scratch_dev == nullptr || counts_host == nullptr || nodes_dev == nullptr ||
        (count > 0 && idx_dev == nullptr) ||
        (h->m > 0 && (edges_dev == nullptr || u_dev == nullptr || v_dev == nullptr)))
      return fail(ERC_E_INVALID_ARG, "NULL buffer");
    if (items == ERC_EDGES && h->m == 0 && count > 0)
      return fail(ERC_E_INVALID_ARG, "the graph has no edges");
    const SubLayout L = sub_layout(h);
    if (static_cast<int64_t>(scratch_bytes) < L.total)
      return fail(ERC_E_WORKSPACE, "scratch smaller than erc_subgraph_scratch_bytes");
    char* b = static_cast<char*>(scratch_dev);
    SubgraphWork w{};
    w.npos = reinterpret_cast<uint32_t*>(b + L.npos);
    w.epos = reinterpret_cast<uint32_t*>(b + L.epos);
    w.bsum = reinterpret_cast<uint32_t*>(b + L.bsum);
    w.status = reinterpret_cast<uint32_t*>(b + L.status);
    hipStream_t s = static_cast<hipStream_t>(stream);
    ERC_HIP(launch_fill_u32(w.status, 0u, 1, s));
    ERC_HIP(launch_subgraph(h->dg, items == ERC_NODES ? 0 : 1, idx_dev, count, w, nodes_dev,
                            edges_dev, u_dev, v_dev, s));
    uint32_t tot[2] = {0u, 0u};
    ERC_HIP(hipMemcpyAsync(&tot[0], w.npos + h->n, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
    ERC_HIP(hipMemcpyAsync(&tot[1], w.epos + h->m, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
    uint32_t st = 0;
    erc_status rs = read_status(w.status, s, &st);
    if (rs != ERC_OK) return rs;
    if (st & kSubBadIndex) return fail(ERC_E_INVALID_ARG, "a drawn index is out of range");
    counts_host[0] = tot[0];
    counts_host[1] = tot[1];
    return ERC_OK;
  });
}

erc_status erc_probe_out_bytes(int64_t count, int32_t row_bytes, size_t* bytes) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (bytes == nullptr) return fail(ERC_E_INVALID_ARG, "bytes is NULL");
    if (count < 0) return fail(ERC_E_INVALID_ARG, "count must be >= 0");
    if (row_bytes < 64 || row_bytes > 1024 || (row_bytes & (row_bytes - 1)) != 0)
      return fail(ERC_E_INVALID_ARG, "row_bytes must be a power of two in 64..1024");
    *bytes = static_cast<size_t>(std::max<int64_t>(1, probe_out_rows(count)) * row_bytes);
    return ERC_OK;
  });
}

erc_status erc_probe_gather_sliced(const int32_t* idx_dev, int64_t count, const void* table_dev,
                                   int64_t rows, int32_t row_bytes, int32_t slices,
                                   void* out_dev, void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (count < 0 || rows < 1) return fail(ERC_E_INVALID_ARG, "count must be >= 0 and rows >= 1");
    if (row_bytes < 64 || row_bytes > 1024 || (row_bytes & (row_bytes - 1)) != 0)
      return fail(ERC_E_INVALID_ARG, "row_bytes must be a power of two in 64..1024");
    if (slices < 1 || slices > 64)
      return fail(ERC_E_INVALID_ARG, "slices must be in 1..64");
    if (count > 0 && (idx_dev == nullptr || table_dev == nullptr || out_dev == nullptr))
      return fail(ERC_E_INVALID_ARG, "NULL buffer");
    if (reinterpret_cast<uintptr_t>(table_dev) % 16 != 0 || reinterpret_cast<uintptr_t>(out_dev) % 16 != 0)
      return fail(ERC_E_INVALID_ARG, "table and output must be 16-byte aligned");
    if (probe_out_rows(count) * slices > (int64_t{1} << 31) / kWavesPerBlock)
      return fail(ERC_E_INVALID_ARG, "count * slices too large for one launch");
    ERC_HIP(launch_probe_gather(idx_dev, count, table_dev, rows, row_bytes, slices, out_dev,
                                static_cast<hipStream_t>(stream)));
    return ERC_OK;
  });
}

erc_status erc_probe_gather(const int32_t* idx_dev, int64_t count, const void* table_dev,
                            int64_t rows, int32_t row_bytes, void* out_dev, void* stream) {
  return erc_probe_gather_sliced(idx_dev, count, table_dev, rows, row_bytes, 1, out_dev, stream);
}

erc_status erc_debug_check_plan(const erc_graph_desc* desc) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    Canon c;
    erc_status st = canonicalise(desc, &c);
    if (st != ERC_OK) return st;
    const int64_t n = desc->n;
    const int64_t* rp = desc->rowptr;
    const int64_t nnz = rp[n];
    const Shape s = make_shape(n, nnz);
    Plan P;
    build_plan(desc, c, s, &P);
    auto bad = [&](const std::string& what) { return fail(ERC_E_STATE, "plan check: " + what); };
    const int64_t nt = static_cast<int64_t>(P.task_row.size());
    const int64_t nm = static_cast<int64_t>(P.mega_nchunk.size());
    const int64_t np = static_cast<int64_t>(P.piece_row.size());
    if (nt > s.ntask_max || nm > s.nmega_max || np > s.npiece_max || P.nslot > s.nslot_max)
      return bad("list exceeds its size bound");
    if (s.grid < 1 || s.grid > kMaxSpmmGrid || s.waves != s.grid * kWavesPerBlock)
      return bad("grid shape");
    // SpMM coverage: each entry once, by a light row or by a block task
    std::vector<unsigned char> cover(nnz, 0);
    const int64_t nl = static_cast<int64_t>(P.light.size());
    if (static_cast<int64_t>(P.wave_lo.size()) != s.waves + 1 || P.wave_lo[0] != 0 ||
        P.wave_lo[s.waves] != nl)
      return bad("wave ranges do not span the light rows");
    for (int w = 0; w < s.waves; ++w)
      if (P.wave_lo[w] > P.wave_lo[w + 1]) return bad("wave ranges not monotone");
    std::vector<unsigned char> is_light(n, 0);
    for (int64_t k = 0; k < nl; ++k) {
      const int64_t i = P.light[k];
      if (i < 0 || i >= n || (k > 0 && P.light[k - 1] >= i)) return bad("light rows not ascending in range");
      if (rp[i + 1] - rp[i] > s.heavy) return bad("light row above the heavy threshold");
      is_light[i] = 1;
      for (int64_t pos = rp[i]; pos < rp[i + 1]; ++pos) cover[pos] += 1;
    }
    std::vector<int32_t> seen_chunks(nm, 0);
    for (int64_t t = 0; t < nt; ++t) {
      const int64_t i = P.task_row[t];
      if (i < 0 || i >= n || is_light[i]) return bad("task row out of range or also light");
      if (P.task_beg[t] < rp[i] || P.task_end[t] > rp[i + 1] || P.task_beg[t] >= P.task_end[t])
        return bad("task range outside its row");
      const int32_t mh = P.task_mega[t];
      if (mh >= 0) {
        if (mh >= nm || P.task_chunk[t] < 0 || P.task_chunk[t] >= P.mega_nchunk[mh])
          return bad("chunk index out of range");
        if (P.mega_chunk0[mh] + P.mega_nchunk[mh] > P.nslot) return bad("chunk slots out of range");
        if (P.mega_row[mh] != i) return bad("chunk of a split row names another row");
        seen_chunks[mh] += 1;
      } else if (P.task_beg[t] != rp[i] || P.task_end[t] != rp[i + 1]) {
        return bad("single-chunk task does not cover its row");
      }
      for (int64_t pos = P.task_beg[t]; pos < P.task_end[t]; ++pos) cover[pos] += 1;
    }
    for (int64_t mh = 0; mh < nm; ++mh)
      if (seen_chunks[mh] != P.mega_nchunk[mh]) return bad("multi-chunk row missing chunks");
    for (int64_t i = 0; i < n; ++i)
      if (!is_light[i] && rp[i + 1] - rp[i] <= s.heavy) return bad("row in no plan list");
    for (int64_t pos = 0; pos < nnz; ++pos)
      if (cover[pos] != 1) return bad("entry not covered exactly once");
    // edge pieces: each upper entry once, edge ids consistent with eid
    std::fill(cover.begin(), cover.end(), 0);
    for (int64_t t = 0; t < np; ++t) {
      const int64_t u = P.piece_row[t];
      if (u < 0 || u >= n) return bad("piece row out of range");
      const int64_t up = c.ubase[u + 1] - c.ubase[u];
      const int64_t upos = rp[u + 1] - up;
      if (P.piece_beg[t] < upos || P.piece_end[t] > rp[u + 1] || P.piece_beg[t] >= P.piece_end[t])
        return bad("piece outside the upper entries of its row");
      for (int64_t pos = P.piece_beg[t]; pos < P.piece_end[t]; ++pos) {
        if (desc->col[pos] <= u) return bad("piece covers a lower entry");
        const int64_t e = c.ubase[u] + (pos - upos);
        if (e != c.eid[pos]) return bad("piece edge id differs from the entry's edge id");
        cover[pos] += 1;
      }
    }
    for (int64_t u = 0; u < n; ++u)
      for (int64_t pos = rp[u]; pos < rp[u + 1]; ++pos)
        if ((desc->col[pos] > u) != (cover[pos] == 1)) return bad("upper entry not covered exactly once");
    return ERC_OK;
  });
}

erc_status erc_debug_edge_ids(erc_handle h, int32_t* eid_dev, void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (h->nnz > 0 && eid_dev == nullptr) return fail(ERC_E_INVALID_ARG, "eid_dev is NULL");
    ERC_HIP(launch_eids(h->dg, eid_dev, static_cast<hipStream_t>(stream)));
    return ERC_OK;
  });
}

erc_status erc_debug_rhs(erc_handle h, int32_t K_total, int32_t col0, int32_t ncols, uint64_t seed,
                         void* Y_dev, void* ws_dev, size_t ws_bytes, void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (K_total < 1 || ncols < 1 || ncols > max_width(h->dt) || col0 < 0 || col0 + ncols > K_total)
      return fail(ERC_E_INVALID_ARG, "bad column range");
    if (Y_dev == nullptr || ws_dev == nullptr) return fail(ERC_E_INVALID_ARG, "NULL buffer");
    const int kb = padded_width(h->dt, ncols);
    const WorkLayout L = work_layout(h, kb);
    if (static_cast<int64_t>(ws_bytes) < L.total) return fail(ERC_E_WORKSPACE, "workspace too small");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const Work w = carve_work(h, kb, ws_dev, L);
    erc_status st = prepare_work(h, w, L, s);
    if (st != ERC_OK) return st;
    ERC_HIP(launch_rhs(h->dg, w, h->dt, K_total, col0, ncols, splitmix_first(seed),
                       1.0 / std::sqrt(static_cast<double>(K_total)), 0.5, s));
    ERC_HIP(launch_copy_cols(h->dg, w.r, kb, h->dt, ncols, Y_dev, s));
    return ERC_OK;
  });
}

erc_status erc_debug_spmm(erc_handle h, double delta, int32_t ncols, const void* X_dev, void* Y_dev,
                          void* ws_dev, size_t ws_bytes, void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    if (ncols < 1 || ncols > max_width(h->dt) || padded_width(h->dt, ncols) != ncols)
      return fail(ERC_E_INVALID_ARG, "ncols must be a padded block width");
    if (!std::isfinite(delta) || delta < 0.0) return fail(ERC_E_INVALID_ARG, "delta must be finite and >= 0");
    if (X_dev == nullptr || Y_dev == nullptr || ws_dev == nullptr) return fail(ERC_E_INVALID_ARG, "NULL buffer");
    const WorkLayout L = work_layout(h, ncols);
    if (static_cast<int64_t>(ws_bytes) < L.total) return fail(ERC_E_WORKSPACE, "workspace too small");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const Work w = carve_work(h, ncols, ws_dev, L);
    erc_status st = prepare_work(h, w, L, s);
    if (st != ERC_OK) return st;
    ERC_HIP(launch_spmm(h->dg, w, h->dt, delta, X_dev, X_dev, Y_dev, w.cs.one, s));
    return ERC_OK;
  });
}

erc_status erc_debug_solve_block(erc_handle h, const erc_solve_params* params, int32_t col0,
                                 int32_t ncols, void* ws_dev, size_t ws_bytes, void* Z_dev,
                                 int32_t* iters_host, void* stream) {
  return guarded([&]() -> erc_status {
    g_last_error.clear();
    if (check_handle(h) != ERC_OK) return ERC_E_INVALID_ARG;
    erc_status st = check_params(h, params);
    if (st != ERC_OK) return st;
    if (ncols < 1 || ncols > params->k_block || col0 < 0 || col0 + ncols > params->K_total)
      return fail(ERC_E_INVALID_ARG, "bad column range");
    if (Z_dev == nullptr || ws_dev == nullptr) return fail(ERC_E_INVALID_ARG, "NULL buffer");
    const int kb = padded_width(h->dt, params->k_block);
    const WorkLayout L = work_layout(h, kb);
    if (static_cast<int64_t>(ws_bytes) < L.total) return fail(ERC_E_WORKSPACE, "workspace too small");
    hipStream_t s = static_cast<hipStream_t>(stream);
    Work w = carve_work(h, kb, ws_dev, L, (params->flags & ERC_JACOBI) ? 1 : 0);
    if (params->flags & ERC_EARLY_STOP) w.fin2 = 1;
    st = prepare_work(h, w, L, s);
    if (st != ERC_OK) return st;
    BlockStats bs;
    st = solve_block(h, params, w, col0, ncols, nullptr, 0, iters_host, &bs, s);
    if (st != ERC_OK) return st;
    ERC_HIP(launch_copy_cols(h->dg, w.z, kb, h->dt, ncols, Z_dev, s));
    ERC_HIP(hipStreamSynchronize(s));
    if (bs.breakdowns > 0) return fail(ERC_E_NUMERIC, "CG breakdown");
    if (bs.unconverged > 0) return fail(ERC_E_NOT_CONVERGED, "column(s) reached max_iter");
    return ERC_OK;
  });
}

}  // extern "C"
