// Internal declarations shared by the host library and the HIP kernels.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "../../include/erc.h"

namespace erc {

// Threads per block of every kernel (4 wavefronts of 64).
constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / 64;
// Fan-in of one level of the deterministic grid reduction tree.
constexpr int kTreeFan = 32;
// Largest grid of a kernel whose block partials are reduced by a finishing launch.
constexpr int kMaxGrid = 8192;
// Largest grid of a launch that reduces through the ticket tree directly.
constexpr int kMaxTreeGrid = 2048;

// Device view of the graph operator (all pointers are device memory inside the
// caller's graph buffer).
// A light row of the SpMM plan with its CSR range, so that one 16-byte load gives a
// lane group everything it needs to start on the row.
struct alignas(16) LightRow {
  int64_t beg;  // rowptr[row]
  int32_t row;
  int32_t deg;  // rowptr[row + 1] - rowptr[row]
};

struct DevGraph {
  int32_t n;
  int64_t nnz;
  int64_t m;
  int weighted;              // 0: unit weights, w == nullptr
  const int64_t* rowptr;     // n+1
  const int32_t* col;        // nnz, ascending per row
  const void* w;             // nnz, working precision
  const int32_t* eid;        // nnz, canonical edge id of each entry
  const double* sw;          // m, sqrt(w_e) rounded once from fp64(w_e)
  int sw_from_w;             // 1 if w holds the input weights exactly (sqrt on the fly)
  const int64_t* ubase;      // n+1, id of the first edge (u, v>u) of row u
  const double* deg;         // n, d_i = sum_j w_ij in fp64 (diagonal of L)

  // SpMM plan: per-wave ranges over `light`, plus block-cooperative tasks for long rows
  int32_t grid;              // blocks of the SpMM kernel
  const LightRow* light;     // light rows, ascending, with their CSR ranges
  const int32_t* wave_lo;    // grid*4 + 1 boundaries into `light`
  int32_t ntask;             // block tasks (task t runs on block t % grid)
  const int32_t* task_row;
  const int32_t* task_mega;  // -1, or index of the multi-chunk row this chunk belongs to
  const int32_t* task_chunk; // chunk index within its row (0 for single-chunk rows)
  const int64_t* task_beg;   // CSR range of the task
  const int64_t* task_end;
  int32_t nmega;
  const int32_t* mega_row;     // row of each multi-chunk row
  const int32_t* mega_nchunk;
  const int32_t* mega_chunk0;  // first chunk slot of each multi-chunk row
  int32_t nchunk_slots;

  // Edge pieces: ranges of the upper (v > u) entries of one row, for per-edge kernels
  int64_t npiece;
  const int32_t* piece_row;
  const int64_t* piece_beg;  // CSR position
  const int64_t* piece_end;
};

// Per-column CG state of one block, in the workspace.
struct ColState {
  double* rho;      // current r.r, or r.M^-1 r with the Jacobi variant (fp64)
  double* rr;       // current r.r (stopping test and final relative residual)
  double* rho0;     // r.r of the right-hand side
  double* thr;      // tol^2 * rho0
  double* alpha;    // step of the current iteration
  double* beta;     // direction update of the current iteration
  int32_t* active;  // 1 while the column iterates
  int32_t* iters;   // iterations taken
  int32_t* status;  // 0 ok, 1 breakdown
  int32_t* n_active;  // one int: number of active columns (polled by the host)
  int32_t* upd_pending;  // one int: an update ran whose r.r is not yet reduced
  int32_t* pred_done;  // one int: every active column is predicted to stop after the
                       // pending update, so its exact test runs before the next SpMM
  int32_t* nspmm;      // one int: SpMM launches of this block that found active columns
  unsigned long long* fin_word;  // finishing-step counter word: active columns, columns
                                 // predicted to go on and blocks done; zero between launches
  int32_t* one;       // one int holding 1 (keeps debug launches from exiting early)
};

// Reduction scratch for one kernel family: level buffers and tickets.
struct Tree {
  double* lvl0;     // grid * nval
  double* lvl1;     // ceil(grid/32) * nval
  double* lvl2;     // ceil(grid/1024) * nval
  uint32_t* tick;   // ceil(grid/32) + ceil(grid/1024) + 1 counters, zero between launches
};

// Workspace of one column block of padded width kb.
struct Work {
  int kb;            // padded width
  void* z;           // n x kb
  void* r;
  void* p;
  void* q;
  void* chunkbuf;    // nchunk_slots x kb fp64 partial sums of multi-chunk rows
  double* mega_dots; // nmega x 3 x kb compensated (s, c) pairs
  ColState cs;
  double* part;      // block partials of the SpMM / RHS launch: grid x 3 x kb pairs
  double* part_u;    // block partials of the update launch: grid_upd x kb pairs
  Tree tree;         // tickets and levels of the small finishing launches
  double* out;       // small fp64 output area (totals for the host)
  void* minv;        // n: 1 / (d_i + delta) in the working precision (Jacobi variant)
  int pc;            // 1: Jacobi-preconditioned CG, 0: plain CG
  int fin2;          // 1: enqueue the early exact stopping test after each update
  int32_t grid_rhs, grid_upd, grid_ed;
};

// Launchers (erc_kernels.hip).  All return hipSuccess or the launch error.
hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t count, hipStream_t s);
hipError_t launch_fill_f64(double* p, double v, int64_t count, hipStream_t s);
hipError_t launch_rhs(const DevGraph& g, const Work& w, erc_dtype dt, int K, int col0, int ncols,
                      uint64_t base, double inv_sqrt_k, double tol, hipStream_t s);
hipError_t launch_spmm(const DevGraph& g, const Work& w, erc_dtype dt, double delta,
                       const void* p, const void* r, void* q, const int32_t* gate,
                       hipStream_t s);
hipError_t launch_update(const DevGraph& g, const Work& w, erc_dtype dt, hipStream_t s);
// w.minv[i] = 1 / (d_i + delta), rounded to the working precision
hipError_t launch_minv(const DevGraph& g, const Work& w, erc_dtype dt, double delta, hipStream_t s);
hipError_t launch_fin_iter(const DevGraph& g, const Work& w, int mode, hipStream_t s);
hipError_t launch_edge_dist(const DevGraph& g, const Work& w, erc_dtype dt, double* R,
                            int accumulate, hipStream_t s);
hipError_t launch_count_bad(const double* x, int64_t count, const Work& w, hipStream_t s);
hipError_t launch_copy_cols(const DevGraph& g, const void* src, int kb, erc_dtype dt, int ncols,
                            void* dst, hipStream_t s);
hipError_t launch_node_p(const DevGraph& g, erc_dtype dt, const double* R, double* p,
                         hipStream_t s);
hipError_t launch_edge_kappa(const DevGraph& g, const double* R, const double* p, double* kappa,
                             hipStream_t s);
hipError_t launch_endpoints(const DevGraph& g, int32_t* u, int32_t* v, hipStream_t s);
hipError_t launch_eids(const DevGraph& g, int32_t* out, hipStream_t s);

struct SampleWork {
  double* part_mm;   // grid x 3 block partials (-kappa_min, kappa_max, non-finite flag),
                     // then grid edge-weight block sums
  double* part_n;    // up to grid node-weight block sums
  double* totals;    // [0] -kappa_min, [1] kappa_max, [2] node sum, [3] edge sum, [4] bad flag
  int32_t grid;
};
hipError_t launch_sampling(const DevGraph& g, const double* kappa, double eta, int64_t nonisolated,
                           const SampleWork& sw, double* pn, double* pe, hipStream_t s);

// Fixed device scratch (erc_static.hip) of erc_sampling_probs_static.
constexpr size_t kStaticScratchBytes = 64 << 10;
// Looks up this process's copy of the array on `device`, which must be current; once
// per device, later calls return at once.
hipError_t static_scratch_setup(int device);
// The looked-up device address, or nullptr before static_scratch_setup succeeded.
void* static_scratch_ptr(int device);

// Gather probe (erc_probe.hip): rows of sums it stores for `count` indices, and launch.
int64_t probe_out_rows(int64_t count);
hipError_t launch_probe_gather(const int32_t* idx, int64_t count, const void* table, int64_t rows,
                               int row_bytes, int slices, void* out, hipStream_t s);

// Tree sizing helpers (host).
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t tree_ticks(int grid) {
  return ceil_div(grid, kTreeFan) + ceil_div(grid, kTreeFan * kTreeFan) + 1;
}

// Subgraph draws (erc_draw.hip).  Status bits a launch leaves in its status word.
constexpr uint32_t kDrawBadProb = 1u;      // a probability outside [0, 1] or NaN
constexpr uint32_t kDrawSumTooLarge = 2u;  // probabilities sum above 1.5
constexpr uint32_t kDrawAllZero = 4u;      // every integer weight is zero
constexpr uint32_t kSubBadIndex = 8u;      // a drawn index outside the node or edge range
constexpr int64_t kScanTile = 4096;        // items per block of the prefix-sum kernels
inline int64_t scan_blocks(int64_t items) { return ceil_div(items, kScanTile); }

struct DrawWork {
  uint64_t* cdf;     // N+1: exclusive prefix sums of the integer weights, cdf[N] = total
  uint64_t* bsum;    // scan_blocks(N) block sums
  double* psum;      // scan_blocks(N) fp64 block sums of the probabilities
  uint32_t* status;  // one word, zero before the launch
};
struct SubgraphWork {
  uint32_t* npos;    // n+1: node flags, then their exclusive prefix sums (new ids)
  uint32_t* epos;    // m+1: edge flags, then their exclusive prefix sums
  uint32_t* bsum;    // scan_blocks(max(n, m)) block sums
  uint32_t* status;  // one word, zero before the launch
};
hipError_t launch_draw(const double* prob, int64_t N, int64_t draws, uint64_t base,
                       const DrawWork& w, int64_t* idx, hipStream_t s);
// items 0: subgraph induced on the nodes in idx; 1: the edges in idx and their endpoints
hipError_t launch_subgraph(const DevGraph& g, int items, const int64_t* idx, int64_t count,
                           const SubgraphWork& w, int32_t* nodes, int64_t* edges, int32_t* uo,
                           int32_t* vo, hipStream_t s);

}  // namespace erc
