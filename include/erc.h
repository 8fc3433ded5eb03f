/*
 * erc.h -- C ABI of the MI355X resistance-curvature library.
 *
 * The library computes, on one gfx950 GPU, the ERC-LG approximation of effective
 * resistance curvature described in "Scalable Subgraph Sampling via Resistance
 * Curvature" (Fei, Zhou, Hao, Li):
 *
 *   1. Y = B^T W^{1/2} Q for streamed blocks of a K-column JL projection Q with
 *      entries +-1/sqrt(K)                          (Section 3.1.2; Algorithm 1)
 *   2. (L + delta I) Z = Y by column-wise CG to relative residual tol
 *                                                   (Eq. 5; Section 3.1.3; Alg. 1)
 *   3. R_uv += ||Z_u - Z_v||^2 per edge, block by block        (Eq. 6; Alg. 1)
 *   4. p_u = 1 - 1/2 sum_v w_uv R_uv,  kappa_uv = 2 (p_u + p_v) / R_uv   (Eq. 2)
 *   5. node / edge sampling probabilities                (Eqs. 7, 8; Section 3.2)
 *
 * Conventions shared by every call
 *  - Every function returns an erc_status; nothing is thrown across the ABI (host-side
 *    failures such as an allocation that cannot be served become ERC_E_HOST).  On an
 *    error, erc_last_error() returns a message (thread-local, valid until the next
 *    call on the same thread).
 *  - "host" pointers are ordinary CPU memory; "device" pointers are GPU memory on the
 *    current HIP device, owned by the caller.  The library never allocates device
 *    memory: the graph copy and the solve workspace live in caller buffers whose
 *    sizes come from erc_graph_bytes / erc_workspace_bytes, and those buffers must
 *    outlive every call that uses them.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).  All
 *    device work is enqueued on it.  erc_create and erc_resistance return after the
 *    stream has drained; the other calls are asynchronous.
 *  - Edges are numbered canonically: edge e is the e-th pair (u, v), u < v, in
 *    lexicographic order.  Every per-edge array (R, kappa, edge probabilities) is
 *    indexed by that number.  The incidence matrix B has +1 at u and -1 at v.
 *  - A handle is not thread-safe; distinct handles are independent.
 */
#ifndef ERC_H
#define ERC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ERC_OK = 0,
  ERC_E_INVALID_ARG = 1,     /* NULL pointer, bad size, out-of-range parameter        */
  ERC_E_INVALID_GRAPH = 2,   /* CSR not symmetric / unsorted / self-loop / bad weight  */
  ERC_E_WORKSPACE = 3,       /* caller buffer smaller than the size query returned    */
  ERC_E_DEVICE = 4,          /* a HIP runtime call failed                              */
  ERC_E_NOT_CONVERGED = 5,   /* some column hit max_iter above tol (result written)    */
  ERC_E_NUMERIC = 6,         /* CG breakdown (p.q <= 0 or non-finite), R <= 0, NaN     */
  ERC_E_STATE = 7,           /* handle used in an invalid state                        */
  ERC_E_HOST = 8             /* host memory could not be allocated or a thread started */
} erc_status;

typedef enum { ERC_F32 = 0, ERC_F64 = 1 } erc_dtype;

/* Opaque host-side handle: device pointers into the caller's graph buffer plus the
 * host-side plan (sizes, row work lists). */
typedef struct erc_graph_s* erc_handle;

/* Undirected graph as a symmetric CSR adjacency (Section 3.1.1: L = D - A = B^T W B).
 *  n           number of nodes (0 < n < 2^31)
 *  rowptr      host, n+1 int64, rowptr[0] = 0, non-decreasing, rowptr[n] = nnz < 2^31
 *  col         host, nnz int32 column indices, strictly ascending within each row
 *  w           host, nnz weights of type w_dtype, or NULL for unit weights; every
 *              weight finite and > 0, and w_ij == w_ji exactly
 *  w_dtype     type of w (ignored when w == NULL)
 *  solve_dtype working precision of the CG vectors: ERC_F32 or ERC_F64.  With
 *              ERC_F32 the dot products, R, p, kappa and the probabilities are
 *              still fp64, and the SpMM sums the rows it runs as block tasks
 *              (more than max(1024, two wavefront shares) entries) in fp64 and the
 *              other rows in fp32
 * The structure must be symmetric with no self-loops and no repeated entries; each
 * undirected edge is stored twice.  Isolated nodes are allowed. */
typedef struct {
  int64_t n;
  const int64_t* rowptr;
  const int32_t* col;
  const void* w;
  erc_dtype w_dtype;
  erc_dtype solve_dtype;
} erc_graph_desc;

/* Accumulate into R instead of overwriting it (resume, column-range sharding). */
#define ERC_ACCUMULATE 1u
/* Time every SpMM launch with a pair of HIP events on the caller's stream and report
 * the sum in erc_solve_info.ms_spmm / spmm_timed (adds two event records per launch). */
#define ERC_PROFILE_SPMM 2u
/* Solve with Jacobi-preconditioned CG (M^-1 = diag(1 / (d_i + delta)), d_i = sum_j w_ij)
 * instead of the paper's plain column-wise CG (Section 3.1.3).  Same stopping test
 * (||r|| <= tol ||y|| on the unpreconditioned residual) and outputs; on graphs with
 * widely spread degrees it needs far fewer iterations.  A variant, not the paper's
 * method: results equal the plain solve only up to the CG truncation error. */
#define ERC_JACOBI 4u
/* Enqueue every CG iteration as separate kernel launches.  By default each group of
 * check_every iterations is captured once into a HIP graph (on a stream the handle
 * owns) and replayed on the caller's stream, which removes most of the per-launch
 * overhead on small graphs; the kernels, their order and the results are the same.
 * ERC_PROFILE_SPMM implies this flag (its events sit between the launches). */
#define ERC_NO_GRAPH 8u
/* Enqueue, after every CG update, the exact stopping test that runs only when every
 * active column is predicted to stop (it saves the one SpMM that would otherwise follow
 * a block's last update).  By default it is enqueued only where an SpMM gathers at
 * least 4 GB of neighbour rows (nnz * k_block * element size), because elsewhere the
 * extra launch per iteration costs more than the SpMM it saves.  Results are the same
 * either way. */
#define ERC_EARLY_STOP 16u

/* Parameters of one resistance sweep (Algorithm 1, Require line).
 *  K_total     total projection dimension K; the JL scale is 1/sqrt(K_total) even when
 *              only a column range is solved (1 <= K_total)
 *  k_block     columns per CG block, the paper's batch size b (1..256 for ERC_F32,
 *              1..128 for ERC_F64); a block is padded internally to a power of two
 *              (>= 16 columns for ERC_F32, >= 8 for ERC_F64)
 *  col_begin, col_end   global column range [col_begin, col_end) of the sketch to
 *              solve, 0 <= col_begin < col_end <= K_total
 *  delta       diagonal shift (the paper's epsilon in Eq. 5), delta > 0
 *  tol         per-column relative residual tolerance tau (0 < tol < 1): a column
 *              stops once ||r|| <= tol ||y|| on the recursively updated residual
 *  max_iter    iteration cap per block (>= 1)
 *  check_every iterations enqueued between host convergence polls (0 = default 16);
 *              results do not depend on it
 *  seed        projection seed
 *  flags       ERC_ACCUMULATE | ERC_PROFILE_SPMM | ERC_JACOBI | ERC_NO_GRAPH |
 *              ERC_EARLY_STOP, or 0 */
typedef struct {
  int32_t K_total;
  int32_t k_block;
  int32_t col_begin;
  int32_t col_end;
  double delta;
  double tol;
  int32_t max_iter;
  int32_t check_every;
  uint64_t seed;
  uint32_t flags;
} erc_solve_params;

/* Filled by erc_resistance when non-NULL. */
typedef struct {
  int32_t blocks;             /* column blocks solved                                */
  int32_t iters_max;          /* largest per-column iteration count                  */
  int32_t cols_unconverged;   /* columns that reached max_iter above tol             */
  int32_t breakdowns;         /* columns stopped by p.q <= 0 or a non-finite value   */
  int64_t iters_total;        /* sum over columns of their iteration counts          */
  int64_t launches;           /* CG iterations enqueued (per block, summed)          */
  int64_t nonpositive;        /* entries of R that are <= 0 or not finite at the end */
  double max_final_relres;    /* max over columns of sqrt(rho_final / rho_0)         */
  float ms_rhs;               /* GPU time building right-hand sides                  */
  float ms_cg;                /* GPU time in CG iterations                           */
  float ms_accum;             /* GPU time in edge-distance accumulation              */
  float ms_total;             /* whole call, stream time                             */
  float ms_spmm;              /* with ERC_PROFILE_SPMM: summed SpMM kernel time      */
  int64_t spmm_timed;         /* with ERC_PROFILE_SPMM: SpMM launches timed          */
  int64_t spmm_full;          /* SpMM launches that found an active column (the rest
                                 return at once after convergence)                   */
  double bytes_model;         /* algorithmic HBM bytes of the call: per SpMM and update
                                 that found active columns, one pass over every array
                                 they read or write (neighbour gathers counted once),
                                 plus right-hand sides and edge distances per block   */
} erc_solve_info;

/* ---- graph ---------------------------------------------------------------------- */

/* Host-only validation of a graph description (no GPU needed).  On success *m_out
 * (if non-NULL) receives the number of undirected edges.
 * Errors: ERC_E_INVALID_ARG (NULL/size), ERC_E_INVALID_GRAPH (structure, weights). */
erc_status erc_validate(const erc_graph_desc* desc, int64_t* m_out);

/* Size in bytes of the device buffer erc_create needs for this graph (host-only). */
erc_status erc_graph_bytes(const erc_graph_desc* desc, size_t* bytes);

/* Validate and canonicalise the graph on the host, then copy the device copy of the
 * operator (CSR, weights, per-entry edge ids, sqrt(w) per edge, work lists) into
 * dev_mem (device, >= erc_graph_bytes bytes, 256-byte aligned) on `stream`, and wait
 * for the copy.  The handle refers to dev_mem, which must stay allocated until
 * erc_destroy.  (Algorithm 1: construct sparse L; store local sparse operators.) */
erc_status erc_create(const erc_graph_desc* desc, void* dev_mem, size_t bytes, void* stream,
                      erc_handle* out);

erc_status erc_num_nodes(erc_handle h, int64_t* n);
erc_status erc_num_edges(erc_handle h, int64_t* m);

/* Endpoints of every canonical edge: u_dev[e] < v_dev[e] (device, m int32 each). */
erc_status erc_edge_endpoints(erc_handle h, int32_t* u_dev, int32_t* v_dev, void* stream);

/* Frees the host-side handle only (the caller frees dev_mem).  NULL is accepted. */
erc_status erc_destroy(erc_handle h);

/* ---- resistance (Algorithm 1, Eqs. 3-6) ------------------------------------------ */

/* Device workspace size for blocks of k_block columns on this graph. */
erc_status erc_workspace_bytes(erc_handle h, int32_t k_block, size_t* bytes);

/* R_dev[e] (device, m fp64) = sum over the requested columns c of (Z_uc - Z_vc)^2,
 * where Z solves (L + delta I) Z = B^T W^{1/2} Q column by column with CG
 * (or += with ERC_ACCUMULATE).  ws_dev is device memory of >= erc_workspace_bytes
 * bytes.  The call blocks until the stream has drained.
 * Returns ERC_E_NOT_CONVERGED (R still written) when a column hit max_iter above tol,
 * ERC_E_NUMERIC on a CG breakdown or when some R_e ends <= 0 or non-finite (curvature
 * needs R_e > 0). */
erc_status erc_resistance(erc_handle h, const erc_solve_params* params, void* ws_dev,
                          size_t ws_bytes, double* R_dev, erc_solve_info* info,
                          void* stream);

/* ---- curvature and sampling (Eq. 2; Eqs. 7-8; Section 3.2) ------------------------ */

/* p_dev[u] (device, n fp64) = 1 - 1/2 sum_{v in N(u)} w_uv R_uv (1 for isolated u);
 * kappa_dev[e] (device, m fp64) = 2 (p_u + p_v) / R_e.  Asynchronous.  Each R_e should
 * be finite and > 0 (erc_resistance reports otherwise); the outputs are the IEEE
 * results of the formulas whatever R holds. */
erc_status erc_curvature(erc_handle h, const double* R_dev, double* p_dev, double* kappa_dev,
                         void* stream);

/* Node probabilities (device, n fp64): q_u = sum_{v in N(u)} (kappa_uv - kappa_min) /
 * (kappa_max - kappa_min + eta), divided by sum_u q_u; uniform over nodes of degree > 0
 * when every q_u is 0 (Eq. 7).  Edge probabilities (device, m fp64):
 * q_e = sqrt(max(2 kappa_max - kappa_e, 0)) + 1 divided by its sum (Eq. 8).
 * eta > 0.  scratch_dev is device memory of >= erc_sampling_scratch_bytes bytes.
 * Blocks until the stream has drained.  ERC_E_NUMERIC, with every probability written
 * as NaN, when some kappa_e is NaN or infinite. */
erc_status erc_sampling_scratch_bytes(erc_handle h, size_t* bytes);
erc_status erc_sampling_probs(erc_handle h, const double* kappa_dev, double eta,
                              void* scratch_dev, size_t scratch_bytes,
                              double* node_prob_dev, double* edge_prob_dev, void* stream);

/* erc_sampling_probs without a scratch argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same kernels and outputs as erc_sampling_probs; the scratch is a
 * fixed device array of the library (64 KiB per GPU, held until the process ends;
 * every graph's sampling scratch fits, ERC_E_WORKSPACE otherwise).  Every call on one
 * GPU uses that GPU's array, so calls that overlap on one GPU race: order them on one
 * stream.  The handle's device must be current.  Asynchronous: nothing is allocated
 * and the call does not wait, so a NaN or infinite kappa_e is not reported by status;
 * every probability is then written as NaN. */
erc_status erc_sampling_probs_static(erc_handle h, const double* kappa_dev, double eta,
                                     double* node_prob_dev, double* edge_prob_dev,
                                     void* stream);

/* ---- curvature-guided subgraph draws (Section 3.2; Section 4) --------------------- */

/* Which distribution a draw uses and what a subgraph is built from. */
typedef enum { ERC_NODES = 0, ERC_EDGES = 1 } erc_items;

/* Device scratch of erc_draw over the n nodes or the m edges. */
erc_status erc_draw_scratch_bytes(erc_handle h, erc_items items, size_t* bytes);

/* idx_dev[d] (device, draws int64), d = 0 .. draws-1: independent draws from the
 * distribution prob_dev (device fp64, n entries for ERC_NODES, m for ERC_EDGES; each in
 * [0, 1], summing to one up to rounding, as erc_sampling_probs writes them).
 * Definition: W_i = floor(P_i 2^62), C_i = sum_{j<i} W_j, T = C_N (exact 64-bit
 * integers); draw d takes X = x_hi 2^64 + x_lo with x_hi, x_lo the outputs 2d and 2d+1
 * of SplitMix64 started from the first output of SplitMix64(seed), t = floor(X T / 2^128),
 * and returns the i with C_i <= t < C_{i+1}.  Items with W_i = 0 are never drawn.
 * scratch_dev: >= erc_draw_scratch_bytes bytes.  Blocks until the stream has drained.
 * ERC_E_NUMERIC (idx_dev filled with -1) when a probability is NaN or outside [0, 1],
 * when they sum above 1.5, or when every W_i is 0. */
erc_status erc_draw(erc_handle h, erc_items items, const double* prob_dev, int64_t draws,
                    uint64_t seed, void* scratch_dev, size_t scratch_bytes, int64_t* idx_dev,
                    void* stream);

/* Device scratch of erc_subgraph. */
erc_status erc_subgraph_scratch_bytes(erc_handle h, size_t* bytes);

/* Training subgraph from count drawn indices idx_dev (device int64; repeats allowed).
 * ERC_NODES: the subgraph induced on the distinct drawn nodes.  ERC_EDGES: the distinct
 * drawn edges and their endpoints.  Outputs (device): nodes_dev (int32, capacity n) the
 * kept nodes in increasing id, which renumbers them 0..n_s-1; edges_dev (int64,
 * capacity m) the kept canonical edge ids in increasing order; u_dev, v_dev (int32,
 * capacity m) each kept edge's endpoints u < v in the new numbering.  counts_host[0] =
 * n_s, counts_host[1] = m_s (host).  Blocks until the stream has drained.
 * ERC_E_INVALID_ARG when an index is outside [0, n) or [0, m) (outputs undefined). */
erc_status erc_subgraph(erc_handle h, erc_items items, const int64_t* idx_dev, int64_t count,
                        void* scratch_dev, size_t scratch_bytes, int32_t* nodes_dev,
                        int64_t* edges_dev, int32_t* u_dev, int32_t* v_dev,
                        int64_t* counts_host, void* stream);

/* ---- diagnostics ----------------------------------------------------------------- */

const char* erc_status_string(erc_status s);
const char* erc_last_error(void);

/* ---- measurement hook (memory-system probe for the roofline of gather kernels) ----- */

/* Rows of row_bytes bytes that erc_probe_gather stores for `count` indices. */
erc_status erc_probe_out_bytes(int64_t count, int32_t row_bytes, size_t* bytes);

/* For every k in [0, count): load row idx_dev[k] of table_dev (device, rows x row_bytes
 * bytes, row-major, 16-byte aligned) with the SpMM's gather access pattern (row_bytes/16
 * lanes, one 16-byte load each, eight rows in flight per lane group) and sum the rows
 * of each contiguous range of indices into one row of out_dev (device,
 * erc_probe_out_bytes).  Indices outside [0, rows) read row 0.  row_bytes: a power of
 * two in 64..1024.  Replaying the SpMM's own column indices over a table of the
 * p block's size times its gathers alone; no part of the method is computed.
 * Asynchronous. */
erc_status erc_probe_gather(const int32_t* idx_dev, int64_t count, const void* table_dev,
                            int64_t rows, int32_t row_bytes, void* out_dev, void* stream);

/* erc_probe_gather over `slices` column slices of each row at once: table_dev holds rows
 * of slices * row_bytes bytes, and block b of the launch (slices times as many blocks)
 * gathers the row_bytes at offset (b % slices) * row_bytes of every indexed row for the
 * index range of b / slices.  Blocks go to the GPU's eight XCDs round-robin, so with
 * slices dividing 8 each XCD's L2 sees one slice only: this measures what a
 * column-sliced gather would gain from the smaller per-XCD footprint.  out_dev holds
 * slices * erc_probe_out_bytes(count, row_bytes) bytes.  slices in 1..64;
 * erc_probe_gather is slices = 1.  Asynchronous. */
erc_status erc_probe_gather_sliced(const int32_t* idx_dev, int64_t count, const void* table_dev,
                                   int64_t rows, int32_t row_bytes, int32_t slices,
                                   void* out_dev, void* stream);

/* ---- test hooks (same conventions; used by the parity tests) ---------------------- */

/* Host-only self-check of the work plan erc_create would build for this graph (no GPU
 * needed): every stored entry is covered exactly once by the SpMM plan, every upper
 * entry (v > u) exactly once by the per-edge pieces, every index is in range and every
 * list fits the size bounds behind erc_graph_bytes.  ERC_E_STATE names a violation. */
erc_status erc_debug_check_plan(const erc_graph_desc* desc);

/* Canonical edge id of every stored CSR entry (device, nnz int32). */
erc_status erc_debug_edge_ids(erc_handle h, int32_t* eid_dev, void* stream);

/* Right-hand sides of columns [col0, col0 + ncols) as an n x ncols row-major array in
 * the working precision (device).  1 <= ncols <= the maximum k_block; ws_dev: >=
 * erc_workspace_bytes(h, ncols).  Asynchronous. */
erc_status erc_debug_rhs(erc_handle h, int32_t K_total, int32_t col0, int32_t ncols,
                         uint64_t seed, void* Y_dev, void* ws_dev, size_t ws_bytes,
                         void* stream);

/* Y = (L + delta I) X for an n x ncols row-major X in the working precision (device).
 * ncols must be a padded block width: a power of two in 16..256 for ERC_F32, 8..128
 * for ERC_F64.  ws_dev: >= erc_workspace_bytes(h, ncols). */
erc_status erc_debug_spmm(erc_handle h, double delta, int32_t ncols, const void* X_dev,
                          void* Y_dev, void* ws_dev, size_t ws_bytes, void* stream);

/* Solve one block [col0, col0 + ncols) and copy its Z (n x ncols row-major, working
 * precision, device) out; per-column iteration counts go to iters_host (ncols int32,
 * may be NULL).  Blocks until the stream has drained.  Same return codes as
 * erc_resistance. */
erc_status erc_debug_solve_block(erc_handle h, const erc_solve_params* params, int32_t col0,
                                 int32_t ncols, void* ws_dev, size_t ws_bytes, void* Z_dev,
                                 int32_t* iters_host, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ERC_H */
