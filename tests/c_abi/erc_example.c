/*
 * The library used from C alone, through include/erc.h and the HIP runtime: no Python,
 * no torch.  erc_example_tree() builds a random weighted tree, sizes and allocates every
 * device buffer the calls need, runs resistance (fp64, one column block), curvature and
 * sampling probabilities, and checks the results against closed forms that hold for
 * every projection on a tree: each edge is a bridge, so its sketched resistance is 1/w_e
 * up to the shift (1e-12) and the CG tolerance (1e-13) (Section 3.1.2: a bridge's row of W^{1/2} B L^+
 * is a unit vector); then p_u = 1 - deg(u)/2 and kappa_uv = w_uv (4 - deg(u) - deg(v))
 * (Eq. 2), sum_u p_u = 1, and each probability vector sums to 1 (Eqs. 7-8).
 *
 * Built as a shared library (tests call erc_example_tree through ctypes, so no second
 * program is started from a process that uses the GPU).  Returns 0 when every check
 * holds; otherwise a non-zero code and a message in msg.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "erc.h"

#define FAIL(code, ...)                    \
  do {                                     \
    snprintf(msg, (size_t)msg_len, __VA_ARGS__); \
    rc = (code);                           \
    goto done;                             \
  } while (0)

#define ERC_OK_OR(call)                                                             \
  do {                                                                              \
    erc_status st_ = (call);                                                        \
    if (st_ != ERC_OK) FAIL(10 + (int)st_, "%s: %s (%s)", #call, erc_status_string(st_), \
                            erc_last_error());                                      \
  } while (0)

#define HIP_OK_OR(call)                                                             \
  do {                                                                              \
    hipError_t e_ = (call);                                                         \
    if (e_ != hipSuccess) FAIL(2, "%s: %s", #call, hipGetErrorString(e_));          \
  } while (0)

static uint64_t lcg(uint64_t* s) {
  *s = *s * 6364136223846793005ull + 1442695040888963407ull;
  return *s >> 11;
}

int erc_example_tree(int32_t n, uint64_t seed, char* msg, int32_t msg_len) {
  int rc = 0;
  int64_t nnz = 2 * (int64_t)(n - 1), m = 0;
  int64_t* rowptr = NULL;
  int32_t* col = NULL;
  double* w = NULL;
  int32_t* parent = NULL;
  double* pw = NULL;
  int32_t* deg = NULL;
  double *R = NULL, *p = NULL, *kappa = NULL, *pn = NULL, *pe = NULL;
  int32_t *eu = NULL, *ev = NULL;
  void *d_graph = NULL, *d_ws = NULL, *d_scratch = NULL;
  double *d_R = NULL, *d_p = NULL, *d_kappa = NULL, *d_pn = NULL, *d_pe = NULL;
  int32_t *d_u = NULL, *d_v = NULL;
  erc_handle h = NULL;
  hipStream_t stream = NULL;
  if (n < 2 || msg == NULL || msg_len < 1) return 1;
  msg[0] = '\0';

  /* a random recursive tree: node i > 0 hangs off a uniform earlier node, with weight
   * in [0.5, 2) */
  parent = (int32_t*)calloc((size_t)n, sizeof(int32_t));
  pw = (double*)calloc((size_t)n, sizeof(double));
  deg = (int32_t*)calloc((size_t)n, sizeof(int32_t));
  rowptr = (int64_t*)calloc((size_t)n + 1, sizeof(int64_t));
  col = (int32_t*)calloc((size_t)nnz, sizeof(int32_t));
  w = (double*)calloc((size_t)nnz, sizeof(double));
  if (!parent || !pw || !deg || !rowptr || !col || !w) FAIL(3, "host allocation");
  uint64_t s = seed;
  for (int32_t i = 1; i < n; ++i) {
    parent[i] = (int32_t)(lcg(&s) % (uint64_t)i);
    pw[i] = 0.5 + 1.5 * (double)(lcg(&s) >> 11) / 9007199254740992.0;
    deg[i] += 1;
    deg[parent[i]] += 1;
  }
  for (int32_t i = 0; i < n; ++i) rowptr[i + 1] = rowptr[i] + deg[i];
  {
    /* symmetric CSR with ascending columns: the neighbours of u are its parent (smaller
     * id) and its children (larger ids, in increasing order) */
    int64_t* fill = (int64_t*)calloc((size_t)n, sizeof(int64_t));
    if (!fill) FAIL(3, "host allocation");
    for (int32_t i = 0; i < n; ++i) fill[i] = rowptr[i];
    for (int32_t i = 1; i < n; ++i) {
      col[fill[i]] = parent[i];
      w[fill[i]++] = pw[i];
    }
    for (int32_t i = 1; i < n; ++i) {
      col[fill[parent[i]]] = i;
      w[fill[parent[i]]++] = pw[i];
    }
    free(fill);
  }

  erc_graph_desc desc;
  memset(&desc, 0, sizeof desc);
  desc.n = n;
  desc.rowptr = rowptr;
  desc.col = col;
  desc.w = w;
  desc.w_dtype = ERC_F64;
  desc.solve_dtype = ERC_F64;
  ERC_OK_OR(erc_validate(&desc, &m));
  if (m != n - 1) FAIL(4, "erc_validate counted %lld edges, expected %d", (long long)m, n - 1);

  HIP_OK_OR(hipStreamCreate(&stream));
  size_t gbytes = 0, wbytes = 0, sbytes = 0;
  ERC_OK_OR(erc_graph_bytes(&desc, &gbytes));
  HIP_OK_OR(hipMalloc(&d_graph, gbytes));
  ERC_OK_OR(erc_create(&desc, d_graph, gbytes, stream, &h));

  const int32_t kb = 32;
  ERC_OK_OR(erc_workspace_bytes(h, kb, &wbytes));
  HIP_OK_OR(hipMalloc(&d_ws, wbytes));
  HIP_OK_OR(hipMalloc((void**)&d_R, (size_t)m * 8));
  HIP_OK_OR(hipMalloc((void**)&d_p, (size_t)n * 8));
  HIP_OK_OR(hipMalloc((void**)&d_kappa, (size_t)m * 8));
  HIP_OK_OR(hipMalloc((void**)&d_pn, (size_t)n * 8));
  HIP_OK_OR(hipMalloc((void**)&d_pe, (size_t)m * 8));
  HIP_OK_OR(hipMalloc((void**)&d_u, (size_t)m * 4));
  HIP_OK_OR(hipMalloc((void**)&d_v, (size_t)m * 4));
  ERC_OK_OR(erc_sampling_scratch_bytes(h, &sbytes));
  HIP_OK_OR(hipMalloc(&d_scratch, sbytes));

  erc_solve_params prm;
  memset(&prm, 0, sizeof prm);
  prm.K_total = kb;
  prm.k_block = kb;
  prm.col_begin = 0;
  prm.col_end = kb;
  prm.delta = 1e-12;
  prm.tol = 1e-13;
  prm.max_iter = 20000;
  prm.seed = seed;
  erc_solve_info info;
  ERC_OK_OR(erc_resistance(h, &prm, d_ws, wbytes, d_R, &info, stream));
  ERC_OK_OR(erc_curvature(h, d_R, d_p, d_kappa, stream));
  ERC_OK_OR(erc_sampling_probs(h, d_kappa, 1e-12, d_scratch, sbytes, d_pn, d_pe, stream));
  ERC_OK_OR(erc_edge_endpoints(h, d_u, d_v, stream));
  HIP_OK_OR(hipStreamSynchronize(stream));

  R = (double*)malloc((size_t)m * 8);
  kappa = (double*)malloc((size_t)m * 8);
  pe = (double*)malloc((size_t)m * 8);
  p = (double*)malloc((size_t)n * 8);
  pn = (double*)malloc((size_t)n * 8);
  eu = (int32_t*)malloc((size_t)m * 4);
  ev = (int32_t*)malloc((size_t)m * 4);
  if (!R || !kappa || !pe || !p || !pn || !eu || !ev) FAIL(3, "host allocation");
  HIP_OK_OR(hipMemcpy(R, d_R, (size_t)m * 8, hipMemcpyDeviceToHost));
  HIP_OK_OR(hipMemcpy(kappa, d_kappa, (size_t)m * 8, hipMemcpyDeviceToHost));
  HIP_OK_OR(hipMemcpy(pe, d_pe, (size_t)m * 8, hipMemcpyDeviceToHost));
  HIP_OK_OR(hipMemcpy(p, d_p, (size_t)n * 8, hipMemcpyDeviceToHost));
  HIP_OK_OR(hipMemcpy(pn, d_pn, (size_t)n * 8, hipMemcpyDeviceToHost));
  HIP_OK_OR(hipMemcpy(eu, d_u, (size_t)m * 4, hipMemcpyDeviceToHost));
  HIP_OK_OR(hipMemcpy(ev, d_v, (size_t)m * 4, hipMemcpyDeviceToHost));

  /* canonical edges of a tree: (parent(v), v) sorted by (parent, v); edge e = (u < v)
   * must be a tree edge with v's parent u */
  double worst_R = 0.0, worst_p = 0.0, worst_k = 0.0, sum_p = 0.0, sum_pn = 0.0, sum_pe = 0.0;
  for (int64_t e = 0; e < m; ++e) {
    const int32_t u = eu[e], v = ev[e];
    if (!(u < v) || v >= n || parent[v] != u) FAIL(5, "edge %lld = (%d, %d) is not a tree edge", (long long)e, u, v);
    if (e > 0 && !(eu[e - 1] < u || (eu[e - 1] == u && ev[e - 1] < v))) FAIL(5, "edges not in canonical order at %lld", (long long)e);
    const double r = fabs(R[e] * pw[v] - 1.0);
    if (r > worst_R) worst_R = r;
    const double kx = pw[v] * (4.0 - deg[u] - deg[v]);
    const double ke = fabs(kappa[e] - kx) / (fabs(kx) + 2.0 * pw[v] * 0.5 * (deg[u] + deg[v]));
    if (ke > worst_k) worst_k = ke;
    sum_pe += pe[e];
  }
  for (int32_t u = 0; u < n; ++u) {
    const double px = 1.0 - 0.5 * deg[u];
    const double pd = fabs(p[u] - px) / (0.5 * deg[u]);
    if (pd > worst_p) worst_p = pd;
    sum_p += p[u];
    sum_pn += pn[u];
  }
  if (info.cols_unconverged != 0 || info.breakdowns != 0) FAIL(6, "solve: %d unconverged, %d breakdowns", info.cols_unconverged, info.breakdowns);
  if (worst_R > 1e-7) FAIL(7, "R_e w_e - 1 up to %.3e", worst_R);
  if (worst_p > 1e-7) FAIL(7, "p_u off by %.3e of its scale", worst_p);
  if (worst_k > 1e-7) FAIL(7, "kappa off by %.3e of its scale", worst_k);
  if (fabs(sum_p - 1.0) > 1e-6 * n) FAIL(7, "sum of p = %.12f", sum_p);
  if (fabs(sum_pn - 1.0) > 1e-12 || fabs(sum_pe - 1.0) > 1e-12) FAIL(7, "probabilities sum to %.15f and %.15f", sum_pn, sum_pe);
  snprintf(msg, (size_t)msg_len,
           "tree n=%d: R*w-1 %.2e, p %.2e, kappa %.2e, sum p %.9f, %d iterations", n,
           worst_R, worst_p, worst_k, sum_p, info.iters_max);

done:
  if (h) erc_destroy(h);
  hipFree(d_graph); hipFree(d_ws); hipFree(d_scratch); hipFree(d_R); hipFree(d_p);
  hipFree(d_kappa); hipFree(d_pn); hipFree(d_pe); hipFree(d_u); hipFree(d_v);
  if (stream) hipStreamDestroy(stream);
  free(parent); free(pw); free(deg); free(rowptr); free(col); free(w);
  free(R); free(p); free(kappa); free(pn); free(pe); free(eu); free(ev);
  return rc;
}
