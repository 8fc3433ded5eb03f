"""The oracle's pins must catch a planted mistake.

Each case copies oracle/ into a temporary directory, changes one expression of one
module (a dropped factor or term, a wrong sign, index, constant or comparison: the
mistakes a reading of the paper, or a slip in writing it down, plausibly makes), and
runs the oracle's own pin tests for that module (tests/test_oracle_*.py) against the
copy in a child process.  The unchanged copy must pass them; every changed copy must make at least one
of them fail (pytest exit status 1: a failed test, not an import or collection error).
CPU only; the HIP library is not involved.
"""
import glob
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor


ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_TESTS = sorted(glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py")))
# the pin files that exercise each module (a mutant runs only these, to keep time down)
_T = os.path.join(ROOT, "tests")
PINS_OF = {
    "erc.py": [os.path.join(_T, f) for f in ("test_oracle_pipeline.py", "test_oracle_exact.py",
                                             "test_oracle_pcg.py")],
    "hashing.py": [os.path.join(_T, "test_oracle_hash.py")],
    "graph.py": [os.path.join(_T, "test_oracle_exact.py")],
    "exact.py": [os.path.join(_T, f) for f in ("test_oracle_exact.py", "test_oracle_pipeline.py",
                                               "test_oracle_agreement.py")],
    "accurate.py": [os.path.join(_T, "test_oracle_accurate.py")],
    "sampling.py": [os.path.join(_T, "test_oracle_sampling.py")],
    "agreement.py": [os.path.join(_T, "test_oracle_agreement.py")],
    "parallel.py": [os.path.join(_T, "test_oracle_parallel.py")],
}

# (id, module, original text, planted text); the first occurrence is changed, which for
# the CG recurrences is the plain CG (cg_columns precedes pcg_columns)
MUTANTS = [
    # Y = B^T W^{1/2} Q (Section 3.1.2)
    ("rhs_orientation", "erc.py", "orient = np.where(rows[live] < col[pos], 1.0, -1.0)",
     "orient = np.where(rows[live] > col[pos], 1.0, -1.0)"),
    ("rhs_scale_1_over_K", "erc.py", "inv_sqrt_k = 1.0 / math.sqrt(K)", "inv_sqrt_k = 1.0 / K"),
    ("rhs_w_not_sqrt_w", "erc.py", "sw = np.sqrt(GR.edge_weights(g))", "sw = GR.edge_weights(g)"),
    # (L + delta I) Z = Y by column-wise CG (Eq. 5, Section 3.1.3)
    ("operator_minus_delta", "erc.py", "return L @ X + delta * X", "return L @ X - delta * X"),
    ("cg_beta_inverted", "erc.py", "beta = rho_new / rho[a]", "beta = rho[a] / rho_new"),
    ("cg_residual_sign", "erc.py", "Ra = R[:, a] - alpha * Qa", "Ra = R[:, a] + alpha * Qa"),
    ("cg_iterate_not_updated", "erc.py", "Z[:, a] += alpha * Pa", "Z[:, a] += Pa"),
    ("cg_stop_tol_not_squared", "erc.py", "thr = tol * tol * rho0", "thr = tol * rho0"),
    # the Jacobi-preconditioned variant
    ("pcg_direction_unpreconditioned", "erc.py",
     "P[:, a[keep]] = Sa[:, keep] + beta[keep] * Pa[:, keep]",
     "P[:, a[keep]] = Ra[:, keep] + beta[keep] * Pa[:, keep]"),
    ("pcg_rho_r_dot_r", "erc.py", "rho_new = dot2_columns(Ra, Sa)", "rho_new = dot2_columns(Ra, Ra)"),
    ("pcg_diagonal_without_shift", "erc.py",
     "return 1.0 / (np.asarray(L.diagonal(), dtype=np.float64) + delta)",
     "return 1.0 / np.asarray(L.diagonal(), dtype=np.float64)"),
    # R_e = ||Z_u - Z_v||^2 (Eq. 6)
    ("distance_not_squared", "erc.py", 'np.einsum("ij,ij->i", d, d)',
     'np.sqrt(np.einsum("ij,ij->i", d, d))'),
    # p and kappa (Eq. 2)
    ("curvature_no_half", "erc.py", "p = 1.0 - 0.5 * s", "p = 1.0 - s"),
    ("curvature_no_two", "erc.py", "kappa = 2.0 * (p[eu] + p[ev]) / R",
     "kappa = (p[eu] + p[ev]) / R"),
    ("curvature_wrong_endpoint", "erc.py", "kappa = 2.0 * (p[eu] + p[ev]) / R",
     "kappa = 2.0 * (p[eu] + p[eu]) / R"),
    ("curvature_weight_dropped", "erc.py", "weights=w * R[eid]", "weights=R[eid]"),
    # sampling weights (Eqs. 7, 8)
    ("edge_weight_no_sqrt", "erc.py", "np.sqrt(np.maximum(2.0 * kmax - kappa, 0.0)) + 1.0",
     "np.maximum(2.0 * kmax - kappa, 0.0) + 1.0"),
    ("edge_weight_kmax_not_doubled", "erc.py",
     "np.sqrt(np.maximum(2.0 * kmax - kappa, 0.0)) + 1.0",
     "np.sqrt(np.maximum(kmax - kappa, 0.0)) + 1.0"),
    ("edge_weight_no_plus_one", "erc.py", "np.sqrt(np.maximum(2.0 * kmax - kappa, 0.0)) + 1.0",
     "np.sqrt(np.maximum(2.0 * kmax - kappa, 0.0))"),
    ("node_weight_reversed", "erc.py", "(kappa[eid] - kmin) / (kmax - kmin + eta)",
     "(kmax - kappa[eid]) / (kmax - kmin + eta)"),
    ("node_fallback_counts_isolated", "erc.py",
     "qn = (np.diff(g.rowptr) > 0).astype(np.float64)", "qn = np.ones(g.n)"),
    # projection signs (SplitMix64)
    ("splitmix_shift", "hashing.py", "z = (z ^ (z >> U64(30))) * MUL1",
     "z = (z ^ (z >> U64(29))) * MUL1"),
    ("sign_bit_order", "hashing.py", "bits = (words >> (cols % 64).astype(U64)",
     "bits = (words >> (63 - cols % 64).astype(U64)"),
    # graph, incidence, exact references
    ("incidence_orientation", "graph.py", "v = np.concatenate([np.ones(m), -np.ones(m)])",
     "v = np.concatenate([-np.ones(m), np.ones(m)])"),
    ("edge_id_transposed", "graph.py", "eid = np.searchsorted(keys, lo * g.n + hi)",
     "eid = np.searchsorted(keys, hi * g.n + lo)"),
    ("pinv_resistance_sign", "exact.py", "return Lp[eu, eu] + Lp[ev, ev] - 2.0 * Lp[eu, ev]",
     "return Lp[eu, eu] + Lp[ev, ev] + 2.0 * Lp[eu, ev]"),
    ("self_loop_accepted", "graph.py", "    if np.any(rows == col):\n        raise ValueError(\"self-loop\")",
     "    if False:\n        raise ValueError(\"self-loop\")"),
    ("repeated_entries_accepted", "graph.py", "if np.any(np.diff(key) <= 0):",
     "if np.any(np.diff(key) < 0):"),
    ("base_is_the_seed", "hashing.py", "return U64(splitmix64(seed, 1)[0])", "return U64(seed)"),
    # the column-parallel driver
    ("parallel_ranges_overlap", "parallel.py",
     "chunks = [(bounds[k], bounds[k + 1]) for k in range(procs)]",
     "chunks = [(bounds[k], min(bounds[k + 1] + 1, col_end)) for k in range(procs)]"),
    ("dense_Q_scale", "exact.py", "np.arange(col0, col0 + ncols)) / math.sqrt(K)",
     "np.arange(col0, col0 + ncols)) / K"),
    ("reg_resistance_sign", "exact.py", "return M[eu, eu] + M[ev, ev] - 2.0 * M[eu, ev]",
     "return M[eu, eu] + M[ev, ev] - M[eu, ev]"),
    ("jl_dense_unshifted", "exact.py", "Z = np.linalg.solve(L + delta * np.eye(g.n), Y)",
     "Z = np.linalg.lstsq(L, Y, rcond=None)[0]"),
    # Table 2 metrics
    ("pearson_uncentred", "agreement.py", "    da = a - a.mean()\n    db = b - b.mean()",
     "    da = a\n    db = b"),
    ("sign_zero_merged", "agreement.py",
     "return float(np.mean(np.sign(np.asarray(a, np.float64)) == np.sign(np.asarray(b, np.float64))))",
     "return float(np.mean((np.asarray(a, np.float64) > 0) == (np.asarray(b, np.float64) > 0)))"),
    # subgraphs of the draws
    ("node_subgraph_union", "sampling.py", "ekeep = keep[eu] & keep[ev]", "ekeep = keep[eu] | keep[ev]"),
    ("relabel_from_one", "sampling.py", "new_id[nodes] = np.arange(nodes.size)",
     "new_id[nodes] = np.arange(1, nodes.size + 1)"),
    ("edge_subgraph_one_endpoint", "sampling.py", "    keep[ev[ekeep]] = True\n", ""),
    # compensated dot products
    ("two_prod_low_part_dropped", "accurate.py", "    al = a - ah\n", "    al = 0.0 * a\n"),
    ("two_sum_error_term", "accurate.py", "e = (a - (s - z)) + (b - z)", "e = (a - (s - z)) - (b - z)"),
    # Table 2 metrics
    ("rank_ties_not_averaged", "agreement.py", "ranks[order[i:j + 1]] = 0.5 * (i + j) + 1.0",
     "ranks[order[i:j + 1]] = i + 1.0"),
    ("mae_signed", "agreement.py", "return float(np.mean(np.abs(a - b)))",
     "return float(np.abs(np.mean(a - b)))"),
    # curvature-guided draws
    ("draw_search_boundary", "sampling.py", 'side="right")) - 1', 'side="left")) - 1'),
    ("draw_scale_bits", "sampling.py", "SCALE_BITS = 62", "SCALE_BITS = 61"),
]


def _run_pins(mutant=None):
    with tempfile.TemporaryDirectory(prefix="oracle_mutant_") as tmp:
        dst = os.path.join(tmp, "oracle")
        shutil.copytree(os.path.join(ROOT, "oracle"), dst,
                        ignore=shutil.ignore_patterns("__pycache__"))
        if mutant is not None:
            _, module, old, new = mutant
            path = os.path.join(dst, module)
            with open(path) as f:
                src = f.read()
            assert old in src, f"{module} no longer contains {old!r}"
            with open(path, "w") as f:
                f.write(src.replace(old, new, 1))
        env = dict(os.environ, PYTHONPATH=tmp + os.pathsep + ROOT,
                   PYTHONDONTWRITEBYTECODE="1")
        # the child runs in the copy's directory (first on its path) and must import the
        # copy, not the repository's oracle
        probe = subprocess.run([sys.executable, "-c", "import oracle; print(oracle.__file__)"],
                               cwd=tmp, env=env, capture_output=True, text=True, timeout=120)
        assert probe.stdout.strip().startswith(dst), probe.stdout + probe.stderr
        files = PIN_TESTS if mutant is None else PINS_OF[mutant[1]]
        return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                               "-m", "not gpu", *files],
                              cwd=tmp, env=env, capture_output=True, text=True, timeout=600)


def test_unchanged_copy_passes_the_pins():
    r = _run_pins()
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]


def test_pins_catch_every_planted_mistake():
    # four children at a time; each stops at its first failing pin
    with ThreadPoolExecutor(4) as ex:
        results = list(ex.map(_run_pins, MUTANTS))
    escaped = []
    for m, r in zip(MUTANTS, results):
        if r.returncode != 1:
            tail = r.stdout.strip().splitlines()[-1:] if r.stdout.strip() else [r.stderr[-300:]]
            escaped.append(f"{m[0]}: pytest exit {r.returncode}; {tail}")
    assert not escaped, "\n".join(escaped)
