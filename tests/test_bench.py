"""bench.py's contract: one JSON line with the fields the benchmark driver reads, the
roofline and CPU-baseline objects, the block-width sweep, and a refusal of more than one
GPU.  The GPU cases run bench.main() in this process on the 20,000-node workload."""
import json
import math
import os
import sys

import numpy as np
import pytest

import gen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _main(monkeypatch, *args):
    monkeypatch.setattr(sys, "argv", ["bench.py", *args])
    return bench.main()


def test_refuses_more_than_one_gpu(monkeypatch, capsys):
    assert _main(monkeypatch, "--gpus", "2") == 2
    cap = capsys.readouterr()
    assert cap.out == ""
    assert "one GPU" in cap.err


def test_padded_widths():
    assert [bench.padded(k, "f32") for k in (1, 16, 17, 64, 100, 256)] == [16, 16, 32, 64, 128, 256]
    assert [bench.padded(k, "f64") for k in (1, 8, 9, 128)] == [8, 8, 16, 128]


@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_spmm_byte_models(weighted, dtype):
    g = gen.erdos_renyi(300, 0.03, 7, weighted=weighted)
    kb = 32
    vt = np.float32 if dtype == "f32" else np.float64
    # compulsory bytes: column indices, weights in the working precision, row pointers,
    # the diagonal (one n-vector) and the n x kb blocks p (read) and q (written)
    arrays = [g.col.astype(np.int32), g.rowptr.astype(np.int64), np.zeros(g.n, vt)]
    if weighted:
        arrays.append(np.asarray(g.w).astype(vt))
    block = np.zeros((g.n, kb), dtype=vt)
    expect = sum(a.nbytes for a in arrays) + 2 * block.nbytes
    assert bench.spmm_bytes_per_launch(g, kb, dtype) == expect
    # what the fused kernel streams: no diagonal, plus r for the fused r.q
    assert bench.spmm_fused_bytes_per_launch(g, kb, dtype) == \
        expect - g.n * vt().itemsize + block.nbytes
    # an iteration counts 11 n x kb passes in all (SpMM: p, q; a z, r update reading z, p,
    # r, q and writing z, r; a p update reading r, p and writing p): 9 beyond the SpMM's
    assert bench.iteration_bytes(g, kb, dtype) == expect + 9 * block.nbytes


def test_byte_model_of_the_largest_workload():
    """4 nnz + 4 nnz + 8 (n+1) + 4 n + 2 * 4 * n * 64 on the 2.4M-node workload's shape
    (n = 2.4M, nnz = 124M, weighted, fp32, 64 columns) is 2.2496 GB."""
    class Shape:
        n = 2_400_000
        nnz = 124_000_000
        w = True
    assert bench.spmm_bytes_per_launch(Shape, 64, "f32") == 2_249_600_008


def test_host_cpu_record():
    c = bench.host_cpu()
    assert c["nproc"] >= 1 and 1 <= c["usable"] <= max(c["nproc"], c["usable"]) and c["model"]


def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.gpu
def test_bench_line(monkeypatch, capsys):
    _gpu()
    assert _main(monkeypatch, "--config", "sbm20k", "--steps", "2", "--warmup", "1",
                 "--no-variants") == 0
    lines = capsys.readouterr().out.strip().splitlines()
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline", "cpu_baseline"):
        assert k in d, k
    assert (d["n_gpus"], d["steps"], d["warmup"]) == (1, 2, 1)
    assert len(d["step_ms"]) == 2 and d["ms_per_step_median"] == max(d["step_ms"])
    assert d["higher_is_better"] is True and d["vs_baseline"] is None
    assert d["config"]["workload"] == "sbm20k" and d["dtype"] == "f32"
    g = gen.make_graph("sbm20k")
    assert math.isclose(d["value"], g.m / (d["ms_per_step"] / 1e3), rel_tol=1e-6)
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert 0.0 < r["frac"] < 1.0
    assert math.isclose(r["frac"], r["achieved"] / r["peak"], abs_tol=1e-4)
    # avg_launch_ms is printed to 4 decimals
    assert math.isclose(r["achieved"], r["bytes_per_launch"] / (r["avg_launch_ms"] / 1e3) / 1e9,
                        rel_tol=1e-3 + 0.5e-4 / r["avg_launch_ms"])
    assert r["traffic"] is None  # counters were taken on the 2.4M-node workload only
    il = r["inner_loop"]
    assert il["iterations"] == r["launches_full"] and 0.0 < il["frac"] < 1.0
    gc = r["gather_ceiling"]
    assert gc["gathered_bytes"] == g.nnz * 64 * 4 and gc["ms"] > 0
    c = d["cpu_baseline"]
    assert c["kind"] == "oracle" and c["cores"] >= 1 and c["value"] > 0 and c["sample"]
    assert c["processes"] == c["cores"] and c["nproc"] >= 1 and c["cpu_model"]
    cfg = d["config"]
    assert (cfg["deg_min"], cfg["deg_max"], cfg["components"]) == \
        (g.summary()["deg_min"], g.summary()["deg_max"], gen.component_count(g))
    rc = d["relabelled_copy"]
    assert rc["ms_per_step"] > 0 and rc["iters_max"] > 0
    assert d["subgraph_draw"]["edges"]["draws"] == max(1, g.m // 1000)


@pytest.mark.gpu
def test_block_sweep(monkeypatch, capsys):
    _gpu()
    assert _main(monkeypatch, "--config", "sbm20k", "--block-sweep", "16,32,64") == 0
    lines = capsys.readouterr().out.strip().splitlines()
    assert len(lines) == 1
    d = json.loads(lines[0])
    assert d["table"] == "block_sweep" and d["workload"] == "sbm20k"
    rows = d["rows"]
    assert [r["k_block"] for r in rows] == [16, 32, 64]
    assert [r["blocks"] for r in rows] == [4, 2, 1]  # K = 64
    mem = [r["device_bytes"] for r in rows]
    assert mem[0] < mem[1] < mem[2]
    # the workspace holds the n x b blocks z, r, p, q (fp32) and per-column partials
    n = gen.make_graph("sbm20k").n
    for k in (1, 2):
        assert mem[k] - mem[0] >= 4 * n * (rows[k]["k_block"] - rows[0]["k_block"]) * 4
    assert all(r["ms_per_step"] > 0 and r["iters_max"] > 0 for r in rows)


def test_trace_and_counter_tables(tmp_path, monkeypatch, capsys):
    # rocprofv3's CSV columns; two kernels, one with a short (early-exit) dispatch
    tr = tmp_path / "t_kernel_trace.csv"
    tr.write_text(
        "Kernel_Name,Start_Timestamp,End_Timestamp\n"
        "\"void erc::k_spmm<float, 16, true>(erc::SpmmArgs)\",0,4000000\n"
        "\"void erc::k_spmm<float, 16, true>(erc::SpmmArgs)\",5000000,9000000\n"
        "\"void erc::k_spmm<float, 16, true>(erc::SpmmArgs)\",9000000,9002000\n"
        "\"void erc::k_update<float, 16, false>(erc::UpdArgs)\",9100000,9900000\n")
    ct = tmp_path / "c_counter_collection.csv"
    ct.write_text(
        "Kernel_Name,Counter_Name,Counter_Value,Start_Timestamp,End_Timestamp\n"
        "\"void erc::k_spmm<float, 16, true>(erc::SpmmArgs)\",FETCH_SIZE,10,0,4000000\n"
        "\"void erc::k_spmm<float, 16, true>(erc::SpmmArgs)\",FETCH_SIZE,30,0,4000000\n"
        "\"void erc::k_spmm<float, 16, true>(erc::SpmmArgs)\",FETCH_SIZE,1,0,2000\n")
    assert _main(monkeypatch, "--trace-table", str(tr), "--counter-table", str(ct)) == 0
    out = capsys.readouterr().out
    # 3 dispatches, 8.002 ms in all, 4 ms per full dispatch (2 of them)
    assert "| k_spmm<float, 16, true> | 3 | 8.0 | 2667.3 | 4000.0 | 2 | 90.9% |" in out
    assert "| k_update<float, 16, false> | 1 | 0.8 | 800.0 | 800.0 | 1 | 9.1% |" in out
    # median over the two full dispatches only
    assert "| k_spmm<float, 16, true> | FETCH_SIZE | 3 | 2 | 20.0 |" in out
