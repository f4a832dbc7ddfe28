"""Host-side logic of bench.py: the one-GPU guard, counter parsing and the
rule that a recorded traffic figure counts only for unchanged kernel sources."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import numpy as np

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr


def _write_csv(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w") as f:
        f.write('"Dispatch_Id","Kernel_Name","Counter_Name","Counter_Value"\n')
        for r in rows:
            f.write(",".join(f'"{x}"' for x in r) + "\n")


def test_pmc_mean_sums_rows_of_a_dispatch(tmp_path):
    d = str(tmp_path / "f")
    _write_csv(d, [(1, "void segpa::decode_attn_kernel<128>(x)", "FETCH_SIZE", 10),
                   (1, "void segpa::decode_attn_kernel<128>(x)", "FETCH_SIZE", 5),
                   (2, "void segpa::decode_attn_kernel<128>(x)", "FETCH_SIZE", 25),
                   (3, "other_kernel", "FETCH_SIZE", 1000),
                   (4, "void segpa::decode_attn_kernel<128>(x)", "WRITE_SIZE", 7)])
    mean, n = bench.pmc_mean_kib(d, "FETCH_SIZE", "decode_attn_kernel")
    assert (mean, n) == (20.0, 2)
    with pytest.raises(RuntimeError):
        bench.pmc_mean_kib(d, "FETCH_SIZE", "prefill_kernel")


def test_traffic_entry_and_source_hash(tmp_path, monkeypatch):
    kib = 1024
    _write_csv(str(tmp_path / "cf"), [(1, "__amd_rocclr_copyBuffer", "FETCH_SIZE", (1 << 30) / 2 / kib)])
    _write_csv(str(tmp_path / "cw"), [(1, "__amd_rocclr_copyBuffer", "WRITE_SIZE", (1 << 30) / kib)])
    _write_csv(str(tmp_path / "kf"), [(1, "decode_attn_kernel<128>", "FETCH_SIZE", 1000)])
    _write_csv(str(tmp_path / "kw"), [(1, "decode_attn_kernel<128>", "WRITE_SIZE", 10)])
    out = str(tmp_path / "traffic.json")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", out)

    class A:
        kernel = "decode_attn"
        workload = 1
        fetch, write = str(tmp_path / "kf"), str(tmp_path / "kw")
        calib_fetch, calib_write = str(tmp_path / "cf"), str(tmp_path / "cw")
    bench.write_traffic_entry(A)
    d = json.load(open(out))
    e = d["kernels"]["decode_attn/tiny"]
    assert d["calibration"]["fetch_scale"] == pytest.approx(2.0)
    assert e["hbm_bytes_per_launch"] == 2 * 1000 * kib + 10 * kib
    assert bench.recorded_traffic("decode_attn", "tiny") == e["hbm_bytes_per_launch"]
    assert bench.recorded_traffic("decode_attn", "llama3_8b_decode") is None
    # a changed kernel source voids the figure
    e["sources_sha256"] = "0" * 64
    json.dump(d, open(out, "w"))
    assert bench.recorded_traffic("decode_attn", "tiny") is None


def test_code_text_ignores_comments_only():
    a = "int x = 1;  // one\n/* block\n comment */ int y = 2;\n"
    b = "int x = 1;\n// another note\nint y = 2;"
    c = "int x = 1;\nint y = 3;"
    assert bench._code_text(a) == bench._code_text(b)
    assert bench._code_text(a) != bench._code_text(c)


def test_cpu_baseline_pool_reports_what_it_used():
    from paper_2606_06256_amd import inputs as I
    wl = I.config(1)
    r, first = bench.cpu_baseline(1, wl, seconds=0.5, max_procs=2)
    assert r["kind"] == "oracle" and r["unit"] == "tokens/s"
    assert r["cores"] == 2 and r["value"] > 0
    assert "2 single-threaded" in r["sample"]
    # every sampled unit's first result comes back for the parity entry
    assert sorted(first) == list(range(wl.num_units))
    sel, Oo, LSE = first[0]
    assert Oo.shape == (1, wl.G, wl.D) and LSE.shape == (1, wl.G)


def test_parity_of_sample_counts_what_differs():
    """The bench's parity entry: zero against the oracle's own results, then
    one changed page list and one changed output element are seen."""
    from paper_2606_06256_amd import inputs as I
    wl = I.config(1)
    _, first = bench.cpu_baseline(1, wl, seconds=0.2, max_procs=2)
    G = wl.G
    out = np.zeros((wl.total_q, wl.Hq, wl.D), np.float32)
    lse = np.zeros((wl.total_q, wl.Hq), np.float32)
    lists = []
    for u in range(wl.num_units):
        sel, Oo, LSE = first[u]
        r, g = divmod(u, wl.Hkv)
        q0, q1 = int(wl.q_indptr[r]), int(wl.q_indptr[r + 1])
        out[q0:q1, g * G:(g + 1) * G] = Oo
        lse[q0:q1, g * G:(g + 1) * G] = LSE
        lists.append(sel)
    ind = np.concatenate([[0], np.cumsum([len(x) for x in lists])])
    pages = np.concatenate(lists)
    p = bench.parity_of_sample(wl, first, ind, pages, out, lse)
    assert p["units"] == wl.num_units and p["selection_mismatches"] == 0
    assert p["o_max_abs"] < 1e-6 and p["lse_max_abs"] < 1e-5
    pages2 = pages.copy()
    pages2[int(ind[1])] += 1                  # unit 1's first page
    out2 = out.copy()
    out2[0, 0, 3] += 0.5
    p = bench.parity_of_sample(wl, first, ind, pages2, out2, lse)
    assert p["selection_mismatches"] == 1
    assert abs(p["o_max_abs"] - 0.5) < 1e-6
