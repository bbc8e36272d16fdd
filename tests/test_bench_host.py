"""Host-side bookkeeping of bench.py, on the CPU: the algorithmic bytes and
FLOPs the roofline divides by (checked against a brute-force count of the
visible keys), the HBM-traffic file built from rocprofv3 counter CSVs (on
synthetic CSVs with known values), the rows of each fused LM-head pass, and
the single-GPU guard."""
import json
import os
import subprocess
import sys
import types

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def brute_visible_keys(ctx_len, tree_parent, n_nodes):
    """Keys each query row sees: the whole context plus the node's own path to
    the root (itself included), found by walking the parent pointers."""
    total = 0
    for b in range(len(n_nodes)):
        for i in range(int(n_nodes[b])):
            anc, x = 0, i
            while x >= 0:
                anc += 1
                x = int(tree_parent[b, x])
            total += int(ctx_len[b]) + anc
    return total


def test_attn_work_matches_a_brute_force_count():
    rng = np.random.default_rng(4)
    B, N = 5, 9
    cfg = types.SimpleNamespace(head_dim=8, hq=6, hkv=2)
    n = np.array([1, 9, 4, 0, 6], np.int32)
    L = rng.integers(0, 50, size=B).astype(np.int32)
    tp = np.full((B, N), -1, np.int32)
    td = np.full((B, N), -1, np.int32)
    for b in range(B):
        if n[b]:
            td[b, 0] = 0
        for c in range(1, n[b]):
            tp[b, c] = rng.integers(0, c)
            td[b, c] = td[b, tp[b, c]] + 1
    nbytes, flops = bench.attn_work(cfg, L, n, td)
    # K and V of every context and tree position once, Q in and O out once, bf16
    want_bytes = sum(int(L[b] + n[b]) * cfg.hkv * cfg.head_dim * 2 * 2 + int(n[b]) * cfg.hq * cfg.head_dim * 2 * 2
                     for b in range(B))
    assert nbytes == want_bytes
    # q.k and p.v: 2 + 2 FLOPs per (query head, head dim, visible key)
    assert flops == 4 * cfg.head_dim * cfg.hq * brute_visible_keys(L, tp, n)


def write_csv(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w") as f:
        f.write("Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n")
        for i, (name, v) in enumerate(rows):
            f.write(f'{i},"{name}",X,{v}\n')


def test_counter_file_scales_by_the_copy_calibration(tmp_path, monkeypatch):
    # a 1 GiB copy reads as 2 GiB of FETCH_SIZE (factor 0.5) and exactly 1 GiB
    # of WRITE_SIZE (factor 1); the last five launches of each kernel count
    gib_kib = (1 << 30) / 1024
    d = tmp_path / "run"
    for c, reads in (("FETCH_SIZE", 2 * gib_kib), ("WRITE_SIZE", gib_kib)):
        write_csv(str(d / f"pmc_copy_{c}" / "run_counter_collection.csv"),
                  [("__amd_rocclr_copyBuffer", 10.0)] + [("__amd_rocclr_copyBuffer", reads)] * 5)
    plan, main, comb = bench.ATTN_KERNELS
    fetch = [(plan, 1.0), (main, 999.0)] + [(plan, 2.0), (main, 400.0), (comb, 8.0)] * 5  # KiB per dispatch
    write = [(plan, 0.5), (main, 10.0), (comb, 4.0)] * 5
    write_csv(str(d / "pmc_FETCH_SIZE" / "run_counter_collection.csv"),
              [(f"void (anonymous namespace)::{k}(args)", v) for k, v in fetch])
    write_csv(str(d / "pmc_WRITE_SIZE" / "run_counter_collection.csv"),
              [(f"void (anonymous namespace)::{k}(args)", v) for k, v in write])
    (d / "pmc_FETCH_SIZE.log").write_text("# setup\n" + json.dumps({"roofline": {"algorithmic_bytes": 200000.0}}) + "\n")
    out = tmp_path / "counters.json"
    monkeypatch.setattr(bench, "counters_path", lambda name: str(out))
    bench.write_counter_file(str(d), "tiny")
    res = json.load(open(out))
    assert abs(res["calibration"]["FETCH_SIZE"]["factor"] - 0.5) < 1e-12
    assert abs(res["calibration"]["WRITE_SIZE"]["factor"] - 1.0) < 1e-12
    want_fetch = (2.0 + 400.0 + 8.0) * 1024 * 0.5
    want_write = (0.5 + 10.0 + 4.0) * 1024 * 1.0
    assert abs(res["fetch_bytes_per_launch"] - want_fetch) < 1e-6
    assert abs(res["write_bytes_per_launch"] - want_write) < 1e-6
    assert abs(res["traffic_over_algorithmic"] - (want_fetch + want_write) / 200000.0) < 1e-12
    assert res["source_sha256"] == bench.source_sha(bench.ATTN_SRC)


def test_counter_traffic_ignores_a_stale_kernel(tmp_path, monkeypatch):
    out = tmp_path / "c.json"
    monkeypatch.setattr(bench, "counters_path", lambda name: str(out))
    out.write_text(json.dumps({"source_sha256": "0" * 64, "hbm_bytes_per_launch": 5.0}))
    assert bench.counter_traffic("tiny") is None
    out.write_text(json.dumps({"source_sha256": bench.source_sha(bench.ATTN_SRC), "hbm_bytes_per_launch": 5.0}))
    assert bench.counter_traffic("tiny") == 5.0


def test_head_passes_per_level_then_one_finishing_pass():
    # a 200-node chain walked 4 steps deep under Dmax = 130: the subtrees of
    # the current nodes hold 131, 130, 129 nodes (one row per pass), then 128,
    # which one finishing pass covers; a second sequence stops after 1 step
    N, Dmax = 200, 130
    tp = np.stack([np.arange(-1, N - 1), np.arange(-1, N - 1)]).astype(np.int32)
    tree = {"tree_parent": tp, "n_nodes": np.array([N, 3], np.int32)}
    out_nodes = np.full((2, Dmax + 1), -1, np.int32)
    out_nodes[0, :6] = np.arange(1, 7)
    emitted = np.array([7, 1])
    # level 0: both walkers at the root; the first's subtree alone is 131
    assert bench.head_passes(tree, out_nodes, emitted, Dmax) == [2, 1, 1, 128]
    assert bench.FINISH_ROWS == 128


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
