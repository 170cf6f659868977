"""bench.py's JSON line: the fields the benchmark contract fixes, and the byte
accounting its roofline rests on.

* CPU: more than one GPU is refused with exit status 2 and a JSON message; the
  algorithmic bytes of a sparse launch equal an independent count over a
  compressed cache built by the oracle (bitmap + offset per tile, padded values,
  window, q and output), and the bytes the kernels need leave out exactly the
  per-tile offsets.
* GPU: one short run on the small workload prints one JSON line whose contract
  fields are present, typed and consistent (value from steps and time, frac =
  achieved / peak, the oracle baseline on the host).
"""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import oracle  # noqa: E402
from paper_2505_22913_amd import synth  # noqa: E402


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_is_refused(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == n and "one GPU" in msg["error"]


def test_attention_bytes_match_an_independent_count():
    w = synth.Workload("count", B=2, Hq=8, Hkv=4, N=300, d=128, sK=0.5, sV=0.7, n_tail=32)
    K, V = synth.make_kv(w.B, w.Hkv, w.N, w.d, seed=3)
    ck, cv = oracle.compress(K, w.sK), oracle.compress(V, w.sV)
    k_len = int(np.asarray(ck["stream_len"], dtype=np.int64).sum())
    v_len = int(np.asarray(cv["stream_len"], dtype=np.int64).sum())
    # independent count: per tile an 8-byte bitmap and a 4-byte offset, every
    # tile's kept values padded to a multiple of 8, two bytes each
    tiles = 0
    values = 0
    for c in (ck, cv):
        bm = np.asarray(c["bitmaps"]).reshape(w.B, w.Hkv, -1)[:, :, :w.N * (w.d // 64)]
        counts = np.array([bin(int(b)).count("1") for b in bm.reshape(-1)])
        tiles += bm.size
        values += int(((counts + 7) // 8 * 8).sum())
    assert values == k_len + v_len
    want = 12 * tiles + 2 * values + 2 * 2 * w.B * w.Hkv * w.n_tail * w.d + 2 * 2 * w.B * w.Hq * w.d
    assert bench.attn_alg_bytes(w, k_len, v_len, w.N) == want
    assert bench.attn_offset_bytes(w, w.N) == 4 * tiles
    assert bench.dense_alg_bytes(w, w.N) == 2 * 2 * w.B * w.Hkv * w.N * w.d + 4 * w.B * w.Hq * w.d


@pytest.mark.gpu
def test_bench_line_on_the_small_workload():
    cmd = [sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "tiny-mha-1k",
           "--steps", "3", "--warmup", "1", "--settle-s", "0.05", "--no-window", "--no-variants",
           "--no-channel", "--no-workloads"]
    print("bench contract:", " ".join(cmd[2:]), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    for key, typ in (("metric", str), ("value", float), ("unit", str), ("n_gpus", int), ("steps", int),
                     ("warmup", int), ("ms_per_step", float), ("higher_is_better", bool),
                     ("scaling", str), ("dtype", str), ("data", str), ("config", dict)):
        assert isinstance(d[key], typ), key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["higher_is_better"] is True and d["scaling"] in ("weak", "strong")
    assert d["vs_baseline"] is None
    assert d["config"]["workload"] == "tiny-mha-1k"
    # value = batch x steps / time of the timed steps
    assert d["value"] == pytest.approx(d["config"]["batch"] * d["steps"] / (d["ms_per_step"] * 1e-3 * d["steps"]),
                                       rel=1e-6)
    rf = d["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000
    assert rf["achieved"] > 0 and rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"], rel=1e-9)
    assert rf["traffic"] is None or rf["traffic"] > 0
    assert 0 < rf["needed_bytes"] < d["attention"]["alg_bytes"]
    assert rf["achieved"] == pytest.approx(d["attention"]["alg_bytes"] / d["attention"]["us"] / 1e3, rel=1e-6)
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["unit"] == d["unit"]
    assert isinstance(cb["cores"], int) and cb["cores"] >= 1 and isinstance(cb["sample"], str)
