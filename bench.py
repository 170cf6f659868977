"""Benchmark of the MUSTAFAR decode hot path on one MI355X.

A step is one decode step of the method on the whole batch (Sec. 3, Algorithm
1), through the dense-window lifecycle: every (batch, kv-head) stream receives
a new token into its 32-token dense window; the window's oldest token leaves it
and is pruned, compressed and appended to the compressed K and V caches
(mustafar_window_step); then sparse decode attention runs over the compressed
caches and the window (mustafar_window_decode_attn). value = batch * steps /
time: decode tokens per second of the whole job.

Also measured (reported in the same JSON line):
  * a clock-settle phase right before the timed steps: attention calls alone
    for a fixed wall time, reported (calls and seconds) -- the GPU's clocks
    take a few dozen calls to settle under this load, so the result must not
    depend on --warmup;
  * per attention call: mean, median, min and max of the HIP-event times over
    the timed steps, their algorithmic HBM GB/s and roofline fraction (the
    format's bytes: 12 B of bitmap + offset per tile, the packed values with
    padding, the window, q and the output, over the mean), and the same over
    the bytes the kernel needs (it derives the tile offsets from the bitmaps);
  * the HBM read ceiling and, for the compression, the read + write ceiling
    at its write share and the ceiling of its own access order (the same bytes
    in the same order without its arithmetic) -- the library's streaming
    helpers;
  * the in-house dense fp16 decode-attention kernel on the same tokens;
  * the bulk prune+compress of the whole prefill cache (K and V): tokens/s =
    batch * context / time, and its algorithmic GB/s;
  * the other decode workloads (Llama-2-7B 4K, Llama-3-8B GQA 16K, GQA 128K
    with 256 append+attend steps), sparse and dense, warm (back-to-back calls)
    and cold (a 1 GiB write between calls evicts the caches, which hold these
    smaller caches whole);
  * the CPU oracle on bounded samples of streams, at one thread and at the
    box's thread share (cpu_baseline).

Inputs are synthetic (paper_2505_22913_amd.synth), generated on the GPU and
resident in HBM before any timed region starts.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "sparse decode-attn tokens/s + HBM GB/s (% roofline); prune+compress tokens/s"
HBM_PEAK_GBS = 8000.0
FLUSH_BYTES = 1 << 30      # written between cold-cache calls (the on-die caches hold 256 MB)
OTHER_WORKLOADS = ("llama2-7b-4k", "llama3-8b-gqa-16k", "gqa-128k-decode")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--settle-s", type=float, default=0.5,
                    help="wall seconds of attention-only calls before the timed steps (reported)")
    ap.add_argument("--workload", default="mha-b16-32k")
    ap.add_argument("--route", choices=("default", "walks", "matrix_cores"), default="default",
                    help="kernel route of grouped-query sparse calls (mustafar_attn_set_route)")
    ap.add_argument("--route-ab", action="store_true",
                    help="only: the sparse attention of --workload under the walks and the matrix-core "
                         "kernel, alternating, three rounds (same process, same box)")
    ap.add_argument("--splits", type=int, default=0, help="split-K segments (0: library default)")
    ap.add_argument("--seed", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-window", action="store_true", help="skip the output-aware window leg")
    ap.add_argument("--no-variants", action="store_true", help="skip the pruner-variant leg")
    ap.add_argument("--no-channel", action="store_true",
                    help="skip the per-channel value-pruning leg")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the other decode workloads (warm and cold)")
    ap.add_argument("--channel-only", action="store_true",
                    help="only the per-channel value-pruning leg (for its kernel trace)")
    ap.add_argument("--attn-only", action="store_true",
                    help="only the sparse attention of --workload, warm calls (for kernel traces)")
    ap.add_argument("--attn-reps", type=int, default=50)
    ap.add_argument("--cpu-sample-streams", type=int, default=128,
                    help="streams the oracle runs on at the box's thread share")
    ap.add_argument("--cpu-sample-streams-1t", type=int, default=8,
                    help="streams the oracle runs on at one thread")
    ap.add_argument("--cpu-threads", type=int, default=0, help="0: min(16, usable cpus)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy three times (scales HBM byte counters)")
    return ap.parse_args()


def copy_calibration() -> None:
    """A plain device-to-device copy of known size: what FETCH_SIZE / WRITE_SIZE read
    for it gives the factor that turns those counters into bytes."""
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_per_copy": n, "copies": 3}), flush=True)


def attn_alg_bytes(w, k_len_total: int, v_len_total: int, n_s: int) -> int:
    """Bytes one sparse attention launch must move (format + window + q + out)."""
    T = w.d // 64
    tiles = w.B * w.Hkv * n_s * T
    meta = 12 * tiles * 2                       # K and V: 8-byte bitmap + 4-byte offset per tile
    vals = 2 * (k_len_total + v_len_total)      # packed fp16 values incl. padding
    window = 2 * 2 * w.B * w.Hkv * w.n_tail * w.d
    qo = 2 * 2 * w.B * w.Hq * w.d
    return meta + vals + window + qo


def attn_offset_bytes(w, n_s: int) -> int:
    """The per-tile offsets inside attn_alg_bytes: the kernels read only the first
    tile's offset of each segment and derive the others from the bitmaps."""
    return 4 * w.B * w.Hkv * n_s * (w.d // 64) * 2


def dense_alg_bytes(w, n_tokens: int) -> int:
    return 2 * 2 * w.B * w.Hkv * n_tokens * w.d + 4 * w.B * w.Hq * w.d


def measured_traffic(kernel: str, workload: str, key: str = "bytes_per_launch"):
    """HBM bytes from the committed rocprofv3 counter summary (FETCH_SIZE + WRITE_SIZE,
    scaled by a plain copy's counts), or None when there is none or the kernel
    source changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}.traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    # the kernel's source and every file it includes, hashed in the listed order
    h = hashlib.sha256()
    for rel in rec.get("sources", [rec.get("source")]):
        h.update(open(os.path.join(ROOT, rel), "rb").read())
    if h.hexdigest()[:16] != rec["source_sha256_prefix"]:
        return None
    return rec.get(key)


def read_ceiling_gbs(n_bytes: int = 8 << 30) -> float:
    """HBM read rate of this GPU: the library's 16-byte streaming-read kernel over an
    n_bytes buffer (far beyond the on-chip caches)."""
    import torch

    import paper_2505_22913_amd as mf
    x = torch.empty(n_bytes, dtype=torch.uint8, device="cuda")
    x.fill_(1)
    sink = mf.mustafar_stream_read(x)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(5):
        mf.mustafar_stream_read(x, sink)
    b.record()
    torch.cuda.synchronize()
    t = a.elapsed_time(b) / 1e3 / 5
    del x
    torch.cuda.empty_cache()
    return n_bytes / t / 1e9


def rw_ceiling_gbs(write_16ths: int, n_bytes: int = 8 << 30) -> float:
    """HBM read + write rate of this GPU at a given write share: the library's
    streaming kernel reads an n_bytes buffer and writes write_16ths/16 of it;
    the rate counts both directions."""
    import torch

    import paper_2505_22913_amd as mf
    x = torch.empty(n_bytes, dtype=torch.uint8, device="cuda")
    x.fill_(1)
    y = torch.empty(n_bytes * write_16ths // 16 + 16, dtype=torch.uint8, device="cuda")
    sink = mf.mustafar_stream_mix(x, y, write_16ths)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(5):
        mf.mustafar_stream_mix(x, y, write_16ths, sink)
    b.record()
    torch.cuda.synchronize()
    t = a.elapsed_time(b) / 1e3 / 5
    del x, y
    torch.cuda.empty_cache()
    return n_bytes * (1 + write_16ths / 16) / t / 1e9


def chunk_order_ceiling_gbs(n_streams: int, n_bytes: int, write_16ths: int) -> float:
    """HBM read + write rate of the bulk compression's access order: the library's
    chunk-order helper over n_bytes in n_streams streams of 16 KiB chunks, the
    streams taking turns chunk by chunk, writing write_16ths/16 of every chunk;
    the rate counts both directions."""
    import torch

    import paper_2505_22913_amd as mf
    x = torch.empty(n_bytes, dtype=torch.uint8, device="cuda")
    x.fill_(1)
    y = torch.empty(n_bytes * write_16ths // 16 + 16, dtype=torch.uint8, device="cuda")
    sink = mf.mustafar_stream_chunks(x, n_streams, y, write_16ths)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(5):
        mf.mustafar_stream_chunks(x, n_streams, y, write_16ths, sink)
    b.record()
    torch.cuda.synchronize()
    t = a.elapsed_time(b) / 1e3 / 5
    del x, y, sink
    torch.cuda.empty_cache()
    return n_bytes * (1 + write_16ths / 16) / t / 1e9


def call_stats(marks) -> dict:
    """Per-call HIP-event times (us) of recorded (start, end) pairs: mean, median, min, max."""
    import numpy as np
    us = np.array([a.elapsed_time(b) * 1e3 for a, b in marks])
    return {"mean": float(us.mean()), "median": float(np.median(us)), "min": float(us.min()),
            "max": float(us.max()), "calls": int(us.size)}


def timed_calls(fn, reps: int, flush=None, warm: int = 5) -> dict:
    """call_stats of `reps` calls of fn; with a flush buffer, it is overwritten before
    each call (outside the timed pair of events), so every call starts cold."""
    import torch
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    if flush is None:
        for _ in range(warm):
            fn()
    marks = []
    for i in range(reps):
        if flush is not None:
            flush.fill_(i & 0xFF)
        a, b = ev(), ev()
        a.record()
        fn()
        b.record()
        marks.append((a, b))
    torch.cuda.synchronize()
    return call_stats(marks)


def usable_cpus() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_baseline(w, K, V, KL, VL, q, sample_all: int, sample_1t: int, threads: int) -> dict:
    """The oracle (untuned, as in the test suite) on samples of the same workload's
    (batch, kv-head) streams: prune+compress of K and V and decode attention
    (decompress + float64 Algorithm 1), each timed as the median of three runs, at
    `threads` threads and at one; times are scaled to all B*Hkv streams."""
    import numpy as np

    import oracle
    BH = w.B * w.Hkv
    G = w.G

    def run(sample: int, thr: int) -> dict:
        sample = max(1, min(sample, BH))
        picks = np.linspace(0, BH - 1, sample).round().astype(int)
        pick = lambda t: np.stack([t[p // w.Hkv, p % w.Hkv].cpu().numpy() for p in picks])  # noqa: E731
        Ks, Vs = pick(K)[:, None], pick(V)[:, None]
        KLs, VLs = pick(KL)[:, None], pick(VL)[:, None]
        qs = np.stack([q[p // w.Hkv, (p % w.Hkv) * G:(p % w.Hkv + 1) * G].cpu().numpy() for p in picks])
        t_pc, t_at = [], []
        for _ in range(3):
            t0 = time.perf_counter()
            ek = oracle.compress(Ks, w.sK, threads=thr)
            ev = oracle.compress(Vs, w.sV, threads=thr)
            t_pc.append(time.perf_counter() - t0)
            t0 = time.perf_counter()
            oracle.sparse_decode_attention(qs, ek, ev, KLs, VLs, threads=thr)
            t_at.append(time.perf_counter() - t0)
        scale = BH / sample
        step_s = float(np.median(t_at)) * scale     # the append of one token per stream is negligible
        pc_s = float(np.median(t_pc)) * scale
        return {"value": w.B / step_s, "unit": "tokens/s", "threads": thr,
                "sample": f"{sample} of {BH} (batch, kv-head) streams, scaled by {scale:.2f}",
                "attn_s_per_step_est": step_s,
                "prune_compress_tokens_per_s": w.B * w.N / pc_s,
                "wall_s": float(np.sum(t_pc) + np.sum(t_at))}

    oracle.build()
    many = run(sample_all, threads)
    one = run(sample_1t, 1)
    return {"value": many["value"], "unit": "tokens/s", "cores": threads, "nproc": os.cpu_count(),
            "usable_cpus": usable_cpus(), "kind": "oracle",
            "sample": f"{many['sample']} at {threads} threads (median of 3 runs); decode attention "
                      "= decompress + float64 Algorithm 1; tokens/s = batch / scaled step time",
            "attn_s_per_step_est": many["attn_s_per_step_est"],
            "prune_compress_tokens_per_s": many["prune_compress_tokens_per_s"],
            "single_thread": one, "wall_s": many["wall_s"] + one["wall_s"]}


def workload_leg(name: str, seed: int, splits: int, flush, reps: int = 20) -> dict:
    """Sparse and dense decode attention of one more workload, warm and cold; for a
    workload with decode steps, also the prefill's bulk prune+compress and the
    append+attend steps through the window lifecycle."""
    import numpy as np
    import torch

    import paper_2505_22913_amd as mf
    from paper_2505_22913_amd import synth
    w = synth.WORKLOADS[name]
    dev = "cuda"
    steps = w.decode_steps
    K, V = synth.make_kv_torch(w.B, w.Hkv, w.N + w.n_tail, w.d, seed=seed, device=dev)
    gq = torch.Generator(device=dev)
    gq.manual_seed(seed)
    q = torch.randn((w.B, w.Hq, w.d), generator=gq, device=dev).half()
    pool_k, pool_v = synth.make_kv_torch(w.B, w.Hkv, 64, w.d, seed=seed + 7, device=dev)
    Kc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, w.N + steps + 1, device=dev)
    Vc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, w.N + steps + 1, device=dev)
    win = mf.DenseWindow(w.B, w.Hkv, w.d, w.n_tail, device=dev)
    ws_c = torch.empty(mf.mustafar_compress_workspace_bytes(w.B, w.Hkv, w.N + w.n_tail),
                       dtype=torch.uint8, device=dev)
    ws_a = torch.empty(mf.mustafar_attn_workspace_bytes(w.B, w.Hq, w.Hkv, w.d, w.N + steps + w.n_tail,
                                                        splits), dtype=torch.uint8, device=dev)
    out = torch.empty((w.B, w.Hq, w.d), dtype=torch.float16, device=dev)
    res = {"batch": w.B, "q_heads": w.Hq, "kv_heads": w.Hkv, "context": w.N, "window": w.n_tail,
           "k_sparsity": w.sK, "v_sparsity": w.sV,
           # the library's routing: the matrix-core kernel from 8 query heads per kv-head
           "kernel": "k_sparse_attn_mfma" if w.G >= 8 else "k_sparse_attn"}
    # bulk prune + compress of the prefill (K and V), median of three
    Kp, Vp = K[:, :, :w.N].contiguous(), V[:, :, :w.N].contiguous()
    pc = []
    for _ in range(3):
        Kc.desc.n_tokens = Vc.desc.n_tokens = 0
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        mf.mustafar_prune_compress(Kc, Kp, ws_c)
        mf.mustafar_prune_compress(Vc, Vp, ws_c)
        b.record()
        torch.cuda.synchronize()
        pc.append(a.elapsed_time(b) / 1e3)
    t_pc = float(np.median(pc))
    res["prune_compress"] = {"ms": t_pc * 1e3, "tokens_per_s": w.B * w.N / t_pc}
    del Kp, Vp
    Kc.desc.n_tokens = Vc.desc.n_tokens = 0
    mf.mustafar_window_prefill(win, Kc, Vc, K, V, [w.N + w.n_tail] * w.B, ws_c)
    torch.cuda.synchronize()
    k_len = int(Kc.stream_len.to(torch.int64).sum().item())
    v_len = int(Vc.stream_len.to(torch.int64).sum().item())
    alg = attn_alg_bytes(w, k_len, v_len, w.N)
    dbytes = dense_alg_bytes(w, w.N + w.n_tail)
    sparse = lambda: mf.mustafar_window_decode_attn(q, Kc, Vc, win, out=out, n_splits=splits,  # noqa: E731
                                                    ws=ws_a)
    dense = lambda: mf.mustafar_dense_decode_attn(q, K, V, out=out, n_splits=splits, ws=ws_a)  # noqa: E731
    for mode, fl in (("warm", None), ("cold", flush)):
        s = timed_calls(sparse, reps, fl)
        dn = timed_calls(dense, reps, fl)
        res[mode] = {"sparse_us": s, "dense_us": dn,
                     "sparse_gb_s": alg / (s["median"] * 1e-6) / 1e9,
                     "sparse_frac": alg / (s["median"] * 1e-6) / 1e9 / HBM_PEAK_GBS,
                     "dense_gb_s": dbytes / (dn["median"] * 1e-6) / 1e9,
                     "speedup_vs_dense": dn["median"] / s["median"],
                     "tokens_per_s": w.B / (s["median"] * 1e-6)}
    res["alg_bytes"] = alg
    res["compressed_vs_dense_kv"] = (alg - 4 * w.B * w.Hq * w.d - 4 * w.B * w.Hkv * w.n_tail * w.d) / \
        (4 * w.B * w.Hkv * w.N * w.d)
    if steps:
        # append + attend steps: the window's oldest token leaves for the caches
        ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
        marks = [(ev(), ev()) for _ in range(steps)]
        a, b = ev(), ev()
        a.record()
        for i in range(steps):
            mf.mustafar_window_step(win, Kc, Vc, pool_k[:, :, i % 64].contiguous(),
                                    pool_v[:, :, i % 64].contiguous())
            marks[i][0].record()
            sparse()
            marks[i][1].record()
        b.record()
        torch.cuda.synchronize()
        tot = a.elapsed_time(b) / 1e3 / steps
        res["decode_steps"] = {"steps": steps, "us_per_step": tot * 1e6,
                               "attention_us": call_stats(marks), "tokens_per_s": w.B / tot,
                               "how": "mustafar_window_step (a new token per stream; the oldest "
                                      "window token is pruned, compressed and appended) + "
                                      "mustafar_window_decode_attn"}
    del K, V, Kc, Vc, win, ws_c, ws_a, out, pool_k, pool_v
    torch.cuda.empty_cache()
    return res


ROUTES = {"default": 0, "walks": 1, "matrix_cores": 2}


def route_ab(args) -> None:
    """The grouped-query kernels side by side: warm sparse attention of --workload
    with its compressed segments on the bit walks, then on the matrix-core
    kernel (each with its own default split count), alternating, three rounds;
    per route the median over rounds of each round's median call time."""
    import numpy as np
    import torch

    import paper_2505_22913_amd as mf
    from paper_2505_22913_amd import synth
    w = synth.WORKLOADS[args.workload]
    dev = "cuda"
    K, V = synth.make_kv_torch(w.B, w.Hkv, w.N + w.n_tail, w.d, seed=args.seed, device=dev)
    gq = torch.Generator(device=dev)
    gq.manual_seed(args.seed)
    q = torch.randn((w.B, w.Hq, w.d), generator=gq, device=dev).half()
    Kc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, w.N, device=dev)
    Vc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, w.N, device=dev)
    win = mf.DenseWindow(w.B, w.Hkv, w.d, w.n_tail, device=dev)
    ws_c = torch.empty(mf.mustafar_compress_workspace_bytes(w.B, w.Hkv, w.N + w.n_tail),
                       dtype=torch.uint8, device=dev)
    mf.mustafar_window_prefill(win, Kc, Vc, K, V, [w.N + w.n_tail] * w.B, ws_c)
    del K, V
    out = torch.empty((w.B, w.Hq, w.d), dtype=torch.float16, device=dev)
    torch.cuda.synchronize()
    k_len = int(Kc.stream_len.to(torch.int64).sum().item())
    v_len = int(Vc.stream_len.to(torch.int64).sum().item())
    alg = attn_alg_bytes(w, k_len, v_len, w.N)
    res = {name: {"call_us": []} for name in ("walks", "matrix_cores")}
    try:
        for _ in range(3):
            for name in res:
                mf.mustafar_attn_set_route(ROUTES[name])
                splits = mf.mustafar_attn_default_splits(w.B, w.Hq, w.Hkv, w.N)
                ws_a = torch.empty(mf.mustafar_attn_workspace_bytes(w.B, w.Hq, w.Hkv, w.d, w.N, splits),
                                   dtype=torch.uint8, device=dev)
                st = timed_calls(lambda: mf.mustafar_window_decode_attn(q, Kc, Vc, win, out=out,
                                                                        n_splits=splits, ws=ws_a), 20)
                res[name]["splits"] = splits
                res[name]["call_us"].append(st["median"])
                del ws_a
    finally:
        mf.mustafar_attn_set_route(ROUTES["default"])
    for name, r in res.items():
        r["call_us_median"] = float(np.median(r["call_us"]))
        r["gb_s"] = alg / (r["call_us_median"] * 1e-6) / 1e9
    print(json.dumps({"route_ab": res, "workload": w.name, "q_heads_per_kv_head": w.G, "alg_bytes": alg,
                      "default": "matrix_cores" if w.G >= 8 else "walks"}), flush=True)


def attn_only(args) -> None:
    """Warm sparse attention calls of --workload alone (for rocprofv3 kernel traces
    and counters of the attention kernels)."""
    import torch

    import paper_2505_22913_amd as mf
    from paper_2505_22913_amd import synth
    w = synth.WORKLOADS[args.workload]
    dev = "cuda"
    K, V = synth.make_kv_torch(w.B, w.Hkv, w.N + w.n_tail, w.d, seed=args.seed, device=dev)
    gq = torch.Generator(device=dev)
    gq.manual_seed(args.seed)
    q = torch.randn((w.B, w.Hq, w.d), generator=gq, device=dev).half()
    Kc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, w.N, device=dev)
    Vc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, w.N, device=dev)
    win = mf.DenseWindow(w.B, w.Hkv, w.d, w.n_tail, device=dev)
    ws_c = torch.empty(mf.mustafar_compress_workspace_bytes(w.B, w.Hkv, w.N + w.n_tail),
                       dtype=torch.uint8, device=dev)
    mf.mustafar_window_prefill(win, Kc, Vc, K, V, [w.N + w.n_tail] * w.B, ws_c)
    ws_a = torch.empty(mf.mustafar_attn_workspace_bytes(w.B, w.Hq, w.Hkv, w.d, w.N, args.splits),
                       dtype=torch.uint8, device=dev)
    out = torch.empty((w.B, w.Hq, w.d), dtype=torch.float16, device=dev)
    torch.cuda.synchronize()
    k_len = int(Kc.stream_len.to(torch.int64).sum().item())
    v_len = int(Vc.stream_len.to(torch.int64).sum().item())
    alg = attn_alg_bytes(w, k_len, v_len, w.N)
    st = timed_calls(lambda: mf.mustafar_window_decode_attn(q, Kc, Vc, win, out=out, n_splits=args.splits,
                                                            ws=ws_a), args.attn_reps)
    print(json.dumps({"workload": w.name, "route": args.route, "attention_us": st, "alg_bytes": alg,
                      "gb_s": alg / (st["mean"] * 1e-6) / 1e9,
                      "frac": alg / (st["mean"] * 1e-6) / 1e9 / HBM_PEAK_GBS}), flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(json.dumps({"error": "one GPU only: every (batch, kv-head) stream is independent, "
                                   "so N GPUs would each run this benchmark on their own share",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2505_22913_amd as mf
    from paper_2505_22913_amd import synth

    torch.cuda.set_device(0)
    if args.route_ab:
        route_ab(args)
        return
    mf.mustafar_attn_set_route(ROUTES[args.route])
    if args.attn_only:
        attn_only(args)
        return
    w = synth.WORKLOADS[args.workload]
    steps, warm = args.steps, args.warmup
    dev = "cuda"
    cap = w.N + warm + steps + 1

    # ---- synthetic inputs, resident in HBM ----
    K, V = synth.make_kv_torch(w.B, w.Hkv, w.N + w.n_tail, w.d, seed=args.seed, device=dev)
    KL = K[:, :, w.N:].contiguous()                    # the dense window after the prefill
    VL = V[:, :, w.N:].contiguous()
    Kp = K[:, :, :w.N].contiguous()
    Vp = V[:, :, :w.N].contiguous()
    gq = torch.Generator(device=dev)
    gq.manual_seed(args.seed)
    q = torch.randn((w.B, w.Hq, w.d), generator=gq, device=dev).half()
    # the new tokens of the decode steps: 64 distinct ones per stream, in turn
    pool_k, pool_v = synth.make_kv_torch(w.B, w.Hkv, 64, w.d, seed=args.seed + 7, device=dev)
    pool_k = [pool_k[:, :, i].contiguous() for i in range(64)]
    pool_v = [pool_v[:, :, i].contiguous() for i in range(64)]
    new_k, new_v = pool_k[0], pool_v[0]
    Kc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, cap, device=dev)
    Vc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, cap, device=dev)
    ws_c = torch.empty(mf.mustafar_compress_workspace_bytes(w.B, w.Hkv, w.N + w.n_tail),
                       dtype=torch.uint8, device=dev)
    ws_a = torch.empty(mf.mustafar_attn_workspace_bytes(w.B, w.Hq, w.Hkv, w.d, cap, args.splits),
                       dtype=torch.uint8, device=dev)
    out = torch.empty((w.B, w.Hq, w.d), dtype=torch.float16, device=dev)
    torch.cuda.synchronize()

    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731

    # ---- per-channel value pruning in groups of 32 tokens: bulk compression of
    # the prefill values (magnitude and output-aware), attention over per-token
    # keys + per-channel values, and the grouped window lifecycle with scores ----
    def channel_leg(v_len_ref):
        torch.cuda.empty_cache()
        Vg = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, cap, device=dev, grouped=True)
        Kg = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, cap, device=dev)
        gtw = torch.Generator(device=dev)
        gtw.manual_seed(args.seed + 2)
        tok_w = (torch.rand((w.B, w.Hkv, w.N), generator=gtw, device=dev) * 0.01).float()

        def timed_v(fn, reps=3):
            ts = []
            for _ in range(reps):
                Vg.desc.n_tokens = 0
                a, b = ev(), ev()
                a.record()
                fn()
                b.record()
                torch.cuda.synchronize()
                ts.append(a.elapsed_time(b) / 1e3)
            return float(np.median(ts))

        vtoks = w.B * w.Hkv * w.N
        t_oa = timed_v(lambda: mf.mustafar_prune_compress_ex(
            Vg, Vp, mode=mf.PRUNE_CHANNEL_OUTPUT_AWARE, weights=tok_w, ws=ws_c))
        t_mag = timed_v(lambda: mf.mustafar_prune_compress(Vg, Vp, ws_c))
        mf.mustafar_prune_compress(Kg, Kp, ws_c)
        torch.cuda.synchronize()
        kg_len = int(Kg.stream_len.to(torch.int64).sum().item())
        vg_len = int(Vg.stream_len.to(torch.int64).sum().item())
        for _ in range(3):
            mf.mustafar_sparse_decode_attn(q, Kg, Vg, KL, VL, out=out, n_splits=args.splits, ws=ws_a)
        a, b = ev(), ev()
        reps = 10
        a.record()
        for _ in range(reps):
            mf.mustafar_sparse_decode_attn(q, Kg, Vg, KL, VL, out=out, n_splits=args.splits, ws=ws_a)
        b.record()
        torch.cuda.synchronize()
        t_ga = a.elapsed_time(b) / 1e3 / reps
        g_bytes = attn_alg_bytes(w, kg_len, vg_len, w.N)
        del Kg, Vg
        torch.cuda.empty_cache()
        # the grouped lifecycle: a 64-slot ring, 32 tokens per stream dense after the prefill
        Kw = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, cap + 64, device=dev)
        Vw = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, cap + 64, device=dev, grouped=True)
        win = mf.DenseWindow(w.B, w.Hkv, w.d, 64, device=dev)
        acc = torch.zeros((w.B, w.Hkv, 64), dtype=torch.float32, device=dev)
        mf.mustafar_window_prefill(win, Kw, Vw, K, V, [w.N + w.n_tail] * w.B, ws_c)
        gsteps = 96   # graduations after 33 and 65 steps: two per stream

        def gstep(marks=None):
            mf.mustafar_window_step_grouped(win, Kw, Vw, new_k, new_v, None, acc)
            if marks is not None:
                marks[0].record()
            mf.mustafar_window_decode_attn_scores(q, Kw, Vw, win, acc, out=out,
                                                  n_splits=args.splits, ws=ws_a)
            if marks is not None:
                marks[1].record()

        torch.cuda.synchronize()
        gmarks = [(ev(), ev()) for _ in range(gsteps)]
        a, b = ev(), ev()
        a.record()
        for i in range(gsteps):
            gstep(gmarks[i])
        b.record()
        torch.cuda.synchronize()
        g_total = a.elapsed_time(b) / 1e3 / gsteps
        g_attn = float(np.mean([m[0].elapsed_time(m[1]) for m in gmarks])) / 1e3
        channel = {
            "cache": f"V, {w.sV:.0%} per channel in groups of 32 (keys per token, {w.sK:.0%})",
            "compress_magnitude_tokens_per_s": vtoks / t_mag,
            "compress_output_aware_tokens_per_s": vtoks / t_oa,
            "attention_us": t_ga * 1e6, "attention_gb_s": g_bytes / t_ga / 1e9,
            "attention_frac": g_bytes / t_ga / 1e9 / HBM_PEAK_GBS, "attention_alg_bytes": g_bytes,
            "values_stored_vs_per_token": None if v_len_ref is None else vg_len / max(1, v_len_ref),
            "lifecycle_us_per_step": g_total * 1e6,
            "lifecycle_attention_scores_us": g_attn * 1e6,
            "lifecycle_window_step_us": (g_total - g_attn) * 1e6,
            "how": "mustafar_window_step_grouped + mustafar_window_decode_attn_scores, "
                   f"64-slot ring, {gsteps} steps, two graduations of 32 tokens per stream"}
        del Kw, Vw, win, acc, tok_w
        torch.cuda.empty_cache()
        return channel


    if args.channel_only:
        print(json.dumps({"channel_pruning": channel_leg(None), "config": {"workload": w.name}}),
              flush=True)
        return

    # ---- bulk prune + compress of the prefill cache (K and V), median of three ----
    pc_ms = []
    for rep in range(3):
        Kc.desc.n_tokens = 0
        Vc.desc.n_tokens = 0
        a, b = ev(), ev()
        a.record()
        mf.mustafar_prune_compress(Kc, Kp, ws_c)
        mf.mustafar_prune_compress(Vc, Vp, ws_c)
        b.record()
        torch.cuda.synchronize()
        pc_ms.append(a.elapsed_time(b))
    t_pc = float(np.median(pc_ms)) / 1e3
    assert mf.compress_status(ws_c) == 0
    k_len0 = int(Kc.stream_len.to(torch.int64).sum().item())
    v_len0 = int(Vc.stream_len.to(torch.int64).sum().item())
    dense_kv = 2 * 2 * w.B * w.Hkv * w.N * w.d
    comp_kv = 12 * w.B * w.Hkv * w.N * (w.d // 64) * 2 + 2 * (k_len0 + v_len0)
    pc_traffic = measured_traffic("k_compress", w.name, "bytes_k_plus_v")

    # ---- the decode state: the prefill's first N tokens compressed, the last
    # n_tail tokens in the dense window (the same caches, compressed again) ----
    Kc.desc.n_tokens = Vc.desc.n_tokens = 0
    win = mf.DenseWindow(w.B, w.Hkv, w.d, w.n_tail, device=dev)
    mf.mustafar_window_prefill(win, Kc, Vc, K, V, [w.N + w.n_tail] * w.B, ws_c)
    attend = lambda: mf.mustafar_window_decode_attn(q, Kc, Vc, win, out=out,  # noqa: E731
                                                    n_splits=args.splits, ws=ws_a)

    # ---- decode steps: a new token into every window, the oldest one pruned,
    # compressed and appended (a1/a2/a7), then attention (a3-a6) ----
    def step(i, marks=None):
        mf.mustafar_window_step(win, Kc, Vc, pool_k[i % 64], pool_v[i % 64])
        if marks is not None:
            marks[0].record()
        attend()
        if marks is not None:
            marks[1].record()

    marks = [(ev(), ev()) for _ in range(steps)]
    t_start, t_end = ev(), ev()
    for i in range(warm):
        step(i)
    torch.cuda.synchronize()
    n_s_start = Kc.n_tokens
    k_len_start = int(Kc.stream_len.to(torch.int64).sum().item())
    v_len_start = int(Vc.stream_len.to(torch.int64).sum().item())

    # ---- clock settle, right before the timed steps: attention calls alone for
    # a fixed wall time (reported; they change no cache) ----
    t0 = time.perf_counter()
    settle_calls = 0
    while time.perf_counter() - t0 < args.settle_s:
        for _ in range(10):
            attend()
        settle_calls += 10
        torch.cuda.synchronize()
    settle_s = time.perf_counter() - t0

    wall0 = time.perf_counter()
    t_start.record()
    for i in range(steps):
        step(warm + i, marks[i])
    t_end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_s = t_start.elapsed_time(t_end) / 1e3
    attn = call_stats(marks)

    # ---- dense baseline over the same tokens (compressed prefix + window), right
    # after the timed steps, at the same settled clocks ----
    ws_d = torch.empty(mf.mustafar_attn_workspace_bytes(w.B, w.Hq, w.Hkv, w.d, w.N + w.n_tail,
                                                        args.splits), dtype=torch.uint8, device=dev)
    dense_st = timed_calls(lambda: mf.mustafar_dense_decode_attn(q, K, V, out=out, n_splits=args.splits,
                                                                 ws=ws_d), 20)
    t_dense = dense_st["mean"] * 1e-6
    dense_bytes = dense_alg_bytes(w, w.N + w.n_tail)
    del ws_d
    attn_s = attn["mean"] * 1e-6
    n_s_end = Kc.n_tokens

    # algorithmic bytes of the attention launches, averaged over the timed steps
    # (the compressed part grows by one token per step)
    k_len1 = int(Kc.stream_len.to(torch.int64).sum().item())
    v_len1 = int(Vc.stream_len.to(torch.int64).sum().item())
    per_tok_k = (k_len1 - k_len_start) / max(1, n_s_end - n_s_start)
    per_tok_v = (v_len1 - v_len_start) / max(1, n_s_end - n_s_start)
    alg = [attn_alg_bytes(w, int(k_len_start + per_tok_k * (n_s - n_s_start)),
                          int(v_len_start + per_tok_v * (n_s - n_s_start)), n_s)
           for n_s in range(n_s_start + 1, n_s_end + 1)]
    alg_bytes = float(np.mean(alg))
    attn_gbs = alg_bytes / attn_s / 1e9
    read_bytes = alg_bytes - float(np.mean([attn_offset_bytes(w, n_s)
                                            for n_s in range(n_s_start + 1, n_s_end + 1)]))
    del Kc, Vc, win
    torch.cuda.empty_cache()

    # ---- the same steps with output-aware keys: the leaving key is pruned with
    # the weights its window slot gathered from the queries of its 32 steps ----
    window = None
    if not args.no_window:
        Kw = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, cap, device=dev)
        Vw = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, cap, device=dev)
        win = mf.DenseWindow(w.B, w.Hkv, w.d, w.n_tail, device=dev)
        kacc = torch.zeros((w.B, w.Hkv, w.n_tail, w.d), dtype=torch.float32, device=dev)
        mf.mustafar_window_prefill(win, Kw, Vw, K, V, [w.N + w.n_tail] * w.B, ws_c)

        def kstep(i, marks=None):
            mf.mustafar_window_step_weighted(win, Kw, Vw, pool_k[i % 64], pool_v[i % 64], kacc)
            mf.mustafar_window_decode_attn(q, Kw, Vw, win, out=out, n_splits=args.splits, ws=ws_a)
            if marks is not None:
                marks[0].record()
            mf.mustafar_window_key_weights(q, win, kacc)
            if marks is not None:
                marks[1].record()

        kmarks = [(ev(), ev()) for _ in range(steps)]
        a, b = ev(), ev()
        for i in range(warm):
            kstep(i)
        torch.cuda.synchronize()
        a.record()
        for i in range(steps):
            kstep(warm + i, kmarks[i])
        b.record()
        torch.cuda.synchronize()
        k_total = a.elapsed_time(b) / 1e3 / steps
        k_kw = float(np.mean([m[0].elapsed_time(m[1]) for m in kmarks])) / 1e3
        window = {
            "us_per_step": k_total * 1e6, "key_weights_us": k_kw * 1e6,
            "tokens_per_s": w.B / k_total,
            "how": "mustafar_window_step_weighted + mustafar_window_decode_attn + "
                   "mustafar_window_key_weights (|q| of the step into the newest 32 slots)"}
        del Kw, Vw, win, kacc
        torch.cuda.empty_cache()

    # ---- pruner variants on the same prefill cache (K: N tokens per stream) ----
    variants = None
    if not args.no_variants:
        torch.cuda.empty_cache()
        Kv = mf.CompressedCache(w.B, w.Hkv, w.d, 0.5, w.N, device=dev)

        def timed(fn, reps=3):
            ts = []
            for _ in range(reps):
                Kv.desc.n_tokens = 0
                a, b = ev(), ev()
                a.record()
                fn()
                b.record()
                torch.cuda.synchronize()
                ts.append(a.elapsed_time(b) / 1e3)
            return float(np.median(ts))

        toks = w.B * w.Hkv * w.N
        t24 = timed(lambda: mf.mustafar_prune_compress_ex(Kv, Kp, mode=mf.PRUNE_2_4, ws=ws_c))
        hk = [Kv.n_keep if h % 2 == 0 else Kv.n_keep // 2 for h in range(w.Hkv)]
        thead = timed(lambda: mf.mustafar_prune_compress_ex(Kv, Kp, head_keep=hk, ws=ws_c))
        # output-aware keys: the lookahead weights of the queries at every position
        gqh = torch.Generator(device=dev)
        gqh.manual_seed(args.seed + 1)
        qhist = torch.randn((w.B, w.Hq, w.N, w.d), generator=gqh, device=dev).half()
        wts = torch.empty((w.B, w.Hkv, w.N, w.d), dtype=torch.float32, device=dev)
        a, b = ev(), ev()
        a.record()
        mf.mustafar_query_lookahead(qhist, w.Hkv, 32, out=wts)
        b.record()
        torch.cuda.synchronize()
        t_look = a.elapsed_time(b) / 1e3
        toa = timed(lambda: mf.mustafar_prune_compress_ex(Kv, Kp, mode=mf.PRUNE_OUTPUT_AWARE,
                                                          weights=wts, ws=ws_c))
        variants = {"cache": "K, 50%", "tokens": toks,
                    "two_four_tokens_per_s": toks / t24,
                    "per_head_tokens_per_s": toks / thead,
                    "output_aware_tokens_per_s": toks / toa,
                    "query_lookahead_ms": t_look * 1e3,
                    "magnitude_tokens_per_s_for_reference": 2 * toks / t_pc,
                    "rates": "token vectors (one kv-head of one token) per second"}
        del Kv, qhist, wts
        torch.cuda.empty_cache()

    channel = None
    if not args.no_channel:
        channel = channel_leg(v_len0)

    workloads = None
    if not args.no_workloads:
        flush = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)
        workloads = {name: workload_leg(name, args.seed, args.splits, flush) for name in OTHER_WORKLOADS}
        del flush
        torch.cuda.empty_cache()

    ceiling = read_ceiling_gbs()
    pc_w16 = max(1, min(16, round(16 * comp_kv / dense_kv)))  # the compression's write share
    rw_ceiling = rw_ceiling_gbs(pc_w16)
    cache_bytes = w.B * w.Hkv * w.N * w.d * 2
    order_ceiling = (chunk_order_ceiling_gbs(w.B * w.Hkv, cache_bytes, pc_w16)
                     if cache_bytes % (w.B * w.Hkv * mf.STREAM_CHUNK_BYTES) == 0 else None)

    result = {
        "metric": METRIC,
        "value": w.B * steps / total_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warm,
        "ms_per_step": total_s / steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic (seeded; K with 4 outlier channels x10 per head, V and q N(0,1))",
        "config": {"workload": w.name, "batch": w.B, "q_heads": w.Hq, "kv_heads": w.Hkv,
                   "context": w.N, "head_dim": w.d, "window": w.n_tail, "k_sparsity": w.sK,
                   "v_sparsity": w.sV, "splits": args.splits or
                   mf.mustafar_attn_default_splits(w.B, w.Hq, w.Hkv, n_s_end)},
        "step": "mustafar_window_step (new token into each 32-token window; the oldest is pruned, "
                "compressed and appended) + mustafar_window_decode_attn",
        "settle": {"calls": settle_calls, "s": settle_s,
                   "how": "attention calls alone for a fixed wall time right before the timed "
                          "steps, after the warmup steps (the GPU clocks settle under load; the "
                          "dense baseline runs right after the timed steps)"},
        "attention": {"us": attn["mean"], "us_median": attn["median"], "us_min": attn["min"],
                      "us_max": attn["max"], "tokens_per_s": w.B / attn_s,
                      "kv_tokens_per_s": w.B * w.Hkv * (n_s_end + w.n_tail) / attn_s,
                      "alg_bytes": alg_bytes, "gb_s": attn_gbs,
                      "how": "HIP events around mustafar_window_decode_attn on its stream "
                             "(k_sparse_attn + the split-K merge), every timed step"},
        "roofline": {"bound": "hbm", "achieved": attn_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": attn_gbs / HBM_PEAK_GBS,
                     "kernel": "k_sparse_attn",
                     "how": "algorithmic bytes of one launch / mean time of the timed attention "
                            "calls (k_sparse_attn and its split-K merge, about 0.6% of it)",
                     "traffic": measured_traffic("k_sparse_attn", w.name),
                     "needed_bytes": read_bytes,
                     "frac_of_needed_bytes": read_bytes / attn_s / 1e9 / HBM_PEAK_GBS,
                     "needed_how": "algorithmic bytes less the per-tile offsets, which the "
                                   "kernel derives from the bitmaps (one offset per segment)"},
        "read_ceiling": {"gb_s": ceiling, "attn_frac": attn_gbs / ceiling,
                         "how": "mustafar_stream_read (16-byte loads) over an 8 GiB buffer"},
        "dense_baseline": {"us": dense_st["mean"], "us_median": dense_st["median"],
                           "us_min": dense_st["min"], "us_max": dense_st["max"],
                           "tokens_per_s": w.B / t_dense, "gb_s": dense_bytes / t_dense / 1e9},
        "speedup_vs_dense": t_dense / attn_s,
        "prune_compress": {"ms": t_pc * 1e3, "tokens_per_s": w.B * w.N / t_pc,
                           "token_vectors_per_s": 2 * w.B * w.Hkv * w.N / t_pc,
                           "alg_bytes": dense_kv + comp_kv,
                           "gb_s": (dense_kv + comp_kv) / t_pc / 1e9,
                           "frac": (dense_kv + comp_kv) / t_pc / 1e9 / HBM_PEAK_GBS,
                           "traffic": pc_traffic,
                           "order_ceiling": None if order_ceiling is None else {
                               "gb_s": order_ceiling, "write_16ths": pc_w16,
                               "frac_of_ceiling": (dense_kv + comp_kv) / t_pc / 1e9 / order_ceiling,
                               "how": "mustafar_stream_chunks over one cache's bytes (batch x kv-heads "
                                      "streams of 16 KiB chunks, the streams taking turns chunk by "
                                      "chunk): the compression's chunk size, write share and order "
                                      "without its arithmetic; rate of both directions"},
                           "rw_ceiling": {"gb_s": rw_ceiling, "write_16ths": pc_w16,
                                          "frac_of_ceiling": (dense_kv + comp_kv) / t_pc / 1e9 / rw_ceiling,
                                          "how": "mustafar_stream_mix over an 8 GiB buffer: every 16-byte "
                                                 "word read, write_16ths of each 16 written (the "
                                                 "compression's write share); rate of both directions"},
                           "how": "K and V of every kv-head: tokens_per_s = batch x context / time; "
                                  "token_vectors_per_s counts each (kv-head, K or V) vector"},
        "append_us_per_step": (total_s / steps - attn_s) * 1e6,
        "output_aware_keys": window,
        "prune_variants": variants,
        "channel_pruning": channel,
        "workloads": workloads,
        "compression_ratio": comp_kv / dense_kv,
        "paper_reference": {
            "hardware": "NVIDIA RTX 6000 Ada (Sec. 4.3), against cuBLAS dense batched MV",
            "workload": "Llama-2-7B MHA, 2048 input + 1024 generated tokens",
            "speedup_vs_dense_k50_v50": 1 / 0.8107, "speedup_vs_dense_k70_v70": 1 / 0.6187,
            "compression_ratio_k50_v50": 0.65, "compression_ratio_k70_v70": 0.45,
            "note": "context only: other hardware, other dense baseline, no absolute throughput given"},
        "wall_s_timed": wall,
    }
    if not args.no_cpu_baseline:
        threads = args.cpu_threads or min(16, usable_cpus())
        result["cpu_baseline"] = cpu_baseline(w, K[:, :, :w.N], V[:, :, :w.N], KL, VL, q,
                                              args.cpu_sample_streams, args.cpu_sample_streams_1t,
                                              threads)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
