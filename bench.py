"""Benchmark of the MUSTAFAR decode hot path on one MI355X.

A step is one decode step of the method on the whole batch (Sec. 3): the token
leaving the dense local window of every (batch, kv-head) is pruned, compressed
and appended to the compressed K and V caches, then sparse decode attention
runs over compressed caches + the 32-token dense window (Algorithm 1).
value = batch * steps / time: decode tokens per second of the whole job.

Also measured (reported in the same JSON line):
  * the bulk prune+compress of the whole prefill cache (K and V),
  * the attention call alone: time, algorithmic HBM GB/s and roofline fraction
    (bytes the format makes the kernel read: 12 B of bitmap+offset per tile,
    the packed values with padding, the window, q and the output),
  * the in-house dense fp16 decode-attention kernel on the same tokens,
  * the CPU oracle on a bounded sample of streams (cpu_baseline).

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


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    # Long enough for the GPU clocks to settle under this load (the first few
    # dozen calls after an idle period run slower); no idle gap follows it.
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="mha-b16-32k")
    ap.add_argument("--splits", type=int, default=0, help="split-K segments (0: library default)")
    ap.add_argument("--seed", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-window", action="store_true", help="skip the dense-window lifecycle leg")
    ap.add_argument("--no-variants", action="store_true", help="skip the pruner-variant leg")
    ap.add_argument("--no-channel", action="store_true",
                    help="skip the per-channel value-pruning leg")
    ap.add_argument("--channel-only", action="store_true",
                    help="only the per-channel value-pruning leg (for its kernel trace)")
    ap.add_argument("--cpu-sample-streams", type=int, default=256)
    ap.add_argument("--cpu-threads", type=int, default=0, help="0: min(16, cpu count)")
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


def cpu_baseline(w, K, V, KL, VL, q, sample: int, threads: int) -> dict:
    """Oracle (untuned, as in the test suite) on `sample` (b, h) streams of the
    same workload; the decode-step time is scaled to all B*Hkv streams."""
    import numpy as np

    import oracle
    BH = w.B * w.Hkv
    sample = max(1, min(sample, BH))
    picks = np.linspace(0, BH - 1, sample).round().astype(int)
    Ks = np.stack([K[p // w.Hkv, p % w.Hkv].cpu().numpy() for p in picks])[:, None]
    Vs = np.stack([V[p // w.Hkv, p % w.Hkv].cpu().numpy() for p in picks])[:, None]
    KLs = np.stack([KL[p // w.Hkv, p % w.Hkv].cpu().numpy() for p in picks])[:, None]
    VLs = np.stack([VL[p // w.Hkv, p % w.Hkv].cpu().numpy() for p in picks])[:, None]
    G = w.G
    qs = np.stack([q[p // w.Hkv, (p % w.Hkv) * G:(p % w.Hkv + 1) * G].cpu().numpy()
                   for p in picks])
    Ks = Ks.reshape(sample, 1, w.N, w.d)
    Vs = Vs.reshape(sample, 1, w.N, w.d)
    oracle.build()
    t0 = time.perf_counter()
    ek = oracle.compress(Ks, w.sK, threads=threads)
    ev = oracle.compress(Vs, w.sV, threads=threads)
    t_pc = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.sparse_decode_attention(qs, ek, ev, KLs.reshape(sample, 1, w.n_tail, w.d),
                                   VLs.reshape(sample, 1, w.n_tail, w.d), threads=threads)
    t_attn = time.perf_counter() - t0
    scale = BH / sample
    step_s = t_attn * scale            # the append of one token per stream is negligible
    return {"value": w.B / step_s, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{sample} of {BH} (batch, kv-head) streams of the same workload; "
                      f"decode attention (decompress + float64 Algorithm 1) scaled by {scale:.2f}",
            "attn_s_per_step_est": step_s,
            "prune_compress_tokens_per_s": sample * w.N / t_pc,
            "wall_s": t_pc + t_attn}


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

    w = synth.WORKLOADS[args.workload]
    steps, warm = args.steps, args.warmup
    torch.cuda.set_device(0)
    dev = "cuda"
    cap = w.N + warm + steps + 1

    # ---- synthetic inputs, resident in HBM ----
    K, V = synth.make_kv_torch(w.B, w.Hkv, w.N + w.n_tail, w.d, seed=args.seed, device=dev)
    KL = K[:, :, w.N:].contiguous()                    # dense window
    VL = V[:, :, w.N:].contiguous()
    Kp = K[:, :, :w.N].contiguous()
    Vp = V[:, :, :w.N].contiguous()
    gq = torch.Generator(device=dev)
    gq.manual_seed(args.seed)
    q = torch.randn((w.B, w.Hq, w.d), generator=gq, device=dev).half()
    new_k = KL[:, :, 0].contiguous()                  # the token leaving the window each step
    new_v = VL[:, :, 0].contiguous()
    Kc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, cap, device=dev)
    Vc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, cap, device=dev)
    ws_c = torch.empty(mf.mustafar_compress_workspace_bytes(w.B, w.Hkv, w.N), dtype=torch.uint8,
                       device=dev)
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

    # ---- bulk prune + compress of the prefill cache (K and V), timed ----
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
    k_len0 = int(Kc.stream_len.to(torch.int64).sum().item())
    v_len0 = int(Vc.stream_len.to(torch.int64).sum().item())

    # ---- dense baseline over the same tokens ----
    ws_d = torch.empty(mf.mustafar_attn_workspace_bytes(w.B, w.Hq, w.Hkv, w.d, w.N + w.n_tail,
                                                        args.splits), dtype=torch.uint8, device=dev)
    a, b = ev(), ev()
    n_dense_reps = 20
    for _ in range(20):
        mf.mustafar_dense_decode_attn(q, K, V, out=out, n_splits=args.splits, ws=ws_d)
    torch.cuda.synchronize()
    a.record()
    for _ in range(n_dense_reps):
        mf.mustafar_dense_decode_attn(q, K, V, out=out, n_splits=args.splits, ws=ws_d)
    b.record()
    torch.cuda.synchronize()
    t_dense = a.elapsed_time(b) / 1e3 / n_dense_reps
    dense_bytes = 2 * 2 * w.B * w.Hkv * (w.N + w.n_tail) * w.d + 4 * w.B * w.Hq * w.d

    # ---- decode steps: append (prune+compress one token per stream) + attention ----
    def step(marks=None):
        mf.mustafar_append_kv(Kc, Vc, new_k, new_v)
        if marks is not None:
            marks[0].record()
        mf.mustafar_sparse_decode_attn(q, Kc, Vc, KL, VL, out=out, n_splits=args.splits, ws=ws_a)
        if marks is not None:
            marks[1].record()

    marks = [(ev(), ev()) for _ in range(steps)]
    t_start, t_end = ev(), ev()
    for _ in range(warm):
        step()
    torch.cuda.synchronize()
    n_s_start = Kc.n_tokens
    wall0 = time.perf_counter()
    t_start.record()
    for i in range(steps):
        step(marks[i])
    t_end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_s = t_start.elapsed_time(t_end) / 1e3
    attn_s = float(np.mean([m[0].elapsed_time(m[1]) for m in marks])) / 1e3
    n_s_end = Kc.n_tokens

    # algorithmic bytes of the attention launches, averaged over the timed steps
    k_len1 = int(Kc.stream_len.to(torch.int64).sum().item())
    v_len1 = int(Vc.stream_len.to(torch.int64).sum().item())
    per_tok_k = (k_len1 - k_len0) / max(1, n_s_end - w.N)
    per_tok_v = (v_len1 - v_len0) / max(1, n_s_end - w.N)
    alg = []
    for n_s in range(n_s_start + 1, n_s_end + 1):
        extra = n_s - w.N
        alg.append(attn_alg_bytes(w, int(k_len0 + per_tok_k * extra), int(v_len0 + per_tok_v * extra),
                                  n_s))
    alg_bytes = float(np.mean(alg))
    attn_gbs = alg_bytes / attn_s / 1e9
    dense_kv = 2 * 2 * w.B * w.Hkv * w.N * w.d
    comp_kv = 12 * w.B * w.Hkv * w.N * (w.d // 64) * 2 + 2 * (k_len0 + v_len0)

    # ---- the same decode steps through the dense-window lifecycle: the ring of the
    # last n_tail tokens, a push per step that graduates the oldest token of the full
    # ring (prune + compress + append), then attention over compressed + ring ----
    window = None
    if not args.no_window:
        del Kc, Vc
        torch.cuda.empty_cache()
        Kw = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, cap, device=dev)
        Vw = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, cap, device=dev)
        win = mf.DenseWindow(w.B, w.Hkv, w.d, w.n_tail, device=dev)
        mf.mustafar_window_prefill(win, Kw, Vw, K, V, [w.N + w.n_tail] * w.B, ws_c)

        def wstep(marks=None):
            mf.mustafar_window_step(win, Kw, Vw, new_k, new_v)
            if marks is not None:
                marks[0].record()
            mf.mustafar_window_decode_attn(q, Kw, Vw, win, out=out, n_splits=args.splits, ws=ws_a)
            if marks is not None:
                marks[1].record()

        wmarks = [(ev(), ev()) for _ in range(steps)]
        a, b = ev(), ev()
        for _ in range(warm):
            wstep()
        torch.cuda.synchronize()
        a.record()
        for i in range(steps):
            wstep(wmarks[i])
        b.record()
        torch.cuda.synchronize()
        w_total = a.elapsed_time(b) / 1e3 / steps
        w_attn = float(np.mean([m[0].elapsed_time(m[1]) for m in wmarks])) / 1e3
        window = {"us_per_step": w_total * 1e6, "attention_us": w_attn * 1e6,
                  "window_step_us": (w_total - w_attn) * 1e6, "tokens_per_s": w.B / w_total,
                  "how": "mustafar_window_step + mustafar_window_decode_attn, ring of "
                         f"{w.n_tail} tokens per stream"}
        del Kw, Vw, win
        torch.cuda.empty_cache()

        # The same steps with output-aware keys: the leaving key is pruned with the
        # weights its window slot gathered from the queries of its 32 steps.
        Kw = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, cap, device=dev)
        Vw = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, cap, device=dev)
        win = mf.DenseWindow(w.B, w.Hkv, w.d, w.n_tail, device=dev)
        kacc = torch.zeros((w.B, w.Hkv, w.n_tail, w.d), dtype=torch.float32, device=dev)
        mf.mustafar_window_prefill(win, Kw, Vw, K, V, [w.N + w.n_tail] * w.B, ws_c)

        def kstep(marks=None):
            mf.mustafar_window_step_weighted(win, Kw, Vw, new_k, new_v, kacc)
            mf.mustafar_window_decode_attn(q, Kw, Vw, win, out=out, n_splits=args.splits, ws=ws_a)
            if marks is not None:
                marks[0].record()
            mf.mustafar_window_key_weights(q, win, kacc)
            if marks is not None:
                marks[1].record()

        kmarks = [(ev(), ev()) for _ in range(steps)]
        a, b = ev(), ev()
        for _ in range(warm):
            kstep()
        torch.cuda.synchronize()
        a.record()
        for i in range(steps):
            kstep(kmarks[i])
        b.record()
        torch.cuda.synchronize()
        k_total = a.elapsed_time(b) / 1e3 / steps
        k_kw = float(np.mean([m[0].elapsed_time(m[1]) for m in kmarks])) / 1e3
        window["output_aware_keys"] = {
            "us_per_step": k_total * 1e6, "key_weights_us": k_kw * 1e6,
            "tokens_per_s": w.B / k_total,
            "how": "mustafar_window_step_weighted + mustafar_window_decode_attn + "
                   "mustafar_window_key_weights (|q| of the step into the newest 32 slots)"}
        del Kw, Vw, win, kacc

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
                    "magnitude_tokens_per_s_for_reference": 2 * toks / t_pc}
        del Kv, qhist, wts
        torch.cuda.empty_cache()

    channel = None
    if not args.no_channel:
        channel = channel_leg(v_len0)

    ceiling = read_ceiling_gbs()

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
        "attention": {"us": attn_s * 1e6, "tokens_per_s": w.B / attn_s,
                      "kv_tokens_per_s": w.B * w.Hkv * (n_s_end + w.n_tail) / attn_s,
                      "alg_bytes": alg_bytes, "gb_s": attn_gbs},
        "roofline": {"bound": "hbm", "achieved": attn_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": attn_gbs / HBM_PEAK_GBS,
                     "traffic": measured_traffic("k_sparse_attn", w.name)},
        "read_ceiling": {"gb_s": ceiling, "attn_frac": attn_gbs / ceiling,
                         "how": "mustafar_stream_read (16-byte loads) over an 8 GiB buffer"},
        "dense_baseline": {"us": t_dense * 1e6, "tokens_per_s": w.B / t_dense,
                           "gb_s": dense_bytes / t_dense / 1e9},
        "speedup_vs_dense": t_dense / attn_s,
        "prune_compress": {"ms": t_pc * 1e3, "tokens_per_s": w.B * w.Hkv * w.N / t_pc,
                           "alg_bytes": dense_kv + comp_kv,
                           "gb_s": (dense_kv + comp_kv) / t_pc / 1e9,
                           "frac": (dense_kv + comp_kv) / t_pc / 1e9 / HBM_PEAK_GBS,
                           "traffic": measured_traffic("k_compress", w.name, "bytes_k_plus_v")},
        "append_us_per_step": (total_s / steps - attn_s) * 1e6,
        "window_lifecycle": window,
        "prune_variants": variants,
        "channel_pruning": channel,
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
        threads = args.cpu_threads or min(16, os.cpu_count() or 1)
        result["cpu_baseline"] = cpu_baseline(w, Kp, Vp, KL, VL, q, args.cpu_sample_streams,
                                              threads)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
