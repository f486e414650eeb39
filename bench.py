"""Decode-step benchmark of the INT2 KV-cache hot path on one MI355X.

One step = the cache write of each sequence's current token (quantize-append of B tokens) plus
the decode attention over the whole INT2 context (query rotation, split-context scan, merge with
the R_V^T un-rotation, W_O projection). Workload (default): 64 sequences with contexts drawn
uniformly from [512, 32768] (seeded), 40 query / 8 KV heads, head_dim 128, paged blocks of 16
tokens permuted across one shared pool, INT2 groups of 32 with fp16 scale/zero, W_O 5120x5120
bf16. Inputs are seeded synthetic tensors already resident in HBM when timing starts.

Prints one JSON line (rank 0). Progress goes to stderr.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "INT2 decode-attn KV-tokens/s and achieved HBM GB/s (% of peak), 1 MI355X"


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_02691_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def counter_traffic(kernel_key, units_per_launch):
    """HBM bytes per launch of the scan kernel from committed rocprofv3 counter summaries, or
    None when absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    entry = data.get(kernel_key)
    if not entry or entry.get("source_hash") != kernel_source_hash():
        return None
    return entry["hbm_bytes_per_launch"]


class HipEvents:
    """Raw HIP events (the library attaches them to the scan kernel's dispatch: its start and end)."""

    def __init__(self, n):
        import ctypes
        self.ct = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.pairs = []
        for _ in range(n):
            a, b = ctypes.c_void_p(), ctypes.c_void_p()
            for e in (a, b):
                st = self.hip.hipEventCreate(ctypes.byref(e))
                if st != 0:
                    raise RuntimeError(f"hipEventCreate failed: {st}")
            self.pairs.append((a.value, b.value))

    def elapsed_ms(self, i):
        ms = self.ct.c_float()
        a, b = self.pairs[i]
        st = self.hip.hipEventElapsedTime(self.ct.byref(ms), self.ct.c_void_p(a), self.ct.c_void_p(b))
        if st != 0:
            raise RuntimeError(f"hipEventElapsedTime failed: {st}")
        return ms.value

    def destroy(self):
        for a, b in self.pairs:
            self.hip.hipEventDestroy(self.ct.c_void_p(a))
            self.hip.hipEventDestroy(self.ct.c_void_p(b))


def cpu_baseline(w, target_s, group=32):
    """Time the CPU oracle's decode (with W_O) on a bounded sample of this workload's sequences."""
    from oracle import int2kv_oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover - threadpoolctl is optional
        cores = 1
    tokens = 0
    elapsed = 0.0
    seqs = []
    for b in range(w.batch):
        L = int(w.ctx_lens[b])
        nblk = (L + 15) // 16
        pool = O.new_pool(nblk, w.num_kv_heads, group)
        table = np.arange(nblk, dtype=np.int32)[None]
        k, v = w.kv(b)
        pos = np.arange(L)
        O.quantize_append(pool, k, v, (table[0, pos // 16] * 16 + pos % 16), w.R_k, w.R_v, w.mu)
        t0 = time.perf_counter()
        O.decode(pool, w.q[b:b + 1], table, np.array([L], np.int32), w.R_k, w.R_v, w.W_o)
        elapsed += time.perf_counter() - t0
        tokens += L
        seqs.append(b)
        log(f"cpu oracle: sequence {b} ({L} tokens), {elapsed:.1f} s so far")
        if elapsed >= target_s:
            break
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    return {"value": tokens / elapsed, "unit": "KV-tokens/s", "cores": int(cores), "kind": "oracle",
            "host_cpus": os.cpu_count(), "cpu_model": model,
            "sample": f"oracle decode (+W_O) of sequences {seqs[0]}..{seqs[-1]} of the same workload "
                      f"({tokens} KV-tokens, {elapsed:.1f} s, fp64 numpy)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--chunk", type=int, default=0, help="context chunk in tokens (0 = automatic)")
    ap.add_argument("--variant", type=int, default=0, help="decode scan variant (0 auto, 1 VALU, 2 MFMA)")
    ap.add_argument("--wo", choices=("prepared", "folded", "plain"), default="prepared",
                    help="output-projection weights: prepared fp16 tiles with R_V folded in (default), row-major "
                         "bf16 folded with R_V, or row-major bf16 W_O with the merge un-rotating o")
    ap.add_argument("--group", type=int, default=32, choices=(32, 128),
                    help="INT2 group size of the cache (32; 128 is the paper's serving setting: 72 instead of 96 "
                         "bytes per token and KV head)")
    ap.add_argument("--separate", action="store_true",
                    help="append and decode as two calls (default: int2kv_append_decode, the cache write beside "
                         "the query preparation)")
    ap.add_argument("--window", type=str, default="",
                    help="SINK,RECENT: keep the first SINK and last RECENT tokens of each sequence in the BF16 "
                         "window (the paper's serving setting is 64,256 with --group 128); the step is then "
                         "int2kv_window_write + int2kv_quantize_append + int2kv_decode_window")
    ap.add_argument("--event-every", type=int, default=10,
                    help="time the scan kernel with HIP events on every n-th timed step (events attached to a "
                         "dispatch add ~11 us of queue gaps to that step)")
    ap.add_argument("--ctx", type=int, default=0,
                    help="uniform context length override (e.g. --config 1 --ctx 32768: the 402.7 MB uniform "
                         "32K variant of the 16-sequence shape)")
    ap.add_argument("--flush-mall", action="store_true",
                    help="read a 1 GiB scratch buffer before every timed step (evicts L2 and the Infinity "
                         "Cache, for workloads that would otherwise fit in it, and leaves no dirty lines behind); "
                         "steps are then timed one by one")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (see DESIGN.md for "
              "how the decode would shard); run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_02691_amd import int2kv as K
    from paper_2608_02691_amd import workloads as W

    torch.cuda.set_device(0)
    if args.copy_calibration:
        n = 1 << 30
        src_t = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst_t = torch.empty_like(src_t)
        for _ in range(3):
            dst_t.copy_(src_t)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n, "bytes_written": n, "launches": 3}), flush=True)
        return
    K.int2kv_set_decode_tuning(args.chunk, args.variant)
    w = W.make_workload(args.config, ctx=args.ctx or None)
    B, Hq, H = w.batch, w.num_q_heads, w.num_kv_heads
    d_model = w.cfg.d_model or 0
    lens = w.ctx_lens.astype(np.int64)
    log(f"workload cfg{args.config}: B={B} Hq={Hq} H={H} sum(L)={int(lens.sum())} max(L)={int(lens.max())}")

    dev = lambda a: torch.from_numpy(a.view(np.int16).copy() if a.dtype == np.uint16 else np.ascontiguousarray(a)).cuda()
    cache = K.Int2KVCache(w.num_blocks, H, group_size=args.group)
    Rk, Rv = dev(w.R_k), dev(w.R_v)
    mu_rk = K.int2kv_prepare_mu_rot(Rk, dev(w.mu))
    q = dev(w.q)
    table = dev(w.block_table)
    ctx = dev(w.ctx_lens)
    Wo = dev(w.W_o) if w.W_o is not None else None
    # weight preparation, once per layer (the value fold W_O R_V; tiling), outside the timed steps
    wo_format = K.INT2KV_WO_PLAIN
    if Wo is not None and args.wo == "prepared":
        Wo, wo_format = K.int2kv_prepare_wo(Wo, Rv, Hq), K.INT2KV_WO_PREPARED_FOLDED
    elif Wo is not None and args.wo == "folded":
        Wo, wo_format = K.int2kv_fold_wo(Wo, Rv, Hq), K.INT2KV_WO_FOLDED
    k_last = torch.empty((B, H, 128), dtype=torch.bfloat16, device="cuda")
    v_last = torch.empty_like(k_last)
    # BF16 window (--window): tokens [0, sink) and [L - recent, L) of each sequence live in the window
    # store (rows b * cap + t), the rest in the INT2 cache at positions 0 .. L - sink - recent - 1
    sink, recent = (int(x) for x in args.window.split(",")) if args.window else (0, 0)
    cap = sink + recent
    lens_int2 = np.maximum(lens - cap, 0) if cap else lens
    win_lens = np.minimum(lens, cap).astype(np.int32)
    if cap:
        win_k = torch.zeros((B * cap, H, 128), dtype=torch.bfloat16, device="cuda")
        win_v = torch.zeros_like(win_k)
        mu_d = dev(w.mu)
        k_cur = torch.empty_like(k_last)
        v_cur = torch.empty_like(k_last)
        cur_rows = dev(np.array([b * cap + int(win_lens[b]) - 1 for b in range(B)], np.int32))
        win_lens_d = dev(win_lens)
    # the step re-appends the last INT2 token of each sequence (none, slot -1, when all are in the window)
    last_slots = np.array([w.slot_mapping(b, int(lens_int2[b]) - 1)[0] if lens_int2[b] > 0 else -1
                           for b in range(B)], np.int32)
    t0 = time.time()
    for b in range(B):
        k, v = w.kv(b, as_torch=True)
        L = int(lens[b])
        kd, vd = k.cuda(), v.cuda()
        if cap:
            n2 = int(lens_int2[b])
            wi = torch.cat([torch.arange(0, min(sink, L)), torch.arange(max(L - recent, min(sink, L)), L)])
            K.int2kv_window_write(kd[wi], vd[wi], dev(np.arange(b * cap, b * cap + wi.numel(), dtype=np.int32)),
                                  mu_d, win_k, win_v)
            k_cur[b], v_cur[b] = kd[L - 1], vd[L - 1]
            kd, vd, L = kd[sink:sink + n2], vd[sink:sink + n2], n2
        if L > 1:
            K.int2kv_quantize_append(cache, kd[:L - 1], vd[:L - 1], dev(w.slot_mapping(b, 0, L - 1)), Rk, Rv, mu_rk)
        if L > 0:
            k_last[b] = kd[L - 1]
            v_last[b] = vd[L - 1]
        if b % 8 == 7:
            torch.cuda.synchronize()
            log(f"prefilled {b + 1}/{B} sequences ({time.time() - t0:.1f} s)")
    slots_d = dev(last_slots)
    max_ctx = int(lens_int2.max())
    ctx = dev(lens_int2.astype(np.int32))
    ws = torch.empty(K.int2kv_decode_workspace_bytes(B, Hq, H, max_ctx, d_model), dtype=torch.uint8, device="cuda")
    out = torch.empty((B, d_model) if d_model else (B, Hq, 128), dtype=torch.float32, device="cuda")

    def step():
        if cap:
            # the current token enters the recent ring, the token leaving it goes to INT2
            K.int2kv_window_write(k_cur, v_cur, cur_rows, mu_d, win_k, win_v)
            K.int2kv_quantize_append(cache, k_last, v_last, slots_d, Rk, Rv, mu_rk)
            K.int2kv_decode_window(cache, q, table, ctx, max_ctx, Rk, Rv, win_k, win_v, win_lens_d, cap, W_o=Wo,
                                   wo_format=wo_format, d_model=d_model, out=out, workspace=ws)
        elif args.separate:
            K.int2kv_quantize_append(cache, k_last, v_last, slots_d, Rk, Rv, mu_rk)
            K.int2kv_decode(cache, q, table, ctx, max_ctx, Rk, Rv, W_o=Wo, wo_format=wo_format, d_model=d_model,
                            out=out, workspace=ws)
        else:
            K.int2kv_append_decode(cache, k_last, v_last, slots_d, mu_rk, q, table, ctx, max_ctx, Rk, Rv, W_o=Wo,
                                   wo_format=wo_format, d_model=d_model, out=out, workspace=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    if args.flush_mall:
        # every step timed alone (torch events around it), the scan with events on its dispatch; the
        # 1 GiB read before each step is outside both (a read, so no dirty lines are left to write back)
        scratch = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        sampled = list(range(args.steps))
        ev = HipEvents(args.steps)
        t_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in sampled]
        torch.cuda.synchronize()
        for i in range(args.steps):
            sink = scratch.sum()
            K.int2kv_set_decode_events(*ev.pairs[i])
            t_ev[i][0].record()
            step()
            t_ev[i][1].record()
        torch.cuda.synchronize()
        K.int2kv_set_decode_events(None, None)
        ms_step = float(np.mean([a.elapsed_time(b) for a, b in t_ev]))
        scan_ms = float(np.mean([ev.elapsed_ms(j) for j in range(args.steps)]))
        ev.destroy()
        del scratch, sink
        log(f"timed {args.steps} steps one by one after a 1 GiB read each: {ms_step:.3f} ms/step "
            f"(includes the events' own queue gaps), scan kernel {scan_ms:.3f} ms")
    else:
        every = max(1, args.event_every)
        sampled = list(range(0, args.steps, every))
        ev = HipEvents(len(sampled))
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record()
        for i in range(args.steps):
            if i % every == 0:
                K.int2kv_set_decode_events(*ev.pairs[i // every])
            elif i % every == 1:
                K.int2kv_set_decode_events(None, None)
            step()
        stop.record()
        torch.cuda.synchronize()
        K.int2kv_set_decode_events(None, None)
        ms_step = start.elapsed_time(stop) / args.steps
        scan_ms = float(np.mean([ev.elapsed_ms(j) for j in range(len(sampled))]))
        ev.destroy()
        log(f"timed {args.steps} steps: {ms_step:.3f} ms/step, scan kernel {scan_ms:.3f} ms "
            f"(events on {len(sampled)} of the steps)")

    # context: a plain 1 GiB device-to-device copy on the same GPU (read + write bytes over time)
    cp_src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    cp_dst = torch.empty_like(cp_src)
    cp_dst.copy_(cp_src)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(3):
        cp_dst.copy_(cp_src)
    c1.record()
    torch.cuda.synchronize()
    copy_gbps = 3 * 2 * (1 << 30) / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del cp_src, cp_dst

    tokens = int(lens.sum())  # tokens attended (INT2 and window)
    pages = int(((lens_int2 + 15) // 16).sum())
    tok_bytes = 64 + 8 * (128 // args.group)  # K and V codes + one (s, z) fp16 pair per group each: 96 or 72
    scan_bytes = tok_bytes * H * int(lens_int2.sum()) + 4 * pages
    step_bytes = (scan_bytes + B * Hq * 256 + (B * d_model * 4 if d_model else B * Hq * 512)
                  + 2 * H * 128 * 128 * 4 + (2 * d_model * Hq * 128 if d_model else 0)
                  + B * H * (512 + tok_bytes))
    scan_gbps = scan_bytes / (scan_ms * 1e-3) / 1e9
    step_gbps = step_bytes / (ms_step * 1e-3) / 1e9
    if cap:
        step_bytes += int(win_lens.sum()) * H * 512  # bf16 window keys and values
    # the committed counters cover the default scan only (group 32, no window, the configuration's contexts)
    traffic = (counter_traffic(f"decode_scan_cfg{args.config}", 1)
               if args.group == 32 and not cap and not args.ctx else None)

    result = {
        "metric": METRIC,
        "value": tokens / (ms_step * 1e-3),
        "unit": "KV-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int2 codes, fp16 meta, fp32 accumulate",
        "data": "synthetic (seeded; no model weights or traces)",
        "kv_token_heads_per_s": tokens * H / (ms_step * 1e-3),
        "step_hbm_gbps": step_gbps,
        "step_pct_hbm_peak": 100.0 * step_gbps / HBM_PEAK_GBPS,
        "config": {
            "workload": w.cfg.name if not args.ctx else f"{w.cfg.name}; context set to a uniform {args.ctx}",
            "config_id": args.config, "batch": B, "num_q_heads": Hq, "num_kv_heads": H, "head_dim": 128, "block_size": 16,
            "group_size": args.group, "sum_ctx": tokens, "max_ctx": max_ctx, "d_model": d_model,
            "chunk_tokens": args.chunk or "auto", "variant": args.variant or "auto",
            "step_calls": ("int2kv_window_write + int2kv_quantize_append + int2kv_decode_window" if cap else
                           "int2kv_quantize_append + int2kv_decode" if args.separate else
                           "int2kv_append_decode (cache write inside the preparation launch)"),
            "bf16_window": f"{sink} sink + {recent} recent tokens" if cap else None,
            "w_o": {"prepared": "W_O R_V folded, fp16 tiles (prepared once)",
                    "folded": "W_O R_V folded, bf16 row-major (prepared once)",
                    "plain": "W_O bf16 row-major after R_V^T"}[args.wo] if Wo is not None else None,
        },
        "roofline": {
            "kernel": "decode split-context scan",
            "bound": "hbm",
            "achieved": scan_gbps,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": scan_gbps / HBM_PEAK_GBPS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": scan_bytes,
            "avg_launch_ms": scan_ms,
            "timed_launches": len(sampled),
            "caches": "flushed (1 GiB read) before every step" if args.flush_mall else "warm, steps back to back",
        },
        "context": {"hbm_copy_gbps": copy_gbps, "copy": "1 GiB device-to-device copy, read + write bytes"},
    }
    if not args.no_cpu_baseline and not cap:  # the oracle timing covers the INT2-only step
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds, args.group)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
