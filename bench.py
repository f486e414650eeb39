"""Decode-step benchmark of the INT2 KV-cache hot path on one MI355X.

One step = the cache write of each sequence's current token (quantize-append of B tokens) plus
the decode attention over the whole INT2 context (query rotation, split-context scan, merge with
the R_V^T un-rotation, W_O projection). Workload (default): 64 sequences with contexts drawn
uniformly from [512, 32768] (seeded), 40 query / 8 KV heads, head_dim 128, paged blocks of 16
tokens permuted across one shared pool, INT2 groups of 32 with fp16 scale/zero, W_O 5120x5120
bf16. Inputs are seeded synthetic tensors already resident in HBM when timing starts.

Timing: W untimed warm-up steps, then K steps back to back between two events (ms_per_step,
value, gate), then a separate sample phase of --samples steps whose dominant kernel carries HIP
events on its own dispatch; the median of those launches gives the roofline. --mode append times
the prefill-sized cache write instead (configuration 3); --mode outerr times the output-error
diagnostics of Sec. 3.2 over the cache and the full-precision rows it was written from
(configuration 1 by default when chosen), and reports their RMS output error relative to plain INT2.

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


# the sources each measured kernel is built from (its file, the headers it includes, and the host
# code that sizes its launch); counters stay valid while these files are unchanged
_COMMON = ("common.h", "kernels.h", "api.hip")
KERNEL_SOURCES = {
    "decode_scan": ("decode_mfma.hip", "append_core.h") + _COMMON,
    "qprep": ("decode_mfma.hip", "append_core.h") + _COMMON,
    "merge": ("decode_mfma.hip", "append_core.h") + _COMMON,
    "append": ("append.hip", "append_core.h") + _COMMON,
    "wo": ("wo_gemm.hip",) + _COMMON,
    "wo_reduce": ("wo_gemm.hip",) + _COMMON,
    "outerr_scan": ("outerr.hip",) + _COMMON,
}


def kernel_source_hash(kernel_key=None):
    """Hash of the kernel sources a counter entry was taken on (kernel_key such as "decode_scan_cfg4";
    None: every source)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_02691_amd", "csrc")
    files = KERNEL_SOURCES.get(kernel_key.rsplit("_cfg", 1)[0]) if kernel_key else None
    for name in sorted(files or os.listdir(csrc)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def committed_counters(kernel_key):
    """Counter figures of one kernel and workload from the committed rocprofv3 summaries
    (profiles/counters.json): HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, scaled by a plain
    copy's reading), matrix-core busy fraction where taken. None when absent or taken on other
    kernel sources."""
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    entry = data.get(kernel_key)
    if not entry or entry.get("source_hash") != kernel_source_hash(kernel_key):
        return None
    return entry


class HipEvents:
    """Raw HIP events (the library attaches them to its dominant kernel's dispatch: start and end)."""

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


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return int(max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1]))
    except Exception:  # pragma: no cover - threadpoolctl is optional
        return 1


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            return next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        return ""


def cpu_baseline(w, target_s, group=32):
    """Time the CPU oracle's decode (with W_O) on a bounded sample of this workload's sequences."""
    from oracle import int2kv_oracle as O
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
    return {"value": tokens / elapsed, "unit": "KV-tokens/s", "cores": blas_threads(), "kind": "oracle",
            "host_cpus": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": f"oracle decode (+W_O) of sequences {seqs[0]}..{seqs[-1]} of the same workload "
                      f"({tokens} KV-tokens, {elapsed:.1f} s, fp64 numpy)"}


def cpu_baseline_outerr(w, target_s, group=32):
    """Time the CPU oracle's output-error diagnostics on a bounded sample of the workload's sequences."""
    from oracle import int2kv_oracle as O
    tokens, elapsed, seqs = 0, 0.0, []
    for b in range(w.batch):
        L = int(w.ctx_lens[b])
        nblk = (L + 15) // 16
        pool = O.new_pool(nblk, w.num_kv_heads, group)
        table = np.arange(nblk, dtype=np.int32)[None]
        k, v = w.kv(b)
        O.quantize_append(pool, k, v, np.arange(L, dtype=np.int32), w.R_k, w.R_v, w.mu)
        t0 = time.perf_counter()
        O.output_error(pool, [k], [v], w.q[b:b + 1], np.array([L], np.int32), table, w.R_k, w.R_v, w.mu, w.W_o)
        elapsed += time.perf_counter() - t0
        tokens += L
        seqs.append(b)
        log(f"cpu oracle: output error of sequence {b} ({L} tokens), {elapsed:.1f} s so far")
        if elapsed >= target_s:
            break
    return {"value": tokens / elapsed, "unit": "KV-tokens/s (output-error diagnostics)", "cores": blas_threads(),
            "kind": "oracle", "host_cpus": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": f"oracle output-error diagnostics (+W_O) of sequences {seqs[0]}..{seqs[-1]} of the same "
                      f"workload ({tokens} KV-tokens, {elapsed:.1f} s, fp64 numpy)"}


def cpu_baseline_append(w, target_s, group=32):
    """Time the CPU oracle's cache write (center, rotate, quantize, pack) on a bounded sample of the
    workload's sequences."""
    from oracle import int2kv_oracle as O
    tokens, elapsed, seqs = 0, 0.0, []
    for b in range(w.batch):
        L = int(w.ctx_lens[b])
        nblk = (L + 15) // 16
        pool = O.new_pool(nblk, w.num_kv_heads, group)
        k, v = w.kv(b)
        t0 = time.perf_counter()
        O.quantize_append(pool, k, v, np.arange(L, dtype=np.int32), w.R_k, w.R_v, w.mu)
        elapsed += time.perf_counter() - t0
        tokens += L
        seqs.append(b)
        log(f"cpu oracle: append of sequence {b} ({L} tokens), {elapsed:.1f} s so far")
        if elapsed >= target_s:
            break
    return {"value": tokens / elapsed, "unit": "appended KV-tokens/s", "cores": blas_threads(), "kind": "oracle",
            "host_cpus": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": f"oracle cache write of sequences {seqs[0]}..{seqs[-1]} of the same workload "
                      f"({tokens} tokens x {w.num_kv_heads} KV heads, {elapsed:.1f} s, fp64/fp32 numpy)"}


def run_calibrate(args):
    """OptR offline calibration (Algorithm 1) of --layers Qwen3-8B-shaped layers (8 KV heads, 32
    query heads, d_model 4096 each) at the paper's settings (group 128, clips 0.96 / 0.92, 64 sink
    and 256 recent BF16 tokens, final 64 query positions, 80 Adam steps per rotation at lr 0.02,
    held-out selection every 20 steps, lambda_K = 1) on seeded traces: 7 calibration sequences of
    328..560 tokens and 6 held-out sequences of 400..640 tokens. Every layer's heads are calibrated
    in the same launches (the KV-head axis spans the layers). One timed unit is one whole
    calibration."""
    import torch
    from paper_2608_02691_amd import int2kv as K
    from paper_2608_02691_amd import workloads as W
    torch.cuda.set_device(0)
    L = args.layers
    H, Hq, dm = 8 * L, 32 * L, 4096
    kc, vc, qc, sc = W.calibration_traces(7, (328, 560), H, Hq, seed=1)
    kh, vh, qh, sh = W.calibration_traces(6, (400, 640), H, Hq, seed=2)
    calib = K.OptrTraces(kc.cuda(), vc.cuda(), qc.cuda(), sc)
    held = K.OptrTraces(kh.cuda(), vh.cuda(), qh.cuda(), sh)
    R0k = torch.from_numpy(W.haar_rotations(H, 3)).cuda()
    R0v = torch.from_numpy(W.haar_rotations(H, 4)).cuda()
    g = torch.Generator().manual_seed(5)
    # each layer's W_O [4096, 32 * 128]: the layers side by side along the columns
    W_o = (torch.randn((dm, Hq * 128), generator=g) / np.sqrt(dm)).to(torch.bfloat16).cuda()
    mu = K.int2kv_optr_key_mean(calib.k)
    cfg = K.optr_config(H, Hq, dm)
    n_ws = K.int2kv_optr_workspace_bytes(cfg, calib, held)
    ws = torch.empty(n_ws, dtype=torch.uint8, device="cuda")
    log(f"calibrate: {L} layers = {H} KV heads, calib {int(sc[-1])} / held-out {int(sh[-1])} tokens, "
        f"workspace {n_ws / 2**30:.2f} GiB")
    run = lambda: K.int2kv_optr_calibrate(cfg, calib, held, R0k, R0v, mu, W_o, workspace=ws)
    warm = max(1, min(args.warmup, 2))
    steps = max(1, min(args.steps, 5))
    for _ in range(warm):
        out = run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        out = run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    hist = out["history"].cpu().numpy()
    n_ev = 1 + cfg.steps // cfg.eval_every
    held_k, held_v = hist[0, :, cfg.steps:], hist[1, :, cfg.steps:]
    sel_k = held_k.min(axis=1) / held_k[:, 0]
    sel_v = held_v.min(axis=1) / held_v[:, 0]
    log(f"calibration: {ms:.1f} ms; held-out objective of the selected rotation over the base: keys median "
        f"{np.median(sel_k):.3f}, values median {np.median(sel_v):.3f}")
    result = {
        "metric": "OptR offline calibration (Algorithm 1) throughput, 1 MI355X",
        "value": H / (ms * 1e-3),
        "unit": "calibrated KV heads/s",
        "n_gpus": 1, "steps": steps, "warmup": warm, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64 (bf16 traces, fp32 R0; INT2 quantizer on fp32 rows)",
        "data": "synthetic (seeded traces; no model weights)",
        "config": {"workload": f"OptR calibration of {L} Qwen3-8B-shaped layers (8 KV / 32 query heads, d_model 4096)",
                   "kv_heads": H, "calib_tokens": int(sc[-1]), "heldout_tokens": int(sh[-1]), "group_size": 128,
                   "clip": [0.96, 0.92], "window": [64, 256], "n_last": 64, "adam_steps": [cfg.steps, cfg.steps],
                   "lr": cfg.lr, "eval_every": cfg.eval_every, "lambda_k": cfg.lambda_k},
        "selection": {"heldout_key_ratio_median": float(np.median(sel_k)),
                      "heldout_value_ratio_median": float(np.median(sel_v)),
                      "what": "held-out objective of the selected rotation over that of the base rotation R0"},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_calibrate(kc, vc, qc, sc, kh, vh, qh, sh, R0k.cpu().numpy(),
                                                        R0v.cpu().numpy(), mu.cpu().numpy(), W_o, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def cpu_baseline_calibrate(kc, vc, qc, sc, kh, vh, qh, sh, R0k, R0v, mu, W_o, target_s):
    """The oracle's calibration of KV head 0 (its own 4 query heads and its W_O columns), with the
    steps cut to fit the time budget; scaled to whole calibrations (80 + 80 steps) per second."""
    from oracle import optr_oracle as P
    import torch
    bits = lambda t: t.view(torch.int16).numpy().view(np.uint16)
    c0 = (bits(kc[:, :1]), bits(vc[:, :1]), bits(qc[:, :4]), sc)
    h0 = (bits(kh[:, :1]), bits(vh[:, :1]), bits(qh[:, :4]), sh)
    Wo = bits(W_o[:, :4 * 128].cpu().contiguous())
    t0 = time.perf_counter()
    steps = 2
    P.calibrate_head(R0k[:1], R0v[:1], c0, h0, mu[:1], Wo, 0, 4, lam=1.0, clip_k=0.96, clip_v=0.92, group=128,
                     n_last=64, sink=64, recent=256, steps=steps, lr=0.02, eval_every=steps)
    el = time.perf_counter() - t0
    # one oracle step (loss + gradient) costs about one held-out evaluation plus its backward; scale
    # the 2 + 2 steps and 2 + 2 evaluations measured to 80 + 80 steps and 5 + 5 evaluations
    per_head = el * (160 + 10) / (2 * steps + 4)
    log(f"cpu oracle: {2 * steps} calibration steps of one KV head in {el:.1f} s -> {per_head:.1f} s per head")
    return {"value": 1.0 / per_head, "unit": "calibrated KV heads/s", "cores": blas_threads(), "kind": "oracle",
            "host_cpus": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": f"oracle calibrate_head of KV head 0 with {steps} + {steps} steps and {2 + 2} held-out "
                      f"evaluations ({el:.1f} s, fp64 torch), scaled to 80 + 80 steps and 5 + 5 evaluations"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--config", type=int, default=None,
                    help="workload configuration (default 4; 1 with --mode outerr)")
    ap.add_argument("--layers", type=int, default=36,
                    help="calibrate mode: decoder layers calibrated at once (8 KV heads each)")
    ap.add_argument("--mode", choices=("decode", "append", "outerr", "calibrate"), default="decode",
                    help="decode: one decode step (default); append: the cache write of every token of the "
                         "workload in one int2kv_quantize_append call (configuration 3's prefill-sized append); "
                         "outerr: one int2kv_output_error call (key- and value-induced output errors against the "
                         "full-precision rows); calibrate: OptR's offline calibration (Algorithm 1) of --layers "
                         "Qwen3-8B-shaped layers on synthetic traces")
    ap.add_argument("--rope", action="store_true",
                    help="append mode: the keys enter pre-RoPE and the write applies RoPE at each token's position "
                         "(int2kv_quantize_append_rope, fp32 cos/sin table of theta 1e6)")
    ap.add_argument("--hadamard", action="store_true",
                    help="append mode: rotate keys and values by the in-kernel Hadamard matrix instead of R_K, R_V")
    ap.add_argument("--chunk", type=int, default=0, help="context chunk in tokens (0 = automatic)")
    ap.add_argument("--variant", type=int, default=0, help="decode scan variant (0 auto, 1 VALU, 2 MFMA)")
    ap.add_argument("--wo", choices=("prepared", "folded", "plain"), default="prepared",
                    help="output-projection weights: prepared fp16 tiles with R_V folded in (default), row-major "
                         "bf16 folded with R_V, or row-major bf16 W_O with the merge un-rotating o")
    ap.add_argument("--group", type=int, default=32, choices=(32, 128),
                    help="INT2 group size of the cache (32; 128 is the paper's serving setting: 72 instead of 96 "
                         "bytes per token and KV head)")
    ap.add_argument("--clip", type=str, default="1,1",
                    help="clip ratios c_K,c_V of the cache writes (the paper's serving setting uses 0.96,0.92)")
    ap.add_argument("--separate", action="store_true",
                    help="append and decode as two calls (default: int2kv_append_decode, the cache write beside "
                         "the query preparation)")
    ap.add_argument("--window", type=str, default="",
                    help="SINK,RECENT: keep the first SINK and last RECENT tokens of each sequence in the BF16 "
                         "window (the paper's serving setting is 64,256 with --group 128); the step is then "
                         "int2kv_window_write + int2kv_quantize_append + int2kv_decode_window")
    ap.add_argument("--samples", type=int, default=20,
                    help="launches of the dominant kernel timed one by one with HIP events after the timed steps "
                         "(its median gives the roofline; events on a dispatch add queue gaps, so the timed "
                         "steps carry none)")
    ap.add_argument("--steady-steps", type=int, default=400,
                    help="steps run back to back after the timed ones and timed on their own (steady_state): the "
                         "GPU's power management slows every kernel by 10-30 %% over the first ~150 steps of "
                         "sustained load, then settles; the kernel samples are taken after these steps")
    ap.add_argument("--ctx", type=int, default=0,
                    help="uniform context length override (e.g. --config 1 --ctx 32768: the 402.7 MB uniform "
                         "32K variant of the 16-sequence shape)")
    ap.add_argument("--flush-mall", action="store_true",
                    help="read a 1 GiB scratch buffer before every timed step and every sample (evicts L2 and the "
                         "Infinity Cache, for workloads that would otherwise fit in it, and leaves no dirty lines "
                         "behind); steps are then timed one by one")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (the decode would shard "
              "by KV head and sequence, one process per GPU); run it with --gpus 1", file=sys.stderr)
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
    if args.mode == "calibrate":
        run_calibrate(args)
        return
    if args.config is None:
        args.config = 1 if args.mode == "outerr" else 4
    K.int2kv_set_decode_tuning(args.chunk, args.variant)
    clip_k, clip_v = (float(x) for x in args.clip.split(","))
    w = W.make_workload(args.config, ctx=args.ctx or None)
    B, Hq, H = w.batch, w.num_q_heads, w.num_kv_heads
    d_model = w.cfg.d_model or 0
    lens = w.ctx_lens.astype(np.int64)
    append_mode = args.mode == "append"
    log(f"workload cfg{args.config} ({args.mode}): B={B} Hq={Hq} H={H} sum(L)={int(lens.sum())} "
        f"max(L)={int(lens.max())}")

    dev = lambda a: torch.from_numpy(a.view(np.int16).copy() if a.dtype == np.uint16 else np.ascontiguousarray(a)).cuda()
    cache = K.Int2KVCache(w.num_blocks, H, group_size=args.group)
    Rk, Rv = dev(w.R_k), dev(w.R_v)
    mu_rk = K.int2kv_prepare_mu_rot(Rk, dev(w.mu))
    tok_bytes = 64 + 8 * (128 // args.group)  # K and V codes + one (s, z) fp16 pair per group each: 96 or 72
    R_bytes = 2 * H * 128 * 128 * 4
    ev_box = {"ev": None}  # the dominant call of a step attaches these events (sample phase only)

    def with_events(call):
        if ev_box["ev"] is not None:
            K.int2kv_set_decode_events(*ev_box["ev"])
        call()
        if ev_box["ev"] is not None:
            K.int2kv_set_decode_events(None, None)

    outerr_mode = args.mode == "outerr"
    diag = None
    if outerr_mode:
        if d_model == 0:
            raise SystemExit("--mode outerr needs a configuration with W_O (1 or 4)")
        # the cache and the bf16 rows it was written from (row b * row_cap + t), plus a plain INT2
        # cache (identity rotations, no centering) of the same tokens for the relative metric
        row_cap = int(lens.max())
        k_rows = torch.zeros((B * row_cap, H, 128), dtype=torch.bfloat16, device="cuda")
        v_rows = torch.zeros_like(k_rows)
        plain = K.Int2KVCache(w.num_blocks, H, group_size=args.group)
        eye = torch.eye(128, dtype=torch.float32, device="cuda").expand(H, 128, 128).contiguous()
        zero_mu = torch.zeros((H, 128), dtype=torch.float32, device="cuda")
        for b in range(B):
            k, v = w.kv(b, as_torch=True)
            L = int(lens[b])
            kd, vd = k.cuda(), v.cuda()
            k_rows[b * row_cap:b * row_cap + L] = kd
            v_rows[b * row_cap:b * row_cap + L] = vd
            sl = dev(w.slot_mapping(b))
            K.int2kv_quantize_append(cache, kd, vd, sl, Rk, Rv, mu_rk, clip_k, clip_v)
            K.int2kv_quantize_append(plain, kd, vd, sl, eye, eye, zero_mu, 1.0, 1.0)
        torch.cuda.synchronize()
        log(f"prefilled {B} sequences and their bf16 rows")
        q = dev(w.q)
        table = dev(w.block_table)
        Wo = dev(w.W_o)
        ctx = dev(w.ctx_lens.astype(np.int32))
        max_ctx = int(lens.max())
        ws = torch.empty(K.int2kv_output_error_workspace_bytes(B, Hq, H, max_ctx, d_model), dtype=torch.uint8,
                         device="cuda")
        stats = torch.empty((B, Hq, 4), dtype=torch.float32, device="cuda")
        oe_args = (q, table, ctx, max_ctx, Rk, Rv, k_rows, v_rows, row_cap, Wo)

        def step():
            with_events(lambda: K.int2kv_output_error(cache, *oe_args, workspace=ws, stats=stats))

        dom_name = "output-error scan (outerr_scan_kernel)"
        pages = int(((lens + 15) // 16).sum())
        dom_bytes = (tok_bytes + 512) * H * int(lens.sum()) + 4 * pages
        step_bytes = dom_bytes + 2 * d_model * Hq * 128 + R_bytes + B * Hq * 256 + B * Hq * 16
        tokens = int(lens.sum())
        # the per-head metric: RMS output error of the rotated cache as a percentage of plain INT2's
        st_rot = K.int2kv_output_error(cache, *oe_args).cpu().double().numpy()
        st_plain = K.int2kv_output_error(plain, *oe_args).cpu().double().numpy()
        pct = 100.0 * np.sqrt(st_rot[..., 0] / st_plain[..., 0])
        share_k = st_rot[..., 1] / st_rot[..., 0]
        diag = {"what": "E_out of the cache per (sequence, query head) against plain INT2 of the same tokens "
                        "(identity rotations, no centering, no clipping), from int2kv_output_error",
                "rms_percent_of_plain_int2": {"median": float(np.median(pct)), "mean": float(pct.mean()),
                                              "p90": float(np.percentile(pct, 90))},
                "key_share_of_e_out_median": float(np.median(share_k)),
                "cross_term_over_e_out_median": float(np.median(st_rot[..., 3] / st_rot[..., 0]))}
        del plain
    elif append_mode:
        # every token of every sequence in one call, into an empty permuted pool; repeated steps
        # rewrite the same slots
        kk, vv, ss = [], [], []
        for b in range(B):
            k, v = w.kv(b, as_torch=True)
            kk.append(k)
            vv.append(v)
            ss.append(w.slot_mapping(b))
        k_all, v_all = torch.cat(kk).cuda(), torch.cat(vv).cuda()
        slots_all = dev(np.concatenate(ss))
        n_tok = int(slots_all.numel())
        flags = (K.INT2KV_HADAMARD_K | K.INT2KV_HADAMARD_V) if args.hadamard else 0
        if args.hadamard:
            Hd = K.hadamard_rotation(H)
            mu_rk = K.int2kv_prepare_mu_rot(Hd, dev(w.mu))
        pos_all = cs_tab = None
        if args.rope:
            pos_all = dev(np.concatenate([np.arange(int(lens[b]), dtype=np.int32) for b in range(B)]))
            cs_tab = dev(W.rope_cos_sin(int(lens.max())))

        if args.rope or args.hadamard:
            def step():
                with_events(lambda: K.int2kv_quantize_append_rope(
                    cache, k_all, v_all, slots_all, pos_all, cs_tab, None if args.hadamard else Rk,
                    None if args.hadamard else Rv, mu_rk, clip_k, clip_v, flags=flags))
        else:
            def step():
                with_events(lambda: K.int2kv_quantize_append(cache, k_all, v_all, slots_all, Rk, Rv, mu_rk, clip_k,
                                                             clip_v))

        dom_name = "cache write (append_mfma_kernel)"
        dom_bytes = (n_tok * H * (512 + tok_bytes) + 4 * n_tok + (0 if args.hadamard else R_bytes) + H * 128 * 4
                     + (4 * n_tok + int(lens.max()) * 512 if args.rope else 0))
        step_bytes = dom_bytes
        tokens = n_tok
        max_ctx = 0
    else:
        q = dev(w.q)
        table = dev(w.block_table)
        Wo = dev(w.W_o) if w.W_o is not None else None
        # weight preparation, once per layer (the value fold W_O R_V; tiling), outside the timed steps
        wo_format = K.INT2KV_WO_PLAIN
        if Wo is not None and args.wo == "prepared":
            Wo, wo_format = K.int2kv_prepare_wo(Wo, Rv, Hq), K.INT2KV_WO_PREPARED_FOLDED
        elif Wo is not None and args.wo == "folded":
            Wo, wo_format = K.int2kv_fold_wo(Wo, Rv, Hq), K.INT2KV_WO_FOLDED
        k_last = torch.empty((B, H, 128), dtype=torch.bfloat16, device="cuda")
        v_last = torch.empty_like(k_last)
        # BF16 window (--window): tokens [0, sink) and [L - recent, L) of each sequence live in the
        # window store (rows b * cap + t), the rest in the INT2 cache at positions 0 .. L - sink - recent - 1
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
                K.int2kv_quantize_append(cache, kd[:L - 1], vd[:L - 1], dev(w.slot_mapping(b, 0, L - 1)), Rk, Rv,
                                         mu_rk, clip_k, clip_v)
            if L > 0:
                k_last[b] = kd[L - 1]
                v_last[b] = vd[L - 1]
            if b % 8 == 7 or b == B - 1:
                torch.cuda.synchronize()
                log(f"prefilled {b + 1}/{B} sequences ({time.time() - t0:.1f} s)")
        slots_d = dev(last_slots)
        max_ctx = int(lens_int2.max())
        ctx = dev(lens_int2.astype(np.int32))
        ws = torch.empty(K.int2kv_decode_workspace_bytes(B, Hq, H, max_ctx, d_model), dtype=torch.uint8,
                         device="cuda")
        out = torch.empty((B, d_model) if d_model else (B, Hq, 128), dtype=torch.float32, device="cuda")

        def step():
            if cap:
                # the current token enters the recent ring, the token leaving it goes to INT2
                K.int2kv_window_write(k_cur, v_cur, cur_rows, mu_d, win_k, win_v)
                K.int2kv_quantize_append(cache, k_last, v_last, slots_d, Rk, Rv, mu_rk, clip_k, clip_v)
                with_events(lambda: K.int2kv_decode_window(cache, q, table, ctx, max_ctx, Rk, Rv, win_k, win_v,
                                                           win_lens_d, cap, W_o=Wo, wo_format=wo_format,
                                                           d_model=d_model, out=out, workspace=ws))
            elif args.separate:
                K.int2kv_quantize_append(cache, k_last, v_last, slots_d, Rk, Rv, mu_rk, clip_k, clip_v)
                with_events(lambda: K.int2kv_decode(cache, q, table, ctx, max_ctx, Rk, Rv, W_o=Wo,
                                                    wo_format=wo_format, d_model=d_model, out=out, workspace=ws))
            else:
                with_events(lambda: K.int2kv_append_decode(cache, k_last, v_last, slots_d, mu_rk, q, table, ctx,
                                                           max_ctx, Rk, Rv, W_o=Wo, wo_format=wo_format,
                                                           d_model=d_model, clip_k=clip_k, clip_v=clip_v, out=out,
                                                           workspace=ws))

        tokens = int(lens.sum())  # tokens attended (INT2 and window)
        pages = int(((lens_int2 + 15) // 16).sum())
        dom_name = "decode split-context scan (decode_scan_flat_kernel)"
        dom_bytes = tok_bytes * H * int(lens_int2.sum()) + 4 * pages
        # the whole decode step: KV stream + block table, q, outputs, R_K and R_V, W_O, the current
        # tokens' cache write (bf16 in, INT2 out), the BF16 window tokens
        step_bytes = (dom_bytes + B * Hq * 256 + (B * d_model * 4 if d_model else B * Hq * 512) + R_bytes
                      + (2 * d_model * Hq * 128 if d_model else 0) + B * H * (512 + tok_bytes))
        if cap:
            step_bytes += int(win_lens.sum()) * H * 512 + B * H * 1024  # window rows read; current rows written

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    scratch = torch.ones(1 << 28, dtype=torch.float32, device="cuda") if args.flush_mall else None
    flush_sink = []
    if args.flush_mall:
        # every step timed alone after a 1 GiB read (a read, so no dirty lines are left to write back)
        t_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        torch.cuda.synchronize()
        for i in range(args.steps):
            flush_sink.append(scratch.sum())
            t_ev[i][0].record()
            step()
            t_ev[i][1].record()
        torch.cuda.synchronize()
        ms_step = float(np.median([a.elapsed_time(b) for a, b in t_ev]))
        log(f"timed {args.steps} steps one by one after a 1 GiB read each: median {ms_step:.4f} ms/step")
    else:
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record()
        for _ in range(args.steps):
            step()
        stop.record()
        torch.cuda.synchronize()
        ms_step = start.elapsed_time(stop) / args.steps
        log(f"timed {args.steps} steps back to back: {ms_step:.4f} ms/step")

    # steady state: more steps back to back, timed on their own (after the power manager's transient)
    steady_ms = None
    if args.steady_steps > 0 and not args.flush_mall:
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record()
        for _ in range(args.steady_steps):
            step()
        s1.record()
        torch.cuda.synchronize()
        steady_ms = s0.elapsed_time(s1) / args.steady_steps
        log(f"steady state: {args.steady_steps} more steps back to back: {steady_ms:.4f} ms/step")

    # the dominant kernel: args.samples more steps, each with HIP events on that kernel's dispatch
    ev = HipEvents(args.samples)
    torch.cuda.synchronize()
    for i in range(args.samples):
        if args.flush_mall:
            flush_sink.append(scratch.sum())
        ev_box["ev"] = ev.pairs[i]
        step()
    ev_box["ev"] = None
    torch.cuda.synchronize()
    durs = np.array([ev.elapsed_ms(j) for j in range(args.samples)])
    dom_ms = float(np.median(durs))
    ev.destroy()
    del scratch, flush_sink
    log(f"{dom_name}: median {dom_ms:.4f} ms over {args.samples} launches (min {durs.min():.4f}, "
        f"max {durs.max():.4f})")

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
    # and a read-only stream of the same 1 GiB (torch's sum over int64 words: plain loads)
    rd = cp_src.view(torch.int64)
    rd.sum()
    c0.record()
    for _ in range(3):
        rd.sum()
    c1.record()
    torch.cuda.synchronize()
    read_gbps = 3 * (1 << 30) / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del cp_src, cp_dst, rd

    dom_gbps = dom_bytes / (dom_ms * 1e-3) / 1e9
    step_gbps = step_bytes / (ms_step * 1e-3) / 1e9
    key = (f"append_cfg{args.config}" if append_mode else
           f"outerr_scan_cfg{args.config}" if outerr_mode else f"decode_scan_cfg{args.config}")
    counters = (committed_counters(key)
                if args.group == 32 and not args.window and not args.ctx and args.clip == "1,1"
                and not args.rope and not args.hadamard else None)
    caches = ("flushed (1 GiB read) before every step and sample" if args.flush_mall
              else f"warm, after {args.warmup + args.steps + (args.steady_steps if steady_ms else 0)} steps "
                   "back to back")
    if append_mode and (args.rope or args.hadamard):
        step_calls = ("int2kv_quantize_append_rope (all tokens in one call" + (", RoPE at positions 0..L-1" if args.rope
                      else "") + (", in-kernel Hadamard rotation" if args.hadamard else "") + ")")
    elif append_mode:
        step_calls = "int2kv_quantize_append (all tokens in one call)"
    elif outerr_mode:
        step_calls = "int2kv_output_error (statistics only)"
    elif args.window:
        step_calls = "int2kv_window_write + int2kv_quantize_append + int2kv_decode_window"
    elif args.separate:
        step_calls = "int2kv_quantize_append + int2kv_decode"
    else:
        step_calls = "int2kv_append_decode (cache write inside the preparation launch)"
    result = {
        "metric": METRIC,
        "value": tokens / (ms_step * 1e-3),
        "unit": ("appended KV-tokens/s" if append_mode else
                 "KV-tokens/s (output-error diagnostics)" if outerr_mode else "KV-tokens/s"),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("int2 codes with fp16 scale/zero; matrix-core operands fp16 (q', p, p*s) and bf16x3 (R), "
                  "fp32 accumulate"),
        "data": "synthetic (seeded; no model weights or traces)",
        "kv_token_heads_per_s": tokens * H / (ms_step * 1e-3),
        "gate": {"what": "whole step: algorithmic HBM bytes over ms_per_step",
                 "bytes_per_step": step_bytes, "gbps": step_gbps, "frac": step_gbps / HBM_PEAK_GBPS},
        "steady_state": None if steady_ms is None else {
            "what": f"{args.steady_steps} further steps back to back after the timed ones",
            "ms_per_step": steady_ms, "value": tokens / (steady_ms * 1e-3),
            "gate_frac": step_bytes / (steady_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS},
        "config": {
            "workload": w.cfg.name if not args.ctx else f"{w.cfg.name}; context set to a uniform {args.ctx}",
            "config_id": args.config, "mode": args.mode, "batch": B, "num_q_heads": Hq, "num_kv_heads": H,
            "head_dim": 128, "block_size": 16, "group_size": args.group, "clip": [clip_k, clip_v],
            "sum_ctx": int(lens.sum()), "max_ctx": max_ctx, "d_model": 0 if append_mode else d_model,
            "chunk_tokens": args.chunk or "auto", "variant": args.variant or "auto", "step_calls": step_calls,
            "bf16_window": (f"{args.window.split(',')[0]} sink + {args.window.split(',')[1]} recent tokens"
                            if args.window else None),
            "w_o": None if append_mode or not d_model else "W_O bf16 row-major (per query head slices)"
            if outerr_mode else {
                "prepared": "W_O R_V folded, fp16 tiles (prepared once)",
                "folded": "W_O R_V folded, bf16 row-major (prepared once)",
                "plain": "W_O bf16 row-major after R_V^T"}[args.wo],
        },
        "roofline": {
            "kernel": dom_name,
            "bound": "hbm",
            "achieved": dom_gbps,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": dom_gbps / HBM_PEAK_GBPS,
            "traffic": counters["hbm_bytes_per_launch"] if counters else None,
            "algorithmic_bytes_per_launch": dom_bytes,
            "median_launch_ms": dom_ms,
            "timed_launches": args.samples,
            "caches": caches,
        },
        "context": {"hbm_copy_gbps": copy_gbps, "copy": "1 GiB device-to-device copy, read + write bytes",
                    "hbm_read_gbps": read_gbps, "read": "torch sum over the same 1 GiB (plain loads), bytes read"},
    }
    if diag is not None:
        result["diagnostics"] = diag
        result["dtype"] = "int2 codes with fp16 scale/zero and bf16 rows; fp32 vector arithmetic"
    if counters and counters.get("mfma_busy_frac") is not None:
        result["roofline"]["mfma_busy_frac"] = counters["mfma_busy_frac"]
    # the oracle timing covers the INT2-only step with dense rotations and post-RoPE keys
    if not args.no_cpu_baseline and not args.window and not args.rope and not args.hadamard:
        result["cpu_baseline"] = (cpu_baseline_append(w, args.cpu_seconds, args.group) if append_mode else
                                  cpu_baseline_outerr(w, args.cpu_seconds, args.group) if outerr_mode else
                                  cpu_baseline(w, args.cpu_seconds, args.group))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
