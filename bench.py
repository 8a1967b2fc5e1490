"""Benchmark: batch-1 decode tokens/s and prefill TTFT of the HIP path on one GPU.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 8b]

One step = one request of the workload: reset the KV cache, prefill the prompt
(TTFT), then the configured number of greedy decode steps.  Inputs (weights,
prompt ids) are seeded synthetic data generated on the host and uploaded once,
before the timed region.  Prints one JSON line.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12          # MI355X HBM3E, bytes/s
MFMA_BF16_PEAK = 2.5e15    # MI355X dense bf16 matrix peak, flop/s


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def run_request(model, prompt, n_decode, device_resident=False):
    """One request: reset, prefill (TTFT), n_decode greedy steps, either one
    wici_decode_step call per token or one wici_decode_n call for all of them."""
    model.reset_kv()
    t0 = time.perf_counter()
    tok, _ = model.prefill(prompt)
    t1 = time.perf_counter()
    if device_resident:
        model.decode_n(n_decode)
    else:
        for _ in range(n_decode):
            model.decode_step(-1)
    t2 = time.perf_counter()
    return t1 - t0, t2 - t1, tok


def gateup_bytes(cfg) -> int:
    """Algorithmic HBM bytes of one gate/up GEMV launch: both weight matrices once,
    the input vector and norm gain read, the SwiGLU output written."""
    return 2 * cfg.ffn_dim * cfg.d_model * cfg.wbytes + 2 * cfg.d_model * 4 + cfg.ffn_dim * 4


def measured_traffic(cfg):
    """HBM bytes per gate/up GEMV launch from the committed memory-counter summary,
    if it was taken on this workload with the current kernel source; else None."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"traffic_gemv_gateup_{cfg.name}.md")
    src = os.path.join(ROOT, "paper_2608_24204_amd", "csrc", "gemv.hip")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    want = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    if f"gemv.hip: {want}" not in text:
        return None
    for line in text.splitlines():
        if line.startswith("traffic_bytes_per_launch gateup:"):
            return int(line.split(":")[1])
    return None


def profile_pass(model, cfg, prompt, n_decode):
    """Eager decode steps, each launch timed by start/stop events recorded by its
    kernels' dispatches (same positions as a timed request).  Returns mean
    per-launch ms per kernel class and per-token sums."""
    model.reset_kv()
    model.prefill(prompt)
    L = cfg.n_layers
    acc = {k: [] for k in ("embed", "qkv", "attn", "o", "gateup", "down", "lm_head", "argmax")}
    for _ in range(n_decode):
        _, dur = model.profile_decode_step(-1)
        acc["embed"].append(dur[0])
        per = dur[1:1 + 5 * L].reshape(L, 5)
        for j, k in enumerate(("qkv", "attn", "o", "gateup", "down")):
            acc[k].extend(per[:, j].tolist())
        acc["lm_head"].append(dur[1 + 5 * L])
        acc["argmax"].append(dur[2 + 5 * L])
    mean = {k: float(np.mean(v)) for k, v in acc.items()}
    per_token = {k: float(np.sum(v)) / n_decode for k, v in acc.items()}
    return mean, per_token


def stream_ceiling(nbytes=4 << 30, grids=(512, 768, 1024), reps=5):
    """The plain streaming-read rate of this GPU's memory, measured in this run
    with the library's own read kernel (wici_stream_read): the best of a few
    launch shapes, each after one untimed read.  Returns (bytes/s, details)."""
    import torch

    from paper_2608_24204_amd import binding
    buf = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    sink = torch.empty(max(grids) * 1024 + 4, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    per = {}
    for g in grids:
        binding.stream_read(buf, g, 1, sink)
        per[g] = binding.stream_read(buf, g, reps, sink)
    del buf, sink
    best = min(per, key=per.get)
    return nbytes / (per[best] / 1e3), {"bytes": nbytes, "reps": reps, "best_grid": best,
                                        "ms_per_read": {str(g): v for g, v in per.items()}}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, w, n_prompt, n_decode):
    """The float64 oracle on the host cores over a bounded sample of the workload
    (a shorter prompt, a few decode steps); returns the sample's ids and logits so
    the GPU path can be compared with it."""
    from threadpoolctl import threadpool_info

    from oracle import DecoderOracle, greedy, q8_model_f64
    from paper_2608_24204_amd import inputs
    t0 = time.perf_counter()
    # a block-scaled 8-bit model: the oracle quantises the same source weights itself
    w64 = q8_model_f64(w) if cfg.weight_dtype == "q8" else inputs.weights_f64(cfg, w)
    conv_s = time.perf_counter() - t0
    prompt = inputs.make_prompt(cfg, n_prompt)
    orc = DecoderOracle(cfg, w64, max_seq=n_prompt + n_decode + 1)
    t0 = time.perf_counter()
    lg = orc.prefill(prompt)
    t1 = time.perf_counter()
    ids, logs = [greedy(lg)], [lg]
    for _ in range(n_decode):
        lg = orc.decode(ids[-1])
        ids.append(greedy(lg))
        logs.append(lg)
    t2 = time.perf_counter()
    threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    out = {"value": n_decode / (t2 - t1), "unit": "tokens/s", "cores": int(threads),
           "kind": "oracle",
           "sample": f"{cfg.name}: prefill of {n_prompt} prompt ids then {n_decode} greedy decode "
                     f"steps, float64 numpy on the host (weights "
                     f"{'quantised by the oracle and ' if cfg.weight_dtype == 'q8' else ''}"
                     f"widened to float64 beforehand, {conv_s:.1f} s, not timed)",
           "prefill_tok_s": n_prompt / (t1 - t0), "ttft_ms": (t1 - t0) * 1e3,
           "host_cpus": os.cpu_count(), "cpu_model": cpu_model()}
    return out, (prompt, ids, logs)


def model_cache_sweep(cfg_name, store_root, thresholds_mib):
    """Model load time against the caching threshold (the paper's model-caching
    figure): per threshold, the caller's MD5 time over the tensors at or above it,
    a cold load into an empty store (hash, upload, save), a warm load sending only
    those hashes (store reads + upload), the bytes the caller still sends, and a
    plain upload for reference.  Prints one JSON line."""
    import shutil

    import torch

    from paper_2608_24204_amd import binding, configs, inputs
    cfg = configs.CONFIGS[cfg_name]
    w = inputs.make_weights(cfg)
    total = sum(a.nbytes for a in w.values())
    rows = []

    def fresh():
        return binding.WiciModel(cfg, max_seq=64)

    m = fresh()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    m.load_weights(w)
    plain_s = time.perf_counter() - t0
    m.close()
    for t_mib in thresholds_mib:
        thr = int(t_mib * 2 ** 20)
        store = os.path.join(store_root, f"wici_store_{t_mib}")
        shutil.rmtree(store, ignore_errors=True)
        os.makedirs(store)
        big = [n for n, a in w.items() if a.nbytes >= thr]
        t0 = time.perf_counter()
        hashes = {n: binding.md5(w[n]) for n in big}
        hash_s = time.perf_counter() - t0
        m = fresh()
        t0 = time.perf_counter()
        out = m.load_weights_cached(w, store, thr)
        cold_s = time.perf_counter() - t0
        m.close()
        m = fresh()
        t0 = time.perf_counter()
        out2 = m.load_weights_cached(w, store, thr, hashes=hashes)
        warm_s = time.perf_counter() - t0
        m.close()
        sent = sum(w[n].nbytes for n in w if n not in hashes)
        rows.append({"threshold_mib": t_mib, "hashed_tensors": len(big),
                     "hash_s": hash_s, "cold_load_s": cold_s,
                     "warm_load_s": warm_s, "warm_total_s": hash_s + warm_s,
                     "bytes_sent_warm": sent,
                     "hits": sum(o == binding.WICI_CACHE_HIT for o in out2.values()),
                     "saved_cold": sum(o == binding.WICI_CACHE_SAVED for o in out.values())})
        log(f"threshold {t_mib} MiB: {len(big)} hashed, hash {hash_s:.2f} s, cold "
            f"{cold_s:.2f} s, warm {warm_s:.2f} s, caller sends {sent / 1e6:.1f} MB")
        shutil.rmtree(store, ignore_errors=True)
    print(json.dumps({"metric": "model load time vs caching threshold", "config": cfg_name,
                      "tensors": len(w), "model_bytes": total, "plain_load_s": plain_s,
                      "rows": rows}), flush=True)
    return 0


def batch_sweep(cfg_name, batches, n_steps):
    """Aggregate decode tokens/s of B clients sharing one weight copy, advanced
    together by wici_decode_batch (each prefilled with its own prompt of the
    workload's length).  Prints one JSON line."""
    import torch

    from paper_2608_24204_amd import binding, configs, inputs
    cfg = configs.CONFIGS[cfg_name]
    w = inputs.make_weights(cfg)
    rng = np.random.default_rng(123)
    top = max(batches)
    lead = binding.WiciModel(cfg)
    lead.load_weights(w)
    ms = [lead] + [binding.WiciModel(cfg, share_weights_of=lead) for _ in range(top - 1)]
    rows = []
    for B in batches:
        group = ms[:B]
        for m in group:
            m.reset_kv()
            m.prefill(rng.integers(0, cfg.vocab, cfg.prompt_len).astype(np.int32))
        lead.decode_batch(group)                       # warm-up step
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n_steps):
            lead.decode_batch(group)
        dt = time.perf_counter() - t0
        ctx = cfg.prompt_len + 1 + n_steps / 2
        kv = B * ctx * cfg.n_layers * 2 * cfg.kv_dim * cfg.kvbytes
        wbytes = cfg.decode_bytes_per_token(0)
        rows.append({"batch": B, "tok_s": B * n_steps / dt, "step_ms": dt / n_steps * 1e3,
                     "hbm_frac": (wbytes + kv) * n_steps / dt / HBM_PEAK})
        log(f"batch {B}: {B * n_steps / dt:.1f} tok/s, {dt / n_steps * 1e3:.2f} ms/step")
    for m in ms:
        m.close()
    print(json.dumps({"metric": "batched decode tokens/s (clients sharing weights)",
                      "config": cfg_name, "steps": n_steps, "rows": rows}), flush=True)
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="8b")
    ap.add_argument("--decode", type=int, default=None, help="override decode steps per request")
    ap.add_argument("--prefill-mode", default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true")
    ap.add_argument("--cpu-prompt", type=int, default=None,
                    help="prompt ids of the oracle sample (default: the workload's prompt)")
    ap.add_argument("--cpu-decode", type=int, default=3)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="before the timed region, copy MIB MiB device-to-device (a plain "
                         "copy of known size, for calibrating memory counters)")
    ap.add_argument("--model-cache", action="store_true",
                    help="instead of the benchmark: model load time against the caching "
                         "threshold (store under --store-root)")
    ap.add_argument("--store-root", default=os.environ.get("TMPDIR", "/tmp"))
    ap.add_argument("--batch-sweep", default=None, metavar="B1,B2,...",
                    help="instead of the benchmark: aggregate tokens/s of batched decode")
    args = ap.parse_args(argv)
    if args.batch_sweep:
        return batch_sweep(args.config, [int(b) for b in args.batch_sweep.split(",")],
                           args.decode or 32)
    if args.model_cache:
        return model_cache_sweep(args.config, args.store_root,
                                 [0, 0.0625, 1, 16, 64, 256, 4096])
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the decode path runs on a single GPU; it has no multi-GPU sharding)", file=sys.stderr)
        return 2

    import torch

    from paper_2608_24204_amd import binding, configs, inputs
    cfg = configs.CONFIGS[args.config]
    n_decode = cfg.decode_steps if args.decode is None else args.decode
    log(f"config {cfg.name}: generating weights")
    t0 = time.perf_counter()
    w = inputs.make_weights(cfg)
    log(f"weights generated in {time.perf_counter() - t0:.1f} s")
    prompt = inputs.make_prompt(cfg)
    model = binding.WiciModel(cfg, prefill_mode=args.prefill_mode,
                              max_seq=cfg.prompt_len + n_decode)
    t0 = time.perf_counter()
    model.load_weights(w)
    log(f"weights uploaded in {time.perf_counter() - t0:.1f} s")

    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {args.calibrate_copy} MiB done")
        del src, dst
    log("stream-read ceiling")
    ceil_bps, ceil_info = stream_ceiling()
    log(f"stream-read ceiling {ceil_bps / 1e9:.0f} GB/s")
    for i in range(args.warmup):
        ttft, dec, _ = run_request(model, prompt, n_decode)
        log(f"warmup {i}: ttft {ttft * 1e3:.2f} ms, decode {n_decode / dec:.1f} tok/s")
    torch.cuda.synchronize()
    ttfts, decs = [], []
    t_start = time.perf_counter()
    for i in range(args.steps):
        ttft, dec, tok = run_request(model, prompt, n_decode)
        ttfts.append(ttft)
        decs.append(dec)
        log(f"step {i}: ttft {ttft * 1e3:.2f} ms, decode {n_decode / dec:.1f} tok/s")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    # the same requests with the decode steps in one device-resident call
    dn = []
    for i in range(args.steps):
        _, dec, _ = run_request(model, prompt, n_decode, device_resident=True)
        dn.append(dec)
    torch.cuda.synchronize()
    log(f"wici_decode_n: {n_decode * args.steps / sum(dn):.1f} tok/s")

    decode_tok_s = n_decode * args.steps / sum(decs)
    ttft_ms = float(np.median(ttfts)) * 1e3
    mean_ctx = cfg.prompt_len + (n_decode + 1) / 2.0
    bytes_tok = cfg.decode_bytes_per_token(int(round(mean_ctx)))
    pf_flops = cfg.prefill_flops()
    res = {
        "metric": "batch-1 decode tokens/s (+ prefill TTFT ms, % of HBM roofline), 1 MI355X",
        "value": decode_tok_s, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.weight_dtype, "data": "synthetic (seeded N(0,0.02^2) weights, uniform prompt ids)",
        "config": {"workload": f"{cfg.name}-shaped dense decoder: {cfg.n_layers} layers, d {cfg.d_model}, "
                               f"{cfg.n_heads}q/{cfg.n_kv_heads}kv heads x {cfg.head_dim}, FFN {cfg.ffn_dim}, "
                               f"vocab {cfg.vocab}; prompt {cfg.prompt_len}, {n_decode} greedy decode steps, batch 1",
                   "global_batch": 1, "seq_len": cfg.prompt_len + n_decode, "parallelism": "none"},
        "ttft_ms": ttft_ms, "prefill_tok_s": cfg.prompt_len / (ttft_ms / 1e3),
        "decode_bytes_per_token": bytes_tok,
        "decode_hbm_frac": bytes_tok * decode_tok_s / HBM_PEAK,
        "stream_read_ceiling_gbs": ceil_bps / 1e9,
        "decode_frac_of_stream_ceiling": bytes_tok * decode_tok_s / ceil_bps,
        "stream_read": ceil_info,
        "prefill_flops": pf_flops,
        "prefill_mfma_frac": pf_flops / (ttft_ms / 1e3) / MFMA_BF16_PEAK,
        "prefill_mode": args.prefill_mode or ("f32" if cfg.weight_dtype == "f32" else "bf16x3q"),
        "decode_n_tok_s": n_decode * args.steps / sum(dn),
        "decode_n_hbm_frac": bytes_tok * n_decode * args.steps / sum(dn) / HBM_PEAK,
    }

    if not args.no_profile:
        log("profiling pass (eager launches timed by dispatch-recorded HIP events)")
        mean, per_tok = profile_pass(model, cfg, prompt, n_decode)
        gu = gateup_bytes(cfg)
        ach = gu / (mean["gateup"] / 1e3)
        res["roofline"] = {"kernel": "k_gemv gate/up (+RMSNorm prologue, SwiGLU epilogue)",
                           "bound": "hbm", "achieved": ach / 1e9, "peak": HBM_PEAK / 1e9,
                           "unit": "GB/s", "frac": ach / HBM_PEAK, "traffic": measured_traffic(cfg),
                           "bytes_per_launch": gu, "avg_launch_ms": mean["gateup"],
                           "method": "start/stop HIP events recorded by the kernel's dispatch "
                                     "(hipExtLaunchKernelGGL) on the model's stream, eager "
                                     "profiling pass over one request's decode steps"}
        res["decode_kernel_ms_per_token"] = per_tok
        res["decode_kernel_sum_ms"] = float(sum(per_tok.values()))
        res["decode_step_ms"] = 1e3 / decode_tok_s

    if not args.no_cpu_baseline:
        log("cpu baseline (oracle sample)")
        cb, (sp, sids, slogs) = cpu_baseline(cfg, w, args.cpu_prompt or cfg.prompt_len,
                                             args.cpu_decode)
        # same sample through the GPU path
        model.reset_kv()
        g_ids, g_logs = model.generate(sp, args.cpu_decode, want_logits=True)
        rel = max(float(np.max(np.abs(g - o)) / np.max(np.abs(o))) for g, o in zip(g_logs, slogs))
        res["cpu_baseline"] = cb
        res["parity_sample"] = {"ids_equal": [int(i) for i in g_ids] == [int(i) for i in sids],
                                "max_rel_err": rel, "tokens": len(sids)}
    model.close()
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
