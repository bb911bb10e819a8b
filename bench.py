#!/usr/bin/env python3
"""Benchmark: SDSAT greedy generation on the CodeLlama-7B shape at batch 1.

One step = one full sdsat_generate call: prefill of a 512-token prompt, then
two-step-draft-then-verify loops (k = 5 adaptive tokens) until 256 new tokens
exist.  Weights are random-init N(0, 0.02) in bf16 (seed 1) and the prompt is
uniform random ids: synthetic stand-ins for the fine-tuned checkpoints and the
HumanEval / MultiPL-E prompts of the paper's walltime table, which are not
available.  Inputs are resident in HBM before the timed region.

Printed (one JSON line on stdout): whole-step tokens/s; the roofline of the
block forward (every kernel of one draft or verify block, HIP events on the
library stream around every 4th block of the timed steps) with its dominant
kernel (the gate/up GEMM) inside it; and the CPU oracle timed on a bounded
sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC_7B = "generated tokens/s @bs1 (7B shape, k=5) + block-forward HBM GB/s vs peak"
HBM_PEAK_GBS = 8000.0
BLOCK_PERIOD = 4


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def model_name(sh):
    return {4096: "CodeLlama-7B", 5120: "CodeLlama-13B"}.get(sh.d_model, "small")


def metric_for(wl):
    """The headline metric's name; other workloads name their own batch, shape, k and mode."""
    if wl.name == "7b":
        return METRIC_7B
    short = {4096: "7B", 5120: "13B"}.get(wl.shape.d_model, "small")
    return (f"generated tokens/s @bs{wl.batch} ({short} shape, k={wl.k}, {wl.mode}) + block-forward HBM GB/s "
            f"vs peak")


def block_bytes(sh, B, q, ctx_len):
    """Algorithmic HBM bytes of one block forward: every weight once, the KV
    cache read, the block's K/V written, the embedding rows and the logits."""
    d, F, V, L = sh.d_model, sh.d_ffn, sh.vocab, sh.n_layers
    s = 2
    weights = L * (4 * d * d + 3 * d * F) * s + V * d * s + (2 * L + 1) * d * 4
    kv_read = s * 2 * L * d * B * ctx_len
    kv_write = s * 2 * L * d * B * q
    return weights + kv_read + kv_write + B * q * d * s + 4 * B * q * V


def gateup_bytes(sh, M):
    """Algorithmic bytes of one gate/up launch: the [2F, d] bf16 weight tiles, its M input rows and the
    bf16 SwiGLU output.  A block of several rows reads the normalised rows already rounded to bf16; a
    one-row block reads the float row x o g (gain applied by the producing epilogue) and its
    per-16-column sums of squares."""
    d, F = sh.d_model, sh.d_ffn
    x = M * d * 2 if M > 1 else M * d * 4 + M * (d // 16) * 4
    return 2 * F * d * 2 + x + M * F * 2


def profiled_traffic(workload):
    """HBM bytes per gate/up launch from the committed rocprofv3 counter summary of this workload
    (profiles/gateup_gemm_<workload>_decode.md), if there is one and it was taken from the current
    GEMM source (else None)."""
    import hashlib
    prof = os.path.join(ROOT, "profiles", f"gateup_gemm_{workload}_decode.md")
    src = os.path.join(ROOT, "paper_2403_18647_amd", "csrc", "gemm.hip")
    try:
        text = open(prof).read()
        fields = dict(line.split(": ", 1) for line in text.splitlines()
                      if line.startswith(("traffic_bytes_per_launch: ", "gemm_source_sha256: ")))
        if fields.get("gemm_source_sha256", "").strip() != hashlib.sha256(open(src, "rb").read()).hexdigest():
            return None
        return int(fields["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def profiled_block_traffic(workload):
    """HBM bytes per decode block forward from the committed counter summary of this workload
    (profiles/block_forward_<workload>_decode.md), if every decode kernel source it lists still has
    the recorded hash (else None)."""
    import hashlib
    prof = os.path.join(ROOT, "profiles", f"block_forward_{workload}_decode.md")
    try:
        text = open(prof).read().splitlines()
        traffic = None
        for line in text:
            if line.startswith("traffic_bytes_per_block: "):
                traffic = int(line.split(": ", 1)[1])
            elif line.startswith("source_sha256 "):
                name, digest = line[len("source_sha256 "):].split(": ", 1)
                src = os.path.join(ROOT, "paper_2403_18647_amd", "csrc", name)
                if hashlib.sha256(open(src, "rb").read()).hexdigest() != digest.strip():
                    return None
        return traffic
    except (OSError, ValueError):
        return None


def stream_read_peak(B, torch, region_gib=1, regions=4, iters=12):
    """Achievable HBM read rate on this device: the library's read-only stream kernel over rotating
    1 GiB regions (4 GiB in all, far beyond the 256 MB memory-side cache), events around each launch,
    median launch."""
    n = region_gib << 30
    buf = torch.empty(regions * n, dtype=torch.uint8, device="cuda:0")
    st = torch.cuda.current_stream()
    for i in range(2):
        B.sdsat_stream_read(buf[i * n:(i + 1) * n])
    torch.cuda.synchronize()
    times = []
    for i in range(iters):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        B.sdsat_stream_read(buf[(i % regions) * n:(i % regions + 1) * n])
        e1.record(st)
        e1.synchronize()
        times.append(e0.elapsed_time(e1))
    del buf
    torch.cuda.synchronize()
    ms = sorted(times)[len(times) // 2]
    return n / (ms / 1e3) / 1e9


def host_info():
    """CPU model, logical CPUs usable here, host RAM, BLAS library and thread count."""
    info = {"cpu_model": None, "cpus": None, "ram_gib": None, "blas": None, "blas_threads": None}
    try:
        info["cpus"] = len(os.sched_getaffinity(0))
    except Exception:
        info["cpus"] = os.cpu_count()
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                info["cpu_model"] = line.split(":", 1)[1].strip()
                break
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal"):
                info["ram_gib"] = round(int(line.split()[1]) / 2 ** 20, 1)
                break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        pools = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        if pools:
            info["blas"] = f"{pools[0].get('internal_api')} {pools[0].get('version')}"
            info["blas_threads"] = pools[0].get("num_threads")
    except Exception:
        pass
    return info


def host_stream_gbs(n_bytes=1 << 30, reps=5):
    """Host DRAM read rate seen by the oracle's BLAS: a float32 matrix-vector product over a 1 GiB
    matrix (every byte read once per product), best of `reps`."""
    import numpy as np
    a = np.ones((n_bytes // 4 // 4096, 4096), np.float32)
    x = np.ones(4096, np.float32)
    best = float("inf")
    for _ in range(reps):
        t0 = time.perf_counter()
        a @ x
        best = min(best, time.perf_counter() - t0)
    return round(n_bytes / best / 1e9, 1)


def cpu_baseline(wl, m_bar, n_blocks=4):
    """The oracle on the host cores, on a bounded sample of the workload: the whole model in the
    oracle's float32-BLAS mode with the bf16 storage roundings (float32 copies of the same weights),
    the prompt prefilled in 256-row chunks (timed on its own), then `n_blocks` draft blocks of q rows
    with logits and greedy verification (timed); tokens/s = (m_bar + 2) / (2 x block time) with the
    GPU run's m_bar.  Also the tiny fp32 decoder's float64 SDSAT generation (64 tokens) on one BLAS
    thread and on all of them, and the host facts (CPU, RAM, BLAS threads, DRAM read rate)."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    from oracle import decode as D
    from oracle import model as M
    from paper_2403_18647_amd import synth

    sh = wl.shape
    info = host_info()
    host = {}
    for n in synth.tensor_names(sh):
        t = synth.tensor(wl, n)
        host[n] = synth.bf16_bits_to_f32(t) if t.dtype == np.uint16 else t
    W = M.Weights(sh, host, dtype=np.float32)
    prompt = synth.prompts(wl)[0]
    t0 = time.perf_counter()
    cache = M.prefill(sh, W, prompt[:-1], bf16=True, chunk=256)
    t_prefill = time.perf_counter() - t0
    q = wl.k + 1
    ad = [int(a) for a in synth.adaptive_ids(sh, wl.k)]
    toks = [int(prompt[-1])] + ad
    times = []
    for _ in range(n_blocks):
        pos = np.arange(cache.length, cache.length + q)
        t0 = time.perf_counter()
        logits, kv = M.forward_block(sh, W, cache, toks, pos, bf16=True)
        o, _ = D.verify_greedy(logits.astype(np.float32), None)
        times.append(time.perf_counter() - t0)
        cache.commit(kv, [0])
        toks = [int(o[0])] + ad
    del W, host, cache
    per_block = float(np.mean(times))
    fp32_bytes = 2 * block_bytes(sh, 1, q, len(prompt))    # weights read as float32
    # the tiny decoder (float64 oracle) on one BLAS thread and on all of them
    tiny = synth.workload("tiny")
    Wt = M.Weights(tiny.shape, {n: synth.tensor(tiny, n) for n in synth.tensor_names(tiny.shape)})
    pt = synth.prompts(tiny)[0]
    at = synth.adaptive_ids(tiny.shape, tiny.k)
    tiny_tps = {}
    for label, limit in (("one_thread", 1), ("all_threads", None)):
        with threadpool_limits(limits=limit, user_api="blas"):
            t0 = time.perf_counter()
            D.generate_sdsat(tiny.shape, Wt, pt, tiny.k, tiny.max_new, at)
            tiny_tps[label] = round(tiny.max_new / (time.perf_counter() - t0), 2)
    return {
        "value": round((m_bar + 2.0) / (2.0 * per_block), 4), "unit": "tokens/s",
        "cores": info["blas_threads"] or info["cpus"], "kind": "oracle",
        "sample": (f"whole {sh.n_layers}-layer model, oracle float32-BLAS mode with bf16 storage roundings: "
                   f"{n_blocks} draft blocks of q={q} rows over a {len(prompt) - 1}-token cache (prefill "
                   f"{t_prefill:.1f}s, not counted), {per_block:.3f}s per block incl. LM head and greedy verify; "
                   f"tokens/s = (m_bar+2)/(2 block) with the GPU run's m_bar={m_bar:.3f}"),
        "block_s": round(per_block, 4), "prefill_s": round(t_prefill, 2),
        "block_GBs_fp32_weights": round(fp32_bytes / per_block / 1e9, 1),
        "host": dict(info, dram_read_GBs=host_stream_gbs()),
        "tiny_fp64_sdsat_tokens_per_s": tiny_tps,
    }


def ksweep(B, synth, ctx, wl, prompts, new_tokens=64, k_max=13):
    """Block-forward and loop time against k (Section 3.4.1: the loop time stays almost flat as k
    grows), greedy, with identical adaptive ids (every adaptive row the same id; any k) and with
    diverse ones (ids V..V+k-1; k up to the number of adaptive ids).  Per k: HIP events around every
    block forward of a generation of `new_tokens`, and the same generation with the autoregressive
    continuation injected as drafts (full acceptance, synthetic).  On random-init weights the ids
    change neither the work nor the acceptance; what they do to a trained model's acceptance
    (Appendix B) needs the trained weights."""
    import torch
    sh = wl.shape
    rows = []
    cases = [(k, True) for k in range(0, k_max + 1)] + [(k, False) for k in range(1, min(k_max, sh.n_adaptive) + 1)]
    for k, identical in cases:
        ad = synth.adaptive_ids(sh, k, identical=identical) if k else []
        B.sdsat_generate(ctx.handle, prompts, new_tokens, k, ad)   # warm-up at this block size
        B.sdsat_profile_kernel(ctx.handle, "block")
        _, st = B.sdsat_generate(ctx.handle, prompts, new_tokens, k, ad)
        blk_ms, n_blk = B.sdsat_kernel_time(ctx.handle)
        B.sdsat_profile_kernel(ctx.handle, "off")
        ref, _ = B.sdsat_generate(ctx.handle, prompts, new_tokens + k + 1, 0, ad)
        torch.cuda.synchronize()
        out_f, st_f = B.sdsat_generate(ctx.handle, prompts, new_tokens, k, ad, ref=ref)
        rows.append({"k": k, "q": k + 1, "ids": "identical" if identical else "diverse",
                     "block_ms": round(blk_ms / max(1, n_blk), 4), "m_bar": round(st["accepted"] / max(1, st["loops"]), 3),
                     "loop_ms": round(st_f["decode_ms"] / max(1, st_f["loops"]), 4),
                     "tokens_per_loop_full_accept": k + 2 if k else 2,
                     # the loop rate: k + 2 tokens per loop time (the run's own rate also pays for the
                     # overshoot of its last loop past new_tokens, which depends on new_tokens mod k + 2)
                     "loop_tokens_per_s_full_accept": round((k + 2 if k else 2) * wl.batch /
                                                            (st_f["decode_ms"] / max(1, st_f["loops"]) / 1e3), 1),
                     "decode_tokens_per_s_full_accept": round(new_tokens * wl.batch / (st_f["decode_ms"] / 1e3), 2),
                     "tokens_equal_ar": bool((out_f == ref[:, :new_tokens]).all())})
    return {"metric": "k sweep: block forward and loop time vs k", "unit": "ms", "workload": wl.name,
            "data": "synthetic (random-init weights; identical and diverse adaptive ids; full acceptance "
                    "injected)",
            "new_tokens": new_tokens, "rows": rows}


def micro(B, synth):
    """Kernel micro-benchmarks: device-event times on the library stream, weights rotated past the
    256 MB memory-side cache where they are streamed."""
    import numpy as np
    import torch

    torch.cuda.set_device(0)
    res = {"metric": "kernel micro-benchmarks", "unit": "us", "data": "synthetic", "cases": {}}

    def timed(fn, iters, warm=3):
        for _ in range(warm):
            fn(0)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(iters):
            fn(i)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / iters

    # decode attention: 32 heads x 128, batch 8, 16384 cached keys (zero-filled cache: the time does not
    # depend on the values), q rows per sequence
    H, Dh, Bn, L = 32, 128, 8, 16384
    for q in (6, 11):
        shape = synth.small_shape(n_layers=1, d_model=H * Dh, n_heads=H, head_dim=Dh, d_ffn=64, vocab=64,
                                  n_adaptive=2, rope_base=1e6, dtype="bf16")
        wl = synth.Workload("attn", shape, seed=4, batch=Bn, k=q - 1, prompt_len=1, max_new=1)
        w = synth.device_weights(wl, "cuda:0")
        ctx = B.Context(B.make_config(shape, max_batch=Bn, max_ctx=L + q + 32, max_block=q), w)
        B.sdsat_set_cache_len(ctx.handle, np.full(Bn, L, np.int32))
        qin = torch.randn(Bn * q, H * Dh, device="cuda:0")
        out = torch.empty(Bn * q, H * Dh, device="cuda:0")
        B.sdsat_profile_kernel(ctx.handle, "attention")
        timed(lambda i: B.sdsat_attention(ctx.handle, 0, Bn, q, qin, None, out), 50)
        ms, n = B.sdsat_kernel_time(ctx.handle)
        B.sdsat_profile_kernel(ctx.handle, "off")
        us = ms / max(1, n) * 1e3
        kv = 2 * Bn * H * (L + q) * Dh * 2
        res["cases"][f"attention_b8_h32_kv16384_q{q}"] = {"us": round(us, 2), "kv_bytes": kv,
                                                         "GBs": round(kv / us / 1e3, 1),
                                                         "frac_of_peak": round(kv / us / 1e3 / HBM_PEAK_GBS, 4)}
        ctx.close()
        del w
        torch.cuda.empty_cache()

    # verification over [8, 11, 32016] logits ~ N(0, 4), drafts built so that m_b = b mod 11
    shape = synth.small_shape(n_layers=1, d_model=64, n_heads=1, head_dim=64, d_ffn=64, vocab=32016,
                              n_adaptive=10, rope_base=1e4, dtype="fp32")
    wl = synth.Workload("verify", shape, seed=4, batch=8, k=10, prompt_len=1, max_new=1)
    w = synth.device_weights(wl, "cuda:0")
    ctx = B.Context(B.make_config(shape, max_batch=8, max_ctx=64, max_block=11), w)
    g = torch.Generator(device="cuda:0").manual_seed(4)
    nrot = 24   # 24 x 11.3 MB > the memory-side cache
    logits = [torch.randn(8, 11, 32016, device="cuda:0", generator=g) * 4.0 for _ in range(nrot)]
    am = logits[0].argmax(-1).to(torch.int32)
    drafts = am[:, :10].clone()
    for b in range(8):
        if b % 11 < 10:
            drafts[b, b % 11] = (drafts[b, b % 11] + 1) % 32016
    tok = torch.empty(8, 11, dtype=torch.int32, device="cuda:0")
    nacc = torch.empty(8, dtype=torch.int32, device="cuda:0")
    pos0 = torch.full((8,), 100, dtype=torch.int32, device="cuda:0")
    us_g = timed(lambda i: B.sdsat_verify_greedy(ctx.handle, 8, 11, logits[i % nrot], drafts, tok, nacc), 200)
    us_n = timed(lambda i: B.sdsat_verify_nucleus(ctx.handle, 8, 11, logits[i % nrot], drafts, 0.8, 0.95, 0, 4,
                                                  pos0, tok, nacc), 200)
    res["cases"]["verify_greedy_8x11x32016"] = {"us": round(us_g, 2)}
    res["cases"]["verify_nucleus_8x11x32016_p0.95_T0.8"] = {"us": round(us_n, 2)}
    ctx.close()
    del logits, w
    torch.cuda.empty_cache()

    # skinny GEMM X[11, 4096] . W[11008, 4096]^T (bf16 weights, fp32 output), 8 rotated packed copies
    M, K, N = 11, 4096, 11008
    wmat = (torch.randn(N, K, device="cuda:0", generator=g) * 0.02).to(torch.bfloat16)
    nb = B.sdsat_linear_packed_bytes(1, N, K)
    packs = [torch.empty(nb, dtype=torch.uint8, device="cuda:0") for _ in range(8)]
    for p_ in packs:
        B.sdsat_linear_pack(1, N, K, wmat, p_)
    x = torch.randn(M, K, device="cuda:0", generator=g)
    y = torch.empty(M, N, device="cuda:0")
    scr = torch.empty(B.sdsat_linear_scratch_bytes(M, N, K), dtype=torch.uint8, device="cuda:0")
    us_l = timed(lambda i: B.sdsat_linear(1, M, N, K, x, packs[i % 8], y, scr), 100)
    wbytes = N * K * 2
    res["cases"]["skinny_gemm_11x4096x11008"] = {
        "us": round(us_l, 2), "weight_bytes": wbytes, "GBs": round(wbytes / us_l / 1e3, 1),
        "note": "events around sdsat_linear: includes its fp32->bf16 input conversion launch"}
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="7b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--micro", action="store_true",
                    help="kernel micro-benchmarks instead of the generation step: decode attention over a "
                         "16384-token KV cache (batch 8, 32 heads x 128, q 6 and 11), verification over "
                         "[8, 11, 32016] logits, the 11 x 4096 x 11008 skinny GEMM")
    ap.add_argument("--no-ar-baseline", action="store_true")
    ap.add_argument("--no-forced", action="store_true", help="skip the full-acceptance (injected drafts) run")
    ap.add_argument("--ksweep", action="store_true", help="block and loop time for k = 0..13 (prints its own line)")
    ap.add_argument("--tree", type=int, default=1, help="draft tree width of draft step 2 (1: the chain)")
    ap.add_argument("--calibrate-copy-mb", type=int, default=0,
                    help="first run one device-to-device copy of this many MiB (a plain copy kernel of known "
                         "size, for scaling hardware traffic counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library drives the decode path on a single MI355X per "
              "process (the path would shard data-parallel over sequences; there is no multi-GPU run)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2403_18647_amd import binding as B
    from paper_2403_18647_amd import synth

    if args.micro:
        print(json.dumps(micro(B, synth)), flush=True)
        return
    wl = synth.workload(args.workload)
    sh = wl.shape
    q = wl.k + 1
    torch.cuda.set_device(0)
    if args.calibrate_copy_mb:
        n = args.calibrate_copy_mb << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {n} bytes device to device")
        del src, dst
    t0 = time.time()
    weights = synth.device_weights(wl, "cuda:0")
    torch.cuda.synchronize()
    log(f"weights generated and resident ({time.time() - t0:.1f}s)")
    max_ctx = wl.prompt_len + wl.max_new + 2 * q + 32
    cfg = B.make_config(sh, max_batch=wl.batch, max_ctx=max_ctx, max_block=max(q, min(1024, wl.prompt_len)))
    ctx = B.Context(cfg, weights)
    torch.cuda.synchronize()
    log(f"context ready (workspace {ctx.workspace.numel() / 2**30:.2f} GiB)")
    prompts = synth.prompts(wl)
    ad = synth.adaptive_ids(sh, wl.k)
    mode = B.MODE_NUCLEUS if wl.mode == "nucleus" else B.MODE_GREEDY
    if args.ksweep:
        print(json.dumps(ksweep(B, synth, ctx, wl, prompts)), flush=True)
        return

    def step():
        return B.sdsat_generate(ctx.handle, prompts, wl.max_new, wl.k, ad, mode=mode,
                                temperature=wl.temperature if mode else 0.0, top_p=wl.top_p, top_k=wl.top_k,
                                seed=wl.seed, width=args.tree)

    for i in range(args.warmup):
        out, st = step()
        log(f"warmup {i + 1}/{args.warmup}: {st['decode_ms']:.1f} ms decode, loops={st['loops']}")

    # the block forward is timed live in the timed steps: every BLOCK_PERIOD-th block forward (draft and
    # verify blocks) carries a pair of HIP events on the library stream (a few microseconds of queue time
    # per pair, so the period keeps the timed steps undisturbed)
    B.sdsat_profile_kernel(ctx.handle, "block", BLOCK_PERIOD)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    stats = []
    for i in range(args.steps):
        out, st = step()
        stats.append(st)
        log(f"step {i + 1}/{args.steps}: {st['prefill_ms'] + st['decode_ms']:.1f} ms, loops={st['loops']}")
    torch.cuda.synchronize()
    t_total = time.perf_counter() - t_start
    blk_samples = B.sdsat_kernel_samples(ctx.handle)
    B.sdsat_profile_kernel(ctx.handle, "off")

    new_tokens = wl.max_new * wl.batch * args.steps
    value = new_tokens / t_total
    loops = sum(s["loops"] for s in stats)
    accepted = sum(s["accepted"] for s in stats)
    m_bar = accepted / max(1, loops * wl.batch)
    decode_ms = sum(s["decode_ms"] for s in stats) / args.steps
    prefill_ms = sum(s["prefill_ms"] for s in stats) / args.steps

    # the dominant kernel (gate/up GEMM) in one more step: events from the kernel's own dispatch on every
    # launch (the interval a kernel trace reports)
    B.sdsat_profile_kernel(ctx.handle, "gateup")
    step()
    gu_ms, gu_n = B.sdsat_kernel_time(ctx.handle)
    B.sdsat_profile_kernel(ctx.handle, "off")
    blk_ms, blk_n = sum(blk_samples), len(blk_samples)
    per_block_ms = blk_ms / max(1, blk_n)
    avg_ctx = wl.prompt_len - 1 + wl.max_new / 2.0      # mean committed length over the decode
    bblk = block_bytes(sh, wl.batch, q, avg_ctx)
    blk_gbs = bblk / (per_block_ms / 1e3) / 1e9

    # in-library autoregressive baseline: the same kernels with k = 0 (one token per block forward)
    ar = None
    if not args.no_ar_baseline:
        t0 = time.perf_counter()
        _, st_ar = B.sdsat_generate(ctx.handle, prompts, wl.max_new, 0, ad, mode=mode,
                                    temperature=wl.temperature if mode else 0.0, top_p=wl.top_p, top_k=wl.top_k,
                                    seed=wl.seed)
        torch.cuda.synchronize()
        t_ar = time.perf_counter() - t0
        ar = {"tokens_per_s": round(wl.max_new * wl.batch / t_ar, 3),
              "decode_tokens_per_s": round(wl.max_new * wl.batch / (st_ar["decode_ms"] / 1e3), 3),
              "speedup_of_sdsat": round(value / (wl.max_new * wl.batch / t_ar), 4)}
    loop_ms = decode_ms / max(1.0, loops / args.steps)

    # full acceptance, measured (synthetic): every draft step 2 takes its drafts from the autoregressive
    # continuation of the same prompts, which verification accepts in full (m = k, k + 2 tokens per loop)
    forced = None
    if not args.no_forced and wl.k > 0 and args.tree == 1:
        kw = dict(mode=mode, temperature=wl.temperature if mode else 0.0, top_p=wl.top_p, top_k=wl.top_k,
                  seed=wl.seed)
        ref, _ = B.sdsat_generate(ctx.handle, prompts, wl.max_new + wl.k + 1, 0, ad, **kw)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        out_f, st_f = B.sdsat_generate(ctx.handle, prompts, wl.max_new, wl.k, ad, ref=ref, **kw)
        torch.cuda.synchronize()
        t_f = time.perf_counter() - t0
        f_tps = wl.max_new * wl.batch / t_f
        forced = {"tokens_per_s": round(f_tps, 3),
                  "decode_tokens_per_s": round(wl.max_new * wl.batch / (st_f["decode_ms"] / 1e3), 3),
                  "loops": st_f["loops"], "m_bar": round(st_f["accepted"] / max(1, st_f["loops"] * wl.batch), 4),
                  "loop_ms": round(st_f["decode_ms"] / max(1, st_f["loops"]), 4),
                  "tokens_equal_ar": bool(np.array_equal(out_f, ref[:, :wl.max_new])),
                  "speedup_vs_ar": round(f_tps / ar["tokens_per_s"], 4) if ar else None,
                  "note": "synthetic: drafts injected from the autoregressive output (sdsat_generate_forced); "
                          "measures the loop at full acceptance on random weights"}

    stream_gbs = stream_read_peak(B, torch)
    log(f"stream read: {stream_gbs:.0f} GB/s")

    M_rows = wl.batch * q
    gu_avg_s = gu_ms / max(1, gu_n) / 1e3
    gu_bytes = gateup_bytes(sh, M_rows)
    achieved = gu_bytes / gu_avg_s / 1e9 if gu_avg_s > 0 else 0.0

    result = {
        "metric": metric_for(wl),
        "value": round(value, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_total / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if sh.dtype == "bf16" else "fp32",
        "data": "synthetic (random-init weights N(0,0.02) seed %d, uniform random prompt ids)" % wl.seed,
        "config": {"workload": f"{wl.name}: {model_name(sh)}-shaped decoder ({sh.n_layers} layers, d {sh.d_model}, "
                               f"{sh.n_heads} heads x {sh.head_dim}, FFN {sh.d_ffn}, vocab {sh.vocab}+{sh.n_adaptive}), "
                               f"{sh.dtype}, batch {wl.batch}, prompt {wl.prompt_len}, {wl.max_new} new tokens, "
                               f"{wl.mode} SDSAT k={wl.k}"
                               + (f" (T {wl.temperature}, top-p {wl.top_p}, top-k {wl.top_k or 'off'})"
                                  if wl.mode == "nucleus" else "")
                               + (f", draft tree width {args.tree}" if args.tree > 1 else ""),
                   "global_batch": wl.batch, "seq_len": wl.prompt_len + wl.max_new, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm",
                     "kernel": "block forward: all kernels of one draft or verify block (embed .. LM head, "
                               "M=%d rows)" % M_rows,
                     "achieved": round(blk_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(blk_gbs / HBM_PEAK_GBS, 4), "traffic": profiled_block_traffic(wl.name),
                     "bytes_per_launch": int(bblk), "avg_launch_us": round(per_block_ms * 1e3, 2),
                     "launches": blk_n,
                     "dominant_kernel": {"kernel": "gate/up GEMM + SwiGLU (M=%d)" % M_rows,
                                         "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                         "frac": round(achieved / HBM_PEAK_GBS, 4),
                                         "traffic": profiled_traffic(wl.name), "bytes_per_launch": gu_bytes,
                                         "avg_launch_us": round(gu_avg_s * 1e6, 3), "launches": gu_n}},
        "decode": {"tokens_per_s": round(wl.max_new * wl.batch / (decode_ms / 1e3), 3),
                   "decode_ms": round(decode_ms, 3), "prefill_ms": round(prefill_ms, 3),
                   "loops_per_step": loops / args.steps, "m_bar": round(m_bar, 4),
                   "accept_rate": round(m_bar / wl.k, 4) if wl.k else 0.0,
                   "tokens_per_loop": round(m_bar + 2, 4),
                   "accept_hist": [sum(s["accept_hist"][j] for s in stats) for j in range(wl.k + 1)],
                   "loop_ms": round(loop_ms, 4),
                   "projected_tokens_per_s_full_accept": round((wl.k + 2) * wl.batch / (loop_ms / 1e3), 1),
                   "projection_note": "m = k every loop: k+2 tokens per measured loop time (the loop's work "
                                      "does not depend on m); random-init drafts accept nothing"},
        "ar_baseline": ar,
        "full_accept": forced,
        "block_forward": {"avg_ms": round(per_block_ms, 4), "blocks": blk_n,
                          "p50_ms": round(float(np.percentile(blk_samples, 50)), 4) if blk_samples else None,
                          "p90_ms": round(float(np.percentile(blk_samples, 90)), 4) if blk_samples else None,
                          "algorithmic_bytes": int(bblk), "achieved_GBs": round(blk_gbs, 1),
                          "frac_of_peak": round(blk_gbs / HBM_PEAK_GBS, 4),
                          "frac_of_stream_read": round(blk_gbs / stream_gbs, 4),
                          "note": "HIP events around every %d-th draft/verify block forward (embed..LM head) "
                                  "of the timed steps; bytes at the mean decode context" % BLOCK_PERIOD},
        "stream_read": {"GBs": round(stream_gbs, 1), "frac_of_peak": round(stream_gbs / HBM_PEAK_GBS, 4),
                        "note": "achievable HBM read rate: sdsat_stream_read (16 KiB per workgroup, 16-byte "
                                "nontemporal loads) over rotating 1 GiB regions, median of 12 launches"},
    }
    result["roofline"]["frac_of_stream_read"] = round(blk_gbs / stream_gbs, 4)
    result["roofline"]["dominant_kernel"]["frac_of_stream_read"] = round(achieved / stream_gbs, 4)
    if not args.no_cpu_baseline:
        log("cpu baseline: timing the oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(wl, m_bar)
    ctx.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
