"""Benchmark: denoise steps/s and images/s at SD-XL shapes (50 DDIM steps with
classifier-free guidance, batch 1 -> UNet batch 2), on one MI355X.

A benchmark step is one image: dn_denoise over all 50 iterations from a fresh
latent (every row of the hot path: time embedding, conv_in, ResNet blocks,
transformers, down/up sampling, out head, guidance + DDIM). Inputs (random
weights ~ N(0, 1/fan_in), latent and context ~ N(0, 1)) are generated on the
device before timing. Prints one JSON line.

Extra fields: the dominant kernel's roofline (the FF-in GEGLU GEMM of the
32x32 transformer blocks, timed live with HIP events on the library's stream),
the approximate-caching k-sweep (lookup over 100,000 cached embeddings + resume
at step k), and the CPU oracle timed on a bounded sample on the host.
"""

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def kernel_source_hash():
    """sha256 over the sources of the GEMM kernel the roofline reports (so that HBM
    traffic measured with counters is only reported for the kernel it was taken on)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("gemm.hip", "gemm_frag.hip", "gemm_epilogue.h", "common.h", "kernels.h"):
        with open(os.path.join(ROOT, "paper_2511_06724_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch of the FF-in GEMM from profiles/ff_in_gemm_traffic.json
    (FETCH_SIZE + WRITE_SIZE counter passes, scaled by a plain copy of known size),
    or None when the file is missing or was taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", "ff_in_gemm_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("kernel_source_hash") != kernel_source_hash():
        return None
    return t.get("bytes_per_launch")


def unet_flops(cfg, n):
    """(conv + linear, attention) FLOPs of one UNet evaluation on n samples (2 per MAC)."""
    c0, temb = cfg.model_channels, 4 * cfg.model_channels
    H, W = cfg.latent_h, cfg.latent_w
    lin = 2 * n * (c0 * temb + temb * temb) + 2 * n * H * W * c0 * cfg.latent_c * 9
    att = 0.0
    skips = [c0]
    ch = c0

    def res(cin, cout, hw):
        f = 2 * n * hw * cout * 9 * (cin + cout) + 2 * n * temb * cout
        return f + (2 * n * hw * cout * cin if cin != cout else 0)

    def tx(c, depth, hw):
        tok = n * hw
        per = 2 * tok * c * c * 6 + 4 * n * cfg.ctx_len * cfg.ctx_dim * c + 2 * tok * c * c * 3 * cfg.ff_mult
        return 4 * tok * c * c + depth * per, depth * (4 * n * hw * hw * c + 4 * n * hw * cfg.ctx_len * c)

    L = len(cfg.levels)
    for l, (c, d, _, _) in enumerate(cfg.levels):
        for _ in range(cfg.layers_per_block):
            lin += res(ch, c, H * W)
            ch = c
            if d:
                a, b = tx(c, d, H * W)
                lin, att = lin + a, att + b
            skips.append(ch)
        if l < L - 1:
            H, W = H // 2, W // 2
            lin += 2 * n * H * W * c * c * 9
            skips.append(ch)
    c = cfg.levels[-1][0]
    lin += res(ch, c, H * W) + res(c, c, H * W)
    if cfg.mid_depth > 0:
        a, b = tx(c, cfg.mid_depth, H * W)
        lin, att = lin + a, att + b
    for l in reversed(range(L)):
        c, d, _, _ = cfg.levels[l]
        for _ in range(cfg.layers_per_block + 1):
            lin += res(ch + skips.pop(), c, H * W)
            ch = c
            if d:
                a, b = tx(c, d, H * W)
                lin, att = lin + a, att + b
        if l > 0:
            H, W = H * 2, W * 2
            lin += 2 * n * H * W * c * c * 9
    lin += 2 * n * H * W * cfg.latent_c * ch * 9
    return lin, att


def device_weights(torch, dn, cfg, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    table = dn.weight_table(cfg)
    blob = torch.empty(sum(t[0] for t in table), device="cuda")
    off = 0
    for numel, fan, kind in table:
        v = blob[off:off + numel]
        if kind in (0, 1):
            v.normal_(0.0, fan ** -0.5, generator=g)
        elif kind == 2:
            v.normal_(1.0, 0.1, generator=g)
        else:
            v.normal_(0.0, 0.1, generator=g)
        off += numel
    return blob


# Single-GEMM workloads of the 32x32 SD-XL transformer blocks (M = 2048 tokens at batch 2
# with guidance): name -> (M, N outputs, K, GEGLU, fp32 residual + fp32 output).
GEMM_CASES = {
    "ffin": (2048, 5120, 1280, True, False),    # FF-in, 2 x 5120 packed columns -> 5120 GEGLU outputs
    "proj": (2048, 1280, 1280, False, True),    # attention out-projection into the fp32 residual stream
    "qkv": (2048, 3840, 1280, False, False),    # fused Q, K, V projection (bf16 output)
    "ffout": (2048, 1280, 5120, False, True),   # FF-out into the fp32 residual stream
}


def gemm_case(torch, dn, name, stream):
    """Operands of one GEMM case and a function that launches it once on `stream`."""
    M, N, K, geglu, resid = GEMM_CASES[name]
    Nw = 2 * N if geglu else N
    x = torch.randn((M, K), device="cuda").to(torch.bfloat16)
    w = (torch.randn((Nw, K), device="cuda") / math.sqrt(K)).to(torch.bfloat16)
    b = torch.randn(Nw, device="cuda")
    r = torch.randn((M, N), device="cuda") if resid else None
    y = torch.empty((M, N), device="cuda", dtype=torch.float32 if resid else torch.bfloat16)
    w = dn.pack_weight(dn.DN_BF16, w, Nw, K)

    def launch():
        dn.op_linear(dn.DN_BF16, x, w, b, y, M, N, K, resid=r, resid_f32=resid, y_f32=resid, geglu=geglu,
                     stream=stream)
    return launch, 2.0 * M * Nw * K


def roofline_ff_in(torch, dn, stream, iters=20):
    """FF-in GEGLU GEMM of a 32x32 SD-XL transformer block: M = 2048 tokens (batch 2),
    K = 1280, 2 x 5120 packed output columns -> 5120 GEGLU outputs."""
    launch, flops = gemm_case(torch, dn, "ffin", stream)
    for _ in range(3):
        launch()
    # one event pair around each launch, on the stream the kernel runs on
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
    for e0, e1 in ev:
        e0.record(stream)
        launch()
        e1.record(stream)
    torch.cuda.synchronize()
    avg_s = sum(e0.elapsed_time(e1) for e0, e1 in ev) / 1e3 / iters
    achieved = flops / avg_s / 1e12
    return {"kernel": "gemm_frag_kernel<bf16,128x256> FF-in GEGLU 2048x10240x1280", "bound": "mfma",
            "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic(),
            "avg_launch_us": round(avg_s * 1e6, 2), "flops_per_launch": flops,
            "kernel_source_hash": kernel_source_hash()}


def profile_kernel(torch, dn, name):
    """Counter-collection mode: 23 launches of one GEMM case (GEMM_CASES), then a plain
    device copy of 256 MiB (its FETCH_SIZE / WRITE_SIZE calibrate the counters)."""
    stream = torch.cuda.current_stream()
    launch, _ = gemm_case(torch, dn, name, stream)
    for _ in range(23):
        launch()
    a = torch.empty(64 << 20, device="cuda", dtype=torch.float32).fill_(1.0)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"profile_kernel": "done", "copy_bytes": a.numel() * 4,
                      "kernel_source_hash": kernel_source_hash()}))


def lookup_timing(torch, dn, n_entries=100_000, dim=768, queries=4):
    """Nearest-prompt lookup over n_entries cached fp16 embeddings: host time of the
    synchronous call with the table resident in the last-level cache (warm) and after
    it was evicted (cold). Returns (cache, device queries, planted rows, figures)."""
    from paper_2511_06724_amd import workloads as W
    cache = torch.from_numpy(W.cache_embeddings(n_entries, dim, seed=7).view("uint16")).cuda()
    qs, rows = W.planted_queries(cache.cpu().numpy().view("float16"), queries, seed=9)
    qd = [torch.from_numpy(q.view("uint16").copy()).cuda() for q in qs]
    # warm: the 153.6 MB table stays in the 256 MB last-level cache between queries
    dn.ac_lookup(qd[0], cache)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(4):
        for q in qd:
            dn.ac_lookup(q, cache)
    t_warm = (time.perf_counter() - t0) / (4 * len(qd))
    # cold: reading 1 GiB between queries evicts the table from the 256 MB last-level
    # cache with clean lines (a write would leave dirty lines whose write-back then
    # competes with the scan)
    flush = torch.zeros(256 << 20, device="cuda", dtype=torch.float32)
    t_cold = 0.0
    for q in qd:
        flush.sum()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        dn.ac_lookup(q, cache)
        t_cold += time.perf_counter() - t0
    t_cold /= len(qd)
    # batched: 64 planted queries in one call, the table read once (matrix-core scores)
    bq, brows = W.planted_queries(cache.cpu().numpy().view("float16"), 64, seed=11)
    bqd = torch.from_numpy(bq.view("uint16").copy()).cuda()
    bidx, _ = dn.ac_lookup_batch(bqd, cache)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(4):
        dn.ac_lookup_batch(bqd, cache)
    tb_warm = (time.perf_counter() - t0) / 4
    tb_cold = 0.0
    for _ in range(4):
        flush.sum()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        dn.ac_lookup_batch(bqd, cache)
        tb_cold += time.perf_counter() - t0
    tb_cold /= 4
    del flush
    ok = all(dn.ac_lookup(q, cache)[0] == int(r) for q, r in zip(qd, rows))
    fig = {"lookup_us_per_query_warm": round(t_warm * 1e6, 1), "lookup_us_per_query_cold": round(t_cold * 1e6, 1),
           "lookup_GBps_warm": round(n_entries * dim * 2 / t_warm / 1e9, 1),
           "lookup_GBps_cold": round(n_entries * dim * 2 / t_cold / 1e9, 1),
           "lookup_note": "synchronous call timed on the host (includes the two launches and the 12-byte "
                          "result copy); the kernels alone: profiles/ac_lookup_kernels.md",
           "planted_found": ok,
           "lookup_batch64_us_warm": round(tb_warm * 1e6, 1), "lookup_batch64_us_cold": round(tb_cold * 1e6, 1),
           "lookup_batch_us_per_query_cold": round(tb_cold * 1e6 / 64, 2),
           "lookup_batch_GBps_cold": round(n_entries * dim * 2 / tb_cold / 1e9, 1),
           "lookup_batch_note": "ac_lookup_batch with 64 queries: one synchronous call, table read once",
           "lookup_batch_planted_found": [int(i) for i in bidx] == [int(r) for r in brows]}
    return cache, qd, rows, fig


def ac_sweep(torch, dn, model, cfg, ctx, ts, n_entries=100_000, dim=768, per_k=2):
    """Approximate caching: lookup + latent fetch + resume at k for 50 - k steps, per_k
    planted queries per k (each a cosine 0.8-0.95 neighbour of a random cache row)."""
    cache, qd, rows, fig = lookup_timing(torch, dn, n_entries, dim, max(4, per_k))
    if per_k > 64:
        raise ValueError("at most 64 queries per k (one batched search)")
    # cached latents: 100,000 x 4 x 128 x 128 bf16 = 13.1 GB, drawn on the device
    g = torch.Generator(device="cuda").manual_seed(8)
    lat_cache = torch.empty((n_entries, cfg.latent_c, cfg.latent_h, cfg.latent_w), device="cuda",
                            dtype=torch.bfloat16)
    for s in range(0, n_entries, 10_000):
        lat_cache[s:s + 10_000].normal_(generator=g)
    lat = torch.empty((cfg.batch, cfg.latent_c, cfg.latent_h, cfg.latent_w), device="cuda")
    out = dict(fig)
    out.update({"queries_per_k": per_k, "images_per_s_by_k": {}})
    qbatch = torch.stack(qd[:per_k])
    for k in (0, 5, 10, 15, 20, 25):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        # the k's queries in one batched search, then fetch + resume per query
        idxs, _ = dn.ac_lookup_batch(qbatch, cache)
        for idx in idxs:
            dn.ac_fetch_latent(lat_cache, idx, lat)
            model.denoise(lat, ctx, ts, k, 50 - k, 7.5)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / per_k
        out["images_per_s_by_k"][str(k)] = round(1.0 / dt, 4)
        print(f"[bench] ac k={k}: {1.0 / dt:.3f} images/s", file=sys.stderr, flush=True)
    # cache write (Sec. 4.7): a full 50-step run that stores its latents at K = 5 .. 25
    # as bf16 slots of the cache's latent table, against the same run without stores
    caps = [5, 10, 15, 20, 25]
    for store in (False, True):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(per_k):
            if store:
                model.denoise_capture(lat, ctx, ts, 0, 50, 7.5, caps, lat_cache[:len(caps)])
            else:
                model.denoise(lat, ctx, ts, 0, 50, 7.5)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / per_k
        out["cache_write_images_per_s" if store else "no_write_images_per_s"] = round(1.0 / dt, 4)
    del lat_cache
    return out


def cpu_baseline(budget_s=12.0):
    """The CPU oracle on the host cores, on a bounded sample of the SD-XL step: one
    top-level ResBlock (128x128, C = 320) and then single-block transformer stages at
    the 32x32 level (C = 1280, 20 heads x 64, batch 2 with guidance, 77x2048 context)
    until about `budget_s` seconds have passed; the FLOPs done per second are then
    scaled to a full denoise step."""
    import numpy as np
    from oracle import unet as OU
    from paper_2511_06724_amd import workloads as W
    import oracle.topology as OT

    threads = len(os.sched_getaffinity(0))
    cfg = W.sdxl()
    sub = cfg.with_(levels=((320, 0, 5, 64), (640, 0, 10, 64), (1280, 1, 20, 64)))
    rng = np.random.default_rng(0)
    Wt = {}
    for name, shape, kind, fan in OT.tensor_table(sub):
        if not (name.startswith("down2.0.tx") or name.startswith("down0.0.res")):
            continue
        if kind in ("w", "b"):
            Wt[name] = rng.standard_normal(shape, dtype=np.float32) / np.float32(math.sqrt(fan))
        elif kind == "g":
            Wt[name] = 1 + 0.1 * rng.standard_normal(shape, dtype=np.float32)
        else:
            Wt[name] = 0.1 * rng.standard_normal(shape, dtype=np.float32)
    x_tx = rng.standard_normal((2, 1280, 32, 32), dtype=np.float32)
    x_res = rng.standard_normal((2, 320, 128, 128), dtype=np.float32)
    ctx = rng.standard_normal((2, 77, 2048), dtype=np.float32)
    temb = rng.standard_normal((2, 1280), dtype=np.float32)
    hw, c, tok = 1024, 1280, 2048
    tx_flops = 4 * tok * c * c + (2 * tok * c * c * 18 + 4 * 2 * 77 * 2048 * c + 4 * 2 * hw * hw * c
                                  + 4 * 2 * hw * 77 * c)
    res_flops = 2 * 2 * 16384 * 320 * 9 * 640 + 2 * 2 * 1280 * 320
    t0 = time.perf_counter()
    OU.resblock(sub, Wt, "down0.0.res", x_res, temb)
    done, blocks = res_flops, 0
    while True:
        OU.transformer(sub, Wt, "down2.0.tx", x_tx, ctx, 1, 20)
        done += tx_flops
        blocks += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    lin, att = unet_flops(cfg, 2)
    steps_per_s = (done / dt) / (lin + att)
    return {"value": round(steps_per_s, 6), "unit": "denoise steps/s", "cores": threads, "kind": "oracle",
            "sample": (f"one SD-XL 128x128 ResBlock + {blocks} single-block 32x32 transformer stages (batch 2), "
                       f"{done / 1e12:.3f} TFLOP in {dt:.1f} s on {threads} host threads, extrapolated by FLOPs to a "
                       f"full {(lin + att) / 1e12:.3f} TFLOP denoise step"),
            "images_per_s": round(steps_per_s / 50, 8)}


def time_images(torch, model, cfg, ts, images, warmup=1):
    g = torch.Generator(device="cuda").manual_seed(0)
    x0 = torch.randn((cfg.batch, cfg.latent_c, cfg.latent_h, cfg.latent_w), device="cuda", generator=g)
    ctx = torch.randn((2 * cfg.batch, cfg.ctx_len, cfg.ctx_dim), device="cuda", generator=g)
    lat = x0.clone()
    for _ in range(warmup):
        lat.copy_(x0)
        model.denoise(lat, ctx, ts, 0, 50, 7.5)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(images):
        lat.copy_(x0)
        model.denoise(lat, ctx, ts, 0, 50, 7.5)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / images


def sweep_batch(torch, dn, W, args):
    import numpy as np
    ts = np.array([(49 - j) * 20 + 1 for j in range(50)] + [-1], np.int32)
    cases = [("sdxl", b, W.sdxl(W.DN_BF16, batch=b)) for b in (1, 2, 4, 8)]
    cases += [("sdxl_small", 1, W.sdxl_small(W.DN_BF16, batch=1))]
    for name, b, cfg in cases:
        blob = device_weights(torch, dn, cfg, seed=42)
        model = dn.Denoiser(cfg, blob)
        del blob
        torch.cuda.empty_cache()
        sec = time_images(torch, model, cfg, ts, images=max(1, args.steps // b), warmup=1)
        lin, att = unet_flops(cfg, 2 * b)
        print(json.dumps({"variant": name, "batch": b, "latency_s_per_call": round(sec, 4),
                          "images_per_s": round(b / sec, 4), "denoise_steps_per_s": round(50 / sec, 3),
                          "tflop_per_step": round((lin + att) / 1e12, 3),
                          "mfma_util": round((lin + att) * 50 / sec / 1e12 / PEAK_BF16_TFLOPS, 4)}), flush=True)
        model.close()
        torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3, help="timed images (50 denoise iterations each)")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ac", action="store_true")
    ap.add_argument("--ac-queries", type=int, default=2,
                    help="queries per k in the approximate-caching sweep (the workload names 64; 2 keeps the "
                         "default run short)")
    ap.add_argument("--profile-kernel", nargs="?", const="ffin", default=None, choices=sorted(GEMM_CASES),
                    help="only launch one GEMM of a 32x32 transformer block 23 times (default: FF-in) and a "
                         "256 MiB copy (counter collection)")
    ap.add_argument("--lookup-only", action="store_true",
                    help="only the cache lookup (100,000 x 768 fp16, warm and cold): one JSON line")
    ap.add_argument("--sweep-batch", action="store_true",
                    help="instead of the headline line: latency and images/s for batch 1, 2, 4, 8 and the "
                         "smaller variant (4 / 1 transformer blocks per 32x32 / 64x64 stage)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the denoise loop is replicated per GPU, "
              "with no exchange between GPUs; use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2511_06724_amd import dn, workloads as W

    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    if args.profile_kernel:
        profile_kernel(torch, dn, args.profile_kernel)
        return
    if args.sweep_batch:
        sweep_batch(torch, dn, W, args)
        return
    if args.lookup_only:
        print(json.dumps(lookup_timing(torch, dn)[3]))
        return
    cfg = W.sdxl(W.DN_BF16, batch=args.batch)
    print("[bench] generating SD-XL weights on the device", file=sys.stderr, flush=True)
    blob = device_weights(torch, dn, cfg, seed=42)
    model = dn.Denoiser(cfg, blob)
    del blob
    torch.cuda.empty_cache()
    g = torch.Generator(device="cuda").manual_seed(0)
    x0 = torch.randn((cfg.batch, cfg.latent_c, cfg.latent_h, cfg.latent_w), device="cuda", generator=g)
    ctx = torch.randn((2 * cfg.batch, cfg.ctx_len, cfg.ctx_dim), device="cuda", generator=g)
    from_ts = [(49 - j) * 20 + 1 for j in range(50)] + [-1]
    import numpy as np
    ts = np.array(from_ts, np.int32)
    stream = torch.cuda.current_stream()
    lat = x0.clone()
    for i in range(args.warmup):
        lat.copy_(x0)
        model.denoise(lat, ctx, ts, 0, 50, 7.5, stream=stream)
        torch.cuda.synchronize()
        print(f"[bench] warmup image {i} done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        lat.copy_(x0)
        model.denoise(lat, ctx, ts, 0, 50, 7.5, stream=stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    finite = bool(torch.isfinite(lat).all())
    images_per_s = args.steps * cfg.batch / dt
    steps_per_s = args.steps * 50 / dt
    ms_step = dt / args.steps * 1e3
    lin, att = unet_flops(cfg, 2 * cfg.batch)
    mfma_util = (lin + att) * steps_per_s / 1e12 / PEAK_BF16_TFLOPS
    print(f"[bench] {steps_per_s:.2f} denoise steps/s, {images_per_s:.3f} images/s", file=sys.stderr, flush=True)

    roof = roofline_ff_in(torch, dn, stream)
    ac = None if args.no_ac else ac_sweep(torch, dn, model, cfg, ctx, ts, per_k=args.ac_queries)
    model.close()
    cpu = None if args.no_cpu_baseline else cpu_baseline()
    out = {
        "metric": "denoise steps/sec + images/sec at SD-XL shapes (50 steps, CFG); MFMA util %",
        "value": round(steps_per_s, 3),
        "unit": "denoise steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (random weights ~N(0,1/fan_in), latent and context ~N(0,1))",
        "config": {"workload": "SD-XL-shaped UNet, latent 1x4x128x128, 50 DDIM steps, CFG 7.5 (UNet batch 2)",
                   "batch": cfg.batch, "params": int(sum(t[0] for t in dn.weight_table(cfg))),
                   "tflop_per_denoise_step": round((lin + att) / 1e12, 3)},
        "images_per_s": round(images_per_s, 4),
        "ms_per_denoise_step": round(dt / args.steps / 50 * 1e3, 3),
        "mfma_util_whole_step": round(mfma_util, 4),
        "output_finite": finite,
        "roofline": roof,
        "ac_sweep": ac,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
