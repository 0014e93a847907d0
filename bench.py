"""Benchmark of the split-head vocabulary projection on one MI355X.

One step = one pass of the whole hot path over one batch: sph_cloud_partial
(gathered partial logits, clip, per-row int8) then sph_fuse_verify (endpoint
partial, dequantise + fuse + mask, greedy select or temperature + top-p
sample, accepted draft prefix).

Headline workload (default): the largest configuration, dense large-M with
the full vocabulary: d=8192, d_end=512, V=128256, every id kept (no mask),
256 sessions x 8 rows (k=7 drafts) = 2048 rows, bf16 h/W, clip 30, int8
payload with one scale per row (--bits / --block choose another payload
format).  The cloud projection is MFMA bound there.  The other workloads
(dense subset, batched verify, sampling with fp8 weights, single-session
decode, tiny) run after it in the same job and are reported under
"configs" (--workload picks another headline, --others none skips them).

Prints ONE JSON line.  `value` is rows*vocab/s = M*|S| / (seconds per step)
with every input resident in HBM before the timed region; three copies of
the weights are rotated from step to step so the gathered rows stream from
HBM rather than from the 256 MB last-level cache.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16; fp8 weights are widened to bf16 before the MFMA
N_COPIES = 3
PROFILES = os.path.join(ROOT, "profiles")
# workloads reported after the headline one, in this order
OTHER_WORKLOADS = ("dense_sub", "batched", "sample_fp8", "decode", "tiny")
# the kernel source files each traced kernel is built from (for the counter
# summaries' source digests)
KERNEL_SOURCES = {"cloud_gemv": ("gemv.hip", "sph_internal.h"),
                  "cloud_mfma": ("mfma.hip", "sph_internal.h")}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default="dense_full")
    p.add_argument("--others", choices=("all", "none"), default="all",
                   help="also time every other workload (fewer steps) and report it under "
                        "'configs'")
    p.add_argument("--bits", type=int, default=8, choices=(4, 8),
                   help="payload code width b (eq. 18)")
    p.add_argument("--block", type=int, default=0,
                   help="payload scale block: 0 = one scale per row, else 256..4096 positions")
    p.add_argument("--seal", action="store_true",
                   help="seal the payload (codes and scales) with AES-GCM after the cloud call and "
                        "open it before the endpoint call (eq. 19)")
    p.add_argument("--hidden-int8", action="store_true",
                   help="the cloud also quantises the whole hidden row to int8 codes and the "
                        "endpoint projects from them (sph_hidden_quantize + sph_fuse_verify_hq)")
    p.add_argument("--cpu-seconds", type=float, default=10.0,
                   help="bound on the oracle's CPU baseline run (0 to skip)")
    p.add_argument("--sweep", choices=("d_end", "subset", "drafts", "all", "layout"), default=None,
                   help="paper-shape sweeps of the decode step instead of the benchmark line: "
                        "hidden 4096, vocabulary 150000, one session; d_end in "
                        "{48,96,128,256,512}, subset 30/40/100%% of V, drafts k in {1,2,4,5,6,8}; "
                        "'layout': the decode shape with its 49152 ids as one contiguous run, as "
                        "the workload's run plus scattered ids, and all scattered; one JSON line "
                        "per point")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run plain device copies of MIB MiB (to scale rocprofv3 "
                        "FETCH_SIZE / WRITE_SIZE counters), then exit")
    return p.parse_args()


def copy_calibration(mib):
    import torch
    src = torch.empty(mib << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": mib << 20, "copies": 5}), flush=True)


def algorithmic_bytes(cfg, n):
    """Algorithmic HBM bytes of one cloud projection launch (all M rows):
    every gathered weight row once, its id, and the rows of h_cloud."""
    wbytes = 2 if cfg.wtype == "bf16" else 1
    per_id = cfg.d_cloud * wbytes + 4 + (4 if cfg.wtype == "fp8" else 0)
    return n * per_id + cfg.M * cfg.d_cloud * 2


def attainable_peaks(dev, same_shape=None):
    """Attainable peaks measured in this job (best of 5 each):
    - read_gbs: the library's streaming-read probe over 1 GiB (16-byte
      non-temporal loads, as the skinny projection reads weight rows);
    - mfma_bf16_tflops: the library's MFMA probe (32x32x16 bf16 loop on random
      operands that change every iteration);
    - copy_gbs: a 1 GiB device copy (bytes read + written), vendor kernel;
    - gemm_bf16_tflops: an 8192^3 bf16 GEMM on N(0,1) data, vendor library;
    - with same_shape = (M, K, N): gemm_bf16_same_shape_tflops, the vendor
      library's bf16 h @ W^T (bf16 output) on the projection's own shape, for
      scale (the projection writes fp32 partials and row maxima as well)."""
    import torch

    import paper_2607_13093_amd as sph

    def best_ms(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            best = min(best, a.elapsed_time(b))
        return best

    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    nbytes = 1 << 30
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    read_gbs = nbytes / (best_ms(lambda: sph.probe_read(src, sink)) * 1e-3) / 1e9
    copy_gbs = 2 * nbytes / (best_ms(lambda: dst.copy_(src)) * 1e-3) / 1e9
    del src, dst
    iters = 20000
    flops = sph.probe_mfma(iters, sink)
    mfma_tflops = flops / (best_ms(lambda: sph.probe_mfma(iters, sink)) * 1e-3) / 1e12
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    n = 8192
    a = torch.randn((n, n), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    b = torch.randn((n, n), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    gemm_tflops = 2.0 * n ** 3 / (best_ms(lambda: torch.matmul(a, b)) * 1e-3) / 1e12
    del a, b
    torch.cuda.empty_cache()
    out = {"read_gbs": read_gbs, "mfma_bf16_tflops": mfma_tflops, "copy_gbs": copy_gbs,
           "gemm_bf16_tflops": gemm_tflops}
    if same_shape is not None:
        m, k, nn = same_shape
        a = torch.randn((m, k), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
        b = (torch.randn((nn, k), generator=g, device=dev, dtype=torch.float32) / k ** 0.5).to(torch.bfloat16)
        ms = best_ms(lambda: torch.nn.functional.linear(a, b))
        out["gemm_bf16_same_shape"] = f"{m} x {k} x {nn}"
        out["gemm_bf16_same_shape_ms"] = ms
        out["gemm_bf16_same_shape_tflops"] = 2.0 * m * k * nn / (ms * 1e-3) / 1e12
        del a, b
        torch.cuda.empty_cache()
    return out


def source_digest(kernel):
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2607_13093_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(kernel, workload, digest):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    rocprofv3 counter summary (profiles/<kernel>_<workload>_traffic.txt), if
    it was taken on the current kernel source; else None."""
    try:
        kv = {}
        with open(os.path.join(PROFILES, f"{kernel}_{workload}_traffic.txt")) as f:
            for line in f:
                if ":" in line and not line.startswith("#"):
                    k, v = line.split(":", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("kernel_source_sha256_16") != digest:
            return None
        return float(kv["hbm_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def dtype_of(cfg):
    """Arithmetic type of the path: bf16 products with fp32 accumulation;
    fp8 weights are widened exactly to bf16 before the products."""
    return "bf16" if cfg.wtype == "bf16" else "e4m3 weights widened to bf16"


def cpu_baseline(wl, seconds):
    """The oracle, as it stands, on whole steps (one session's rows for the
    batched workloads) until `seconds` pass."""
    import numpy as np

    import oracle
    cfg = wl.cfg
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    sessions = cfg.sessions if cfg.M <= 8 else 1
    h = wl.h_bits[:sessions * cfg.rows_per_session]
    drafts = np.zeros((sessions, cfg.k), np.int32)
    reps = 0
    t0 = time.perf_counter()
    while True:
        orc = oracle.cloud_call(h, cfg.d_end, wl.subset, cfg.clip_c,
                                w_cloud_bits=wl.w_cloud_bits, w_cloud_codes=wl.w_cloud_codes,
                                w_cloud_scale=wl.w_cloud_scale, bias=wl.bias)
        oracle.endpoint_call(orc["q"], orc["scale"], h, cfg.d_end, wl.subset, wl.w_end_bits,
                             sessions, cfg.rows_per_session, drafts=drafts, mode=cfg.mode,
                             temperature=cfg.temperature, top_p=cfg.top_p, seed=cfg.philox_seed)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= seconds:
            break
    what = "whole steps" if sessions == cfg.sessions else f"steps of {sessions} session ({h.shape[0]} rows)"
    return {"value": h.shape[0] * len(wl.subset) * reps / dt, "unit": "rows*vocab/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{reps} {what} of {cfg.name} (cloud + endpoint oracle, fp64 NumPy), {dt:.1f} s"}


SWEEP_D, SWEEP_V = 4096, 150000


def sweep_points(which):
    """(d_end, subset fraction, k) of each point; defaults d_end 256, 40%, k 4."""
    pts = []
    if which in ("d_end", "all"):
        pts += [(de, 0.4, 4) for de in (48, 96, 128, 256, 512)]
    if which in ("subset", "all"):
        pts += [(256, f, 4) for f in (0.3, 0.4, 1.0)]
    if which in ("drafts", "all"):
        pts += [(256, 0.4, k) for k in (1, 2, 4, 5, 6, 8)]
    seen, out = set(), []
    for p in pts:
        if p not in seen:
            seen.add(p)
            out.append(p)
    return out


def sweep(args):
    """Decode-step sweeps at the paper's shapes (Table 6: d_end; the language
    subset fraction; Table 7: draft length).  Weights, hidden states and
    subsets are seeded synthetic data generated on the device; every point
    runs the whole step (cloud call + endpoint call, greedy) on rotated
    weight copies, like the benchmark."""
    import numpy as np
    import torch

    import paper_2607_13093_amd as sph

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    g = torch.Generator(device=dev)
    g.manual_seed(2607)
    w = []
    for _ in range(N_COPIES):
        t = torch.randn((SWEEP_V, SWEEP_D), generator=g, device=dev, dtype=torch.float32)
        w.append((t * (1.0 / SWEEP_D ** 0.5)).to(torch.bfloat16))
        del t
    rng = np.random.default_rng(2607)
    full_perm = rng.permutation(SWEEP_V)
    for de, frac, k in sweep_points(args.sweep):
        M = k + 1
        n = int(round(frac * SWEEP_V))
        ids = np.sort(full_perm[:n]).astype(np.int32)
        sub = sph.Subset(vocab=SWEEP_V, full=True) if n == SWEEP_V else sph.Subset(ids, vocab=SWEEP_V)
        h = torch.randn((M, SWEEP_D), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
        q = torch.empty((M, n), dtype=torch.int8, device=dev)
        sc = torch.empty((M,), dtype=torch.float32, device=dev)
        tok = torch.empty((M,), dtype=torch.int32, device=dev)
        acc = torch.empty((1,), dtype=torch.int32, device=dev)
        ws_c = torch.empty(max(1, sph.cloud_partial_workspace(M, sub)), dtype=torch.uint8, device=dev)
        ws_f = torch.empty(max(1, sph.fuse_verify_workspace(M, sub, sph.GREEDY)), dtype=torch.uint8, device=dev)
        drafts = torch.from_numpy(rng.choice(ids if n < SWEEP_V else np.arange(SWEEP_V, dtype=np.int32),
                                             size=(1, k)).astype(np.int32)).to(dev)

        def step(i):
            c = i % N_COPIES
            sph.cloud_partial(h[:, de:], w[c][:, de:], sub, 30.0, workspace=ws_c, out=(q, sc, None))
            sph.fuse_verify(q, sc, h[:, :de], w[c][:, :de], sub, 1, M, drafts, workspace=ws_f,
                            out=(tok, acc, None))

        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream(dev)
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for i in range(args.steps):
            step(i)
        t1.record(stream)
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / args.steps
        cap = 16 * args.steps + 16
        sph.trace_start(cap)
        for i in range(args.steps):
            step(i)
        torch.cuda.synchronize()
        by = {}
        for name, kms in sph.trace_collect(cap):
            by.setdefault(name, []).append(kms)
        kern = {kk: float(np.mean(v)) * 1e3 for kk, v in by.items()}
        dc = SWEEP_D - de
        cloud_bytes = n * (dc * 2 + 4) + M * dc * 2
        ck = kern.get("cloud_gemv", kern.get("cloud_mfma"))
        print(json.dumps({
            "sweep": args.sweep, "d": SWEEP_D, "vocab": SWEEP_V, "d_end": de, "subset": n,
            "subset_frac": frac, "k": k, "rows": M, "ms_per_step": ms,
            "rows_vocab_per_s": M * n / (ms * 1e-3), "kernels_us": kern,
            "cloud_hbm_frac": cloud_bytes / (ck * 1e-6) / 1e9 / HBM_PEAK_GBS if ck else None,
            "payload_bytes_per_row": n + 4}), flush=True)
        sub.close()


def progress(msg):
    """A progress line on stderr (stdout carries only the JSON result)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def run_workload(wl, args, steps, warmup):
    """Upload one workload, time `steps` steps (after `warmup`), then the same
    steps again with the library's kernel trace on.  Returns the results and
    frees the device tensors."""
    import numpy as np
    import torch

    import paper_2607_13093_amd as sph
    from synth import make_drafts

    cfg = wl.cfg
    n = len(wl.subset)
    dev = torch.device("cuda:0")
    progress(f"{cfg.name}: upload, {warmup} warm-up and {steps} timed steps")

    def up(a, dt=None):
        t = torch.from_numpy(np.ascontiguousarray(a))
        return (t.view(dt) if dt is not None else t).to(dev)

    h = up(wl.h_bits.view(np.int16), torch.bfloat16)
    if cfg.wtype == "bf16":
        wc = [up(wl.w_cloud_bits.view(np.int16), torch.bfloat16) for _ in range(N_COPIES)]
        wsc = None
    else:
        wc = [up(wl.w_cloud_codes, torch.uint8) for _ in range(N_COPIES)]
        wsc = up(wl.w_cloud_scale)
    we = [up(wl.w_end_bits.view(np.int16), torch.bfloat16) for _ in range(N_COPIES)]
    sub = sph.Subset(vocab=cfg.vocab, full=True) if wl.full_vocab else sph.Subset(wl.subset, vocab=cfg.vocab)
    mode = sph.GREEDY if cfg.mode == "greedy" else sph.SAMPLE
    M, de = cfg.M, cfg.d_end
    h_c, h_e = h[:, de:], h[:, :de]
    bits, block = args.bits, args.block
    code_bytes = sph.payload_code_bytes(n, bits)
    nb = sph.payload_scale_count(n, block)
    if code_bytes < 0 or nb < 0:
        raise SystemExit(f"unsupported payload format bits={bits} block={block}")
    q = torch.empty((M, code_bytes), dtype=torch.int8 if bits == 8 else torch.uint8, device=dev)
    s = torch.empty((M,) if block == 0 else (M, nb), dtype=torch.float32, device=dev)
    tok = torch.empty((M,), dtype=torch.int32, device=dev)
    acc = torch.empty((cfg.sessions,), dtype=torch.int32, device=dev)
    ws_c = torch.empty(max(1, sph.cloud_partial_workspace(M, sub)), dtype=torch.uint8, device=dev)
    ws_f = torch.empty(max(1, sph.fuse_verify_workspace(M, sub, mode)), dtype=torch.uint8, device=dev)
    if args.seal:
        # one message per payload row: its codes, then its scales
        gkey = sph.GcmKey(bytes(range(16)))
        s_bytes = s.view(torch.uint8).reshape(M, -1)
        iv = torch.zeros((M, 12), dtype=torch.uint8, device=dev)
        rows_idx = torch.arange(M, device=dev)
        iv[:, 9] = (rows_idx >> 16).to(torch.uint8)        # row number, big-endian, in the last 3 bytes
        iv[:, 10] = ((rows_idx >> 8) & 255).to(torch.uint8)
        iv[:, 11] = (rows_idx & 255).to(torch.uint8)
        aad = torch.zeros((M, 16), dtype=torch.uint8, device=dev)
        cq = torch.empty_like(q, dtype=torch.uint8)
        cs = torch.empty_like(s_bytes)
        tg = torch.empty((M, 16), dtype=torch.uint8, device=dev)
        okm = torch.empty((M,), dtype=torch.int32, device=dev)
        msg_bytes = q.shape[1] * q.element_size() + s_bytes.shape[1]
        ws_g = torch.empty(max(1, sph.gcm_workspace(M, msg_bytes)), dtype=torch.uint8, device=dev)
    hq = torch.empty((M, cfg.d), dtype=torch.int8, device=dev)
    hs = torch.empty((M,), dtype=torch.float32, device=dev)
    if args.hidden_int8:
        ws_f = torch.empty(max(1, sph.fuse_verify_hq_workspace(M, de, sub, mode)), dtype=torch.uint8,
                           device=dev)
    drafts = torch.zeros((cfg.sessions, max(cfg.k, 1)), dtype=torch.int32, device=dev)

    def step(i):
        c = i % N_COPIES
        sph.cloud_partial(h_c, wc[c], sub, cfg.clip_c, w_row_scale=wsc, workspace=ws_c,
                          out=(q, s, None), bits=bits, block=block)
        if args.seal:
            qb = q.view(torch.uint8)
            sph.gcm_seal_segments(gkey, (qb, s_bytes), iv, aad, out=(cq, cs), tag=tg, workspace=ws_g)
            sph.gcm_open_segments(gkey, (cq, cs), iv, tg, aad, out=(qb, s_bytes), ok=okm,
                                  workspace=ws_g)
        if args.hidden_int8:
            sph.hidden_quantize(h, out=(hq, hs))
            sph.fuse_verify_hq(q, s, hq, hs, de, we[c], sub, cfg.sessions, cfg.rows_per_session,
                               drafts if cfg.k else None, mode=mode, temperature=cfg.temperature,
                               top_p=cfg.top_p, seed=cfg.philox_seed, workspace=ws_f,
                               out=(tok, acc, None), bits=bits, block=block)
            return
        sph.fuse_verify(q, s, h_e, we[c], sub, cfg.sessions, cfg.rows_per_session,
                        drafts if cfg.k else None, mode=mode, temperature=cfg.temperature,
                        top_p=cfg.top_p, seed=cfg.philox_seed, workspace=ws_f,
                        out=(tok, acc, None), bits=bits, block=block)

    # drafts: a fair coin between the GPU's own token for the row and a random subset id
    step(0)
    torch.cuda.synchronize()
    if cfg.k:
        drafts.copy_(torch.from_numpy(make_drafts(cfg, tok.cpu().numpy(), wl.subset)))

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream(dev)

    def timed_loop():
        t_start = torch.cuda.Event(enable_timing=True)
        t_stop = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t_start.record(stream)
        for i in range(steps):
            step(i)
        t_stop.record(stream)
        torch.cuda.synchronize()
        return t_start.elapsed_time(t_stop) / steps

    # Timed region: K steps, no instrumentation.
    ms_step = timed_loop()
    if args.seal and int(okm.min()) != 1:
        raise SystemExit("sealed payload rows failed authentication")
    # Kernel durations: the same K steps again with the library's trace on
    # (events attached to the kernel dispatches on the launch stream).
    cap = 16 * steps + 16
    sph.trace_start(cap)
    ms_step_traced = timed_loop()
    recs = sph.trace_collect(cap)

    by = {}
    for name, ms in recs:
        by.setdefault(name, []).append(ms)
    kern = "cloud_mfma" if "cloud_mfma" in by else "cloud_gemv"
    k_ms = float(np.mean(by[kern]))
    nbytes = algorithmic_bytes(cfg, n)
    flops = 2.0 * M * n * cfg.d_cloud
    digest = source_digest(kern)
    traffic = read_traffic(kern, cfg.name, digest)
    if kern == "cloud_mfma":
        achieved = flops / (k_ms * 1e-3) / 1e12
        roof = {"kernel": kern, "bound": "mfma", "achieved": achieved,
                "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / MFMA_BF16_PEAK_TFLOPS, "traffic": traffic,
                "algorithmic_flops_per_launch": flops,
                "algorithmic_bytes_per_launch": nbytes, "avg_launch_ms": k_ms,
                "kernel_source_sha256_16": digest}
    else:
        achieved = nbytes / (k_ms * 1e-3) / 1e9
        roof = {"kernel": kern, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                "algorithmic_bytes_per_launch": nbytes, "avg_launch_ms": k_ms,
                "kernel_source_sha256_16": digest}
    # the roofline of the cloud call's dominant kernel: the slower of its byte
    # and flop times at the nominal peaks (both matter at the ridge)
    t_roof_ms = max(nbytes / (HBM_PEAK_GBS * 1e9), flops / (MFMA_BF16_PEAK_TFLOPS * 1e12)) * 1e3
    res = {
        "cfg": cfg, "n": n, "ms_step": ms_step, "ms_step_traced": ms_step_traced, "roof": roof,
        "roofline_ms": t_roof_ms, "roofline_frac": t_roof_ms / k_ms,
        "kernels_ms": {k: float(np.mean(v)) for k, v in by.items()},
        "calls_ms": {
            "cloud": float(sum(np.mean(v) for k, v in by.items() if k.startswith("cloud_"))),
            "endpoint": float(sum(np.mean(v) for k, v in by.items() if k.startswith("fuse_"))),
            "pair": float(sum(np.mean(v) for k, v in by.items()
                              if k.startswith("cloud_") or k.startswith("fuse_"))),
        },
        "payload_bytes_per_row": code_bytes + 4 * nb,
    }
    del h, wc, we, wsc, q, s, tok, acc, ws_c, ws_f, hq, hs, drafts
    sub.close()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def workload_text(cfg, n):
    return (f"{cfg.name}: d={cfg.d} d_end={cfg.d_end} V={cfg.vocab} |S|={n} "
            f"sessions={cfg.sessions} rows={cfg.rows_per_session} {cfg.wtype} "
            f"{cfg.mode} clip={cfg.clip_c}")


def sweep_layout(args):
    """The decode step's cloud projection with the same number of subset ids
    (49152 of 128256, d = 4096, d_end = 256, 5 rows) laid out as one
    contiguous run, as the decode workload's 32768-id run plus 16384
    scattered ids, and as 49152 scattered ids: whether a table of contiguous
    runs could speed up the gathered weight stream."""
    import numpy as np
    import torch

    import paper_2607_13093_amd as sph
    from synth import CONFIGS, make_workload

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = CONFIGS["decode"]
    wl = make_workload(cfg)
    n, V, de = cfg.n_sub, cfg.vocab, cfg.d_end
    rng = np.random.default_rng(2607)
    layouts = {
        "one_run": np.arange(20000, 20000 + n, dtype=np.int32),
        "run_plus_scattered": wl.subset,
        "scattered": np.sort(rng.choice(V, n, replace=False)).astype(np.int32),
    }
    h = torch.from_numpy(wl.h_bits.view(np.int16)).view(torch.bfloat16).to(dev)
    wc = [torch.from_numpy(wl.w_cloud_bits.view(np.int16)).view(torch.bfloat16).to(dev)
          for _ in range(N_COPIES)]
    M = cfg.M
    q = torch.empty((M, n), dtype=torch.int8, device=dev)
    sc = torch.empty((M,), dtype=torch.float32, device=dev)
    for name, ids in layouts.items():
        sub = sph.Subset(ids, vocab=V)
        ws = torch.empty(sph.cloud_partial_workspace(M, sub), dtype=torch.uint8, device=dev)
        for i in range(args.warmup):
            sph.cloud_partial(h[:, de:], wc[i % N_COPIES], sub, cfg.clip_c, workspace=ws, out=(q, sc, None))
        torch.cuda.synchronize()
        cap = 4 * args.steps + 16
        sph.trace_start(cap)
        for i in range(args.steps):
            sph.cloud_partial(h[:, de:], wc[i % N_COPIES], sub, cfg.clip_c, workspace=ws, out=(q, sc, None))
        torch.cuda.synchronize()
        us = [ms * 1e3 for k, ms in sph.trace_collect(cap) if k == "cloud_gemv"]
        nbytes = algorithmic_bytes(cfg, n)
        runs = int(1 + np.count_nonzero(np.diff(ids) != 1))
        print(json.dumps({"sweep": "layout", "layout": name, "ids": n, "runs": runs,
                          "cloud_gemv_us_mean": float(np.mean(us)),
                          "cloud_gemv_us_median": float(np.median(us)),
                          "hbm_frac": nbytes / (np.median(us) * 1e-6) / 1e9 / HBM_PEAK_GBS}), flush=True)
        sub.close()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the library has no "
              "multi-GPU path, and this job uses a single MI355X", file=sys.stderr)
        sys.exit(2)
    if args.sweep == "layout":
        sweep_layout(args)
        return
    if args.sweep:
        sweep(args)
        return
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return

    import torch

    from synth import CONFIGS, make_workload, with_subset

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = CONFIGS[args.workload]
    progress(f"{cfg.name}: drawing the synthetic inputs")
    wl = make_workload(cfg)
    r = run_workload(wl, args, args.steps, args.warmup)
    progress("attainable peaks")
    n = r["n"]
    roof = r["roof"]
    att = attainable_peaks(dev, (cfg.M, cfg.d - cfg.d_end, n) if roof["bound"] == "mfma" else None)
    att_peak = att["read_gbs"] if roof["bound"] == "hbm" else att["mfma_bf16_tflops"]
    roof["attainable_peak"] = att_peak
    roof["frac_attainable"] = roof["achieved"] / att_peak
    bits, block = args.bits, args.block

    out = {
        "metric": "split-head rows*vocab/s",
        "value": cfg.M * n / (r["ms_step"] * 1e-3),
        "unit": "rows*vocab/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype_of(cfg),
        "data": "synthetic",
        "config": {
            "workload": workload_text(cfg, n),
            "rows": cfg.M,
            "subset": n,
            "payload": f"b={bits} " + ("one scale per row" if block == 0 else
                                       f"one scale per {block} positions"),
            "payload_bytes_per_row": r["payload_bytes_per_row"],
            "hidden_state": "int8 codes + fp32 scale per row" if args.hidden_int8 else "bf16",
            "sealed": "AES-128-GCM, one message per row (codes, then scales)" if args.seal else "no",
        },
        "roofline": roof,
        "attainable": att,
        "kernels_ms": r["kernels_ms"],
        # kernel time of each call per step (the cloud call's and the endpoint
        # call's kernels; launch gaps excluded) and of the pair
        "calls_ms": r["calls_ms"],
        "ms_per_step_traced": r["ms_step_traced"],
    }
    if args.cpu_seconds > 0:
        progress("CPU baseline (the oracle)")
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)

    if args.others == "all":
        # every other workload, fewer steps; the dense subset reuses the dense
        # workload's hidden states and weights (same seed streams)
        configs = {}
        for name in OTHER_WORKLOADS:
            if name == args.workload:
                continue
            c2 = CONFIGS[name]
            progress(f"{name}: drawing the synthetic inputs")
            try:
                w2 = with_subset(wl, c2)
            except ValueError:
                w2 = make_workload(c2)
            r2 = run_workload(w2, args, min(args.steps, 50), min(args.warmup, 5))
            k2 = r2["roof"]["kernel"]
            configs[name] = {
                "workload": workload_text(c2, r2["n"]),
                "dtype": dtype_of(c2),
                "ms_per_step": r2["ms_step"],
                "value": c2.M * r2["n"] / (r2["ms_step"] * 1e-3),
                "unit": "rows*vocab/s",
                "dominant_kernel": k2,
                "dominant_kernel_us": r2["roof"]["avg_launch_ms"] * 1e3,
                "bound": r2["roof"]["bound"],
                "achieved": r2["roof"]["achieved"],
                "achieved_unit": r2["roof"]["unit"],
                "frac": r2["roof"]["frac"],
                "roofline_us": r2["roofline_ms"] * 1e3,
                "roofline_frac": r2["roofline_frac"],
                "traffic": r2["roof"]["traffic"],
                "kernels_ms": r2["kernels_ms"],
            }
            del w2
        out["configs"] = configs
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
