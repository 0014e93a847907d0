"""Benchmark of the split-head vocabulary projection on one MI355X.

One step = one pass of the whole hot path over one batch: sph_cloud_partial
(gathered partial logits, clip, per-row int8) then sph_fuse_verify (endpoint
partial, dequantise + fuse + mask, greedy select, accepted draft prefix).

Default workload: single-session decode, d=4096, d_end=256, V=128256, a
49152-id language subset (one block of 32768 ids plus 16384 scattered ids),
1 session x 5 rows (k=4 drafts), bf16 h/W, clip 30, int8 payload with one
scale per row (--bits / --block choose another payload format).

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
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "cloud_gemv_decode_traffic.txt")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default="decode")
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
    p.add_argument("--sweep", choices=("d_end", "subset", "drafts", "all"), default=None,
                   help="paper-shape sweeps of the decode step instead of the benchmark line: "
                        "hidden 4096, vocabulary 150000, one session; d_end in "
                        "{48,96,128,256,512}, subset 30/40/100%% of V, drafts k in {1,2,4,5,6,8}; "
                        "one JSON line per point")
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


def attainable_peaks(dev):
    """Attainable peaks measured in this job (best of 5 each):
    - read_gbs: the library's streaming-read probe over 1 GiB (16-byte
      non-temporal loads, as the skinny projection reads weight rows);
    - mfma_bf16_tflops: the library's MFMA probe (32x32x16 bf16 loop on random
      operands that change every iteration);
    - copy_gbs: a 1 GiB device copy (bytes read + written), vendor kernel;
    - gemm_bf16_tflops: an 8192^3 bf16 GEMM on N(0,1) data, vendor library."""
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
    return {"read_gbs": read_gbs, "mfma_bf16_tflops": mfma_tflops, "copy_gbs": copy_gbs,
            "gemm_bf16_tflops": gemm_tflops}


def source_digest():
    h = hashlib.sha256()
    for name in ("gemv.hip", "sph_internal.h"):
        with open(os.path.join(ROOT, "paper_2607_13093_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(digest):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source; else None."""
    try:
        kv = {}
        with open(TRAFFIC_PROFILE) as f:
            for line in f:
                if ":" in line:
                    k, v = line.split(":", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("kernel_source_sha256_16") != digest:
            return None
        return float(kv["hbm_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


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


def main():
    args = parse()
    if args.sweep:
        if args.gpus != 1:
            print("bench.py runs on one GPU only", file=sys.stderr)
            sys.exit(2)
        sweep(args)
        return
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2607_13093_amd as sph
    from synth import CONFIGS, make_drafts, make_workload

    cfg = CONFIGS[args.workload]
    wl = make_workload(cfg)
    n = len(wl.subset)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

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

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream(dev)

    def timed_loop():
        t_start = torch.cuda.Event(enable_timing=True)
        t_stop = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t_start.record(stream)
        for i in range(args.steps):
            step(i)
        t_stop.record(stream)
        torch.cuda.synchronize()
        return t_start.elapsed_time(t_stop) / args.steps

    # Timed region: K steps, no instrumentation.
    ms_step = timed_loop()
    if args.seal and int(okm.min()) != 1:
        raise SystemExit("sealed payload rows failed authentication")
    # Kernel durations: the same K steps again with the library's trace on
    # (HIP events recorded on the launch stream around every kernel).
    cap = 16 * args.steps + 16
    sph.trace_start(cap)
    ms_step_traced = timed_loop()
    recs = sph.trace_collect(cap)

    by = {}
    for name, ms in recs:
        by.setdefault(name, []).append(ms)
    if "cloud_mfma" in by:
        kern = "cloud_mfma"
        k_ms = float(np.mean(by[kern]))
        flops = 2.0 * M * n * cfg.d_cloud
        achieved = flops / (k_ms * 1e-3) / 1e12
        roof = {"kernel": kern, "bound": "mfma", "achieved": achieved,
                "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / MFMA_BF16_PEAK_TFLOPS, "traffic": None,
                "algorithmic_flops_per_launch": flops,
                "algorithmic_bytes_per_launch": algorithmic_bytes(cfg, n), "avg_launch_ms": k_ms}
    else:
        kern = "cloud_gemv"
        k_ms = float(np.mean(by[kern]))
        nbytes = algorithmic_bytes(cfg, n)
        achieved = nbytes / (k_ms * 1e-3) / 1e9
        digest = source_digest()
        roof = {"kernel": kern, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                "traffic": read_traffic(digest) if args.workload == "decode" else None,
                "algorithmic_bytes_per_launch": nbytes, "avg_launch_ms": k_ms,
                "kernel_source_sha256_16": digest}

    att = attainable_peaks(dev)
    att_peak = att["read_gbs"] if roof["bound"] == "hbm" else att["mfma_bf16_tflops"]
    roof["attainable_peak"] = att_peak
    roof["frac_attainable"] = roof["achieved"] / att_peak

    out = {
        "metric": "split-head rows*vocab/s",
        "value": M * n / (ms_step * 1e-3),
        "unit": "rows*vocab/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{cfg.name}: d={cfg.d} d_end={cfg.d_end} V={cfg.vocab} |S|={n} "
                        f"sessions={cfg.sessions} rows={cfg.rows_per_session} {cfg.wtype} "
                        f"{cfg.mode} clip={cfg.clip_c}",
            "rows": M,
            "subset": n,
            "payload": f"b={bits} " + ("one scale per row" if block == 0 else
                                       f"one scale per {block} positions"),
            "payload_bytes_per_row": code_bytes + 4 * nb,
            "hidden_state": "int8 codes + fp32 scale per row" if args.hidden_int8 else "bf16",
            "sealed": "AES-128-GCM, one message per row (codes, then scales)" if args.seal else "no",
        },
        "roofline": roof,
        "attainable": att,
        "kernels_ms": {k: float(np.mean(v)) for k, v in by.items()},
        # kernel time of each call per step (the cloud call's and the endpoint
        # call's kernels; launch gaps excluded) and of the pair
        "calls_ms": {
            "cloud": float(sum(np.mean(v) for k, v in by.items() if k.startswith("cloud_"))),
            "endpoint": float(sum(np.mean(v) for k, v in by.items() if k.startswith("fuse_"))),
            "pair": float(sum(np.mean(v) for k, v in by.items()
                              if k.startswith("cloud_") or k.startswith("fuse_"))),
        },
        "ms_per_step_traced": ms_step_traced,
    }
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
