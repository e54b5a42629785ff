#!/usr/bin/env python3
"""Benchmark of the gfx950 block-wise lossless float codec on one MI355X.

Workload: the 1 GiB bf16 weight-sync buffer (a 0.5B-parameter transformer's
weights, 2^29 elements, 64 KiB codec blocks; workloads.weight_sync).  One
step compresses the whole buffer (uzip_compress) and decompresses the
stream again (uzip_decompress), inputs resident in HBM.  ``value`` is the
uncompressed bytes of the buffer divided by the time of one step.  The line
also reports compress and decompress rates separately, the ratio, the HBM
roofline of the dominant kernel, a measured device-copy bandwidth, and the
other configurations: the split-send producer on the same buffer (4 MiB
chunks, host-mapped flags, with the times at which the host sees each
chunk's flags), the 4 MiB bf16 tensor (after a 512 MiB cache flush), fp32
and fp16 gradients in 256 KiB blocks, the 2 GiB KV cache in 1 MiB chunks,
the fused reduce of eight 16 MiB bf16 shares and of eight whole
[8192 x 8192] slices, the stream-wide table modes, FP8 pairs, and the CPU
oracle timed on a bounded sample on one and on all host threads.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--no-extras]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "compress & decompress GB/s (uncompressed) + ratio, % of HBM roofline, 1 GPU"
PREHEAT_MS = 100
HBM_PEAK_GBPS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_weight_sync_bf16_1GiB.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2604_17172_amd", "csrc", "uzip.hip")


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """sha256 of the kernel sources' code: comments, trailing blanks and
    empty lines removed, so that editing a comment keeps the measured
    traffic valid while any change to the code does not."""
    h = hashlib.sha256()
    for name in ("uzip.hip", "uzip_device.h"):
        with open(os.path.join(os.path.dirname(KERNEL_SRC), name)) as fh:
            text = re.sub(r"/\*.*?\*/", "", fh.read(), flags=re.S)
        for line in text.splitlines():
            line = re.sub(r"//.*", "", line).rstrip()
            if line:
                h.update(line.encode() + b"\n")
    return h.hexdigest()


def measured_traffic(kernel: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary, or None if it is missing or the kernels changed since."""
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("kernel_code_sha256") != kernel_source_hash():
        return None
    k = t.get("kernels", {}).get(kernel)
    if not k:
        return None
    return k.get("hbm_bytes_per_launch")


def frac(nbytes: float, ms: float) -> float:
    return round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)


def gbps(nbytes: float, ms: float) -> float:
    return round(nbytes / (ms * 1e-3) / 1e9, 1)


def host_threads() -> int:
    """Threads the CPU baseline may use: the CPUs this process may run on,
    capped by OMP_NUM_THREADS where the host sets it."""
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    omp = os.environ.get("OMP_NUM_THREADS", "")
    if omp.isdigit() and int(omp) > 0:
        n = min(n, int(omp))
    return max(n, 1)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="only the headline step")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a 1 GiB device copy (counter calibration under rocprofv3)")
    ap.add_argument("--fixed-preheat", action="store_true",
                    help="untimed calls by count instead of by time (a dispatch sequence that repeats "
                         "exactly from run to run, for attributing counter runs)")
    ap.add_argument("--no-reduce-full", action="store_true",
                    help="skip the fused reduce on the full-tensor reading (8 slices [8192 x 8192] bf16)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(each GPU codes its own shard and nothing is exchanged between GPUs)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import workloads as W
    import paper_2604_17172_amd as uz  # fails loudly without the HIP library

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()

    def ev():
        return torch.cuda.Event(enable_timing=True)

    open_leg = [False]

    def mark(name):
        """A roctx range per leg (rocprofv3 --marker-trace attributes the
        kernels to legs); the GPU is drained at both ends."""
        torch.cuda.synchronize()
        if open_leg[0]:
            torch.cuda.nvtx.range_pop()
        open_leg[0] = name is not None
        if name is not None:
            torch.cuda.nvtx.range_push(name)

    def timed(fn, reps, flush=None):
        """ms of each of `reps` calls of fn (HIP events on the launch stream
        around each call), after untimed calls for at least 30 ms (the clocks
        ramp up after the leg's host-side set-up); `flush` runs untimed
        before each call."""
        t0 = time.perf_counter()
        k = 0
        while True:
            fn()
            torch.cuda.synchronize()
            k += 1
            if (k >= 2) if args.fixed_preheat else (time.perf_counter() - t0 >= 0.03):
                break
        # the calls go out back to back, so the host's set-up of a call
        # overlaps the GPU work before it; the first, which starts on an idle
        # GPU and would count its own host set-up, is not kept
        pairs = []
        for _ in range(reps + 1):
            if flush is not None:
                flush()
            a, b = ev(), ev()
            a.record(stream)
            fn()
            b.record(stream)
            pairs.append((a, b))
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in pairs[1:]]

    # ---------------- workload: 1 GiB bf16 weight-sync buffer ----------------
    bb = 65536
    t0 = time.time()
    x_host = W.weight_sync()
    n = x_host.size
    nbytes = 2 * n
    log(f"[bench] generated weight_sync n={n} in {time.time() - t0:.1f}s")
    x = torch.from_numpy(x_host.view(np.int16)).to(dev)
    cap = uz.uzip_max_compressed_size(uz.BF16, n, bb)
    out = torch.empty(cap, dtype=torch.uint8, device=dev)
    ws = torch.empty(uz.uzip_workspace_size(uz.OP_COMPRESS, uz.BF16, n, bb), dtype=torch.uint8, device=dev)
    y = torch.empty_like(x)
    dws = torch.empty(uz.uzip_workspace_size(uz.OP_DECOMPRESS, uz.BF16, n, bb), dtype=torch.uint8, device=dev)

    # the size and status words are allocated once, like the buffers: the
    # timed region holds the two library calls and nothing else
    size = torch.zeros(1, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    mark("headline")

    def step():
        uz.compress(x, bb, dtype="bf16", out=out, ws=ws, size=size)
        uz.decompress(out, "bf16", n, out=y, ws=dws, status=status)

    step()
    torch.cuda.synchronize()
    total = int(size.item())
    if int(status.item()) != 0 or not torch.equal(x, y):
        log("[bench] round trip is NOT lossless")
        return 1
    # The GPU reaches its steady clocks only after ~15-20 ms of continuous
    # load (per-step times fall by ~15% over the first 15 steps after an
    # idle moment): untimed steps for at least PREHEAT_MS first, then the W
    # warmup steps, then the timed steps with no idle gap in between (the
    # results are checked after the timed loop).
    t_pre = time.perf_counter()
    pre_steps = 0
    while (pre_steps < 16) if args.fixed_preheat else (time.perf_counter() - t_pre < PREHEAT_MS * 1e-3):
        for _ in range(8):
            step()
        pre_steps += 8
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    log(f"[bench] ratio {total / nbytes:.4f}; {pre_steps} untimed steps ({PREHEAT_MS} ms) + {args.warmup} warmup")

    comp_ms, dec_ms, evs = [], [], []
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        e = [ev() for _ in range(3)]
        e[0].record(stream)
        uz.compress(x, bb, dtype="bf16", out=out, ws=ws, size=size)
        e[1].record(stream)
        uz.decompress(out, "bf16", n, out=y, ws=dws, status=status)
        e[2].record(stream)
        evs.append(e)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    if int(status.item()) != 0 or int(size.item()) != total or not torch.equal(x, y):
        log("[bench] a timed step was NOT lossless")
        return 1
    for e in evs:
        comp_ms.append(e[0].elapsed_time(e[1]))
        dec_ms.append(e[1].elapsed_time(e[2]))
    ms_per_step = 1e3 * wall / args.steps
    c_ms = float(np.mean(comp_ms))
    d_ms = float(np.mean(dec_ms))
    comp_gbps = nbytes / (c_ms * 1e-3) / 1e9
    dec_gbps = nbytes / (d_ms * 1e-3) / 1e9
    value = nbytes / (ms_per_step * 1e-3) / 1e9
    log(f"[bench] compress {c_ms:.3f} ms ({comp_gbps:.0f} GB/s)  decompress {d_ms:.3f} ms ({dec_gbps:.0f} GB/s)")

    # roofline of the dominant kernel: algorithmic HBM bytes per launch
    alg_comp = nbytes + total      # read the tensor, write the stream
    alg_dec = total + nbytes       # read the stream, write the tensor
    if c_ms >= d_ms:
        dom_ms, dom_bytes, kname = c_ms, alg_comp, "encode_kernel<bf16>"
    else:
        dom_ms, dom_bytes, kname = d_ms, alg_dec, "decode_kernel<bf16>"
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": kname, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": measured_traffic(kname),
                "algorithmic_bytes_per_launch": dom_bytes,
                "compress_frac": frac(alg_comp, c_ms), "decompress_frac": frac(alg_dec, d_ms)}

    # ---------------- measured device-copy bandwidth (1 GiB, read + write) ----------------
    mark("device_copy")
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    cp = timed(lambda: dst.copy_(src), 5)
    copy_ms = float(np.median(cp))
    copy_gbps = 2 * (1 << 30) / (copy_ms * 1e-3) / 1e9
    roofline["copy_GBps_measured"] = round(copy_gbps, 1)
    roofline["compress_frac_of_copy"] = round(alg_comp / (c_ms * 1e-3) / 1e9 / copy_gbps, 4)
    roofline["decompress_frac_of_copy"] = round(alg_dec / (d_ms * 1e-3) / 1e9 / copy_gbps, 4)
    log(f"[bench] device copy 1 GiB {copy_ms:.3f} ms ({copy_gbps:.0f} GB/s read+write)")
    if not args.calibrate_copy:
        del src, dst

    extras = {}
    if not args.no_extras:
        reps = 5
        flush_buf = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
        flush_n = [0]

        def flush():
            # a 512 MiB write evicts the 256 MB Infinity Cache
            flush_n[0] += 1
            flush_buf.fill_(flush_n[0] & 0xFF)

        # ------------- split-send producer: 4 MiB chunks, host-mapped flags -------------
        mark("chunked_weight_sync")
        cb = 4 << 20
        chunks = (nbytes + cb - 1) // cb
        flags = torch.zeros(2 * chunks, dtype=torch.int32).pin_memory()
        slot = (uz.uzip_max_compressed_size(uz.BF16, cb // 2, bb) + 255) // 256 * 256
        cout = torch.empty(slot * chunks, dtype=torch.uint8, device=dev)
        cws = torch.empty(uz.uzip_workspace_size(uz.OP_CHUNKED, uz.BF16, n, bb, cb), dtype=torch.uint8, device=dev)
        epoch = [0]

        def produce():
            epoch[0] += 1
            return uz.compress_chunked(x, bb, cb, dtype="bf16", epoch=epoch[0], flags=flags, out=cout, ws=cws)

        times = timed(produce, reps)
        assert bool((flags == epoch[0]).all())
        sizes = uz.compress_chunked(x, bb, cb, dtype="bf16", epoch=epoch[0] + 1, flags=flags, out=cout, ws=cws)[2]
        epoch[0] += 1
        torch.cuda.synchronize()
        ch_ms = float(np.mean(times))
        csize = int(sizes.sum().item())
        # the receiver's side: all 256 chunk streams decoded in one launch
        cy = torch.empty_like(x)
        cst = torch.zeros(1, dtype=torch.int32, device=dev)
        cd_times = timed(lambda: uz.uzip_decompress_chunked(cout.data_ptr(), slot, 0, chunks, uz.BF16, n, bb, cb,
                                                            cy.data_ptr(), nbytes, cst.data_ptr(),
                                                            stream.cuda_stream), reps)
        if int(cst.item()) != 0 or not torch.equal(x, cy):
            log("[bench] chunk streams did NOT decode to the input")
            return 1
        cd_ms = float(np.mean(cd_times))
        del cy
        # when the host sees each chunk's flags: RAW_READY (raw plane final,
        # sendable) and DONE (stream final), from the launch call on
        fl = flags.numpy()
        leads = []
        marks = {k: [] for k in ("raw_first", "raw_median", "raw_last", "done_first", "done_median", "done_last")}
        for _ in range(3):
            epoch[0] += 1
            e_ = epoch[0]
            t_raw = np.full(chunks, np.nan)
            t_done = np.full(chunks, np.nan)
            torch.cuda.synchronize()
            t_launch = time.perf_counter()
            uz.compress_chunked(x, bb, cb, dtype="bf16", epoch=e_, flags=flags, out=cout, ws=cws)
            while np.isnan(t_done).any() and time.perf_counter() - t_launch < 10.0:
                now = time.perf_counter()
                done = fl[1::2] == e_
                raw = fl[0::2] == e_
                t_raw[raw & np.isnan(t_raw)] = now
                t_done[done & np.isnan(t_done)] = now
            torch.cuda.synchronize()
            t_raw = 1e6 * (t_raw - t_launch)
            t_done = 1e6 * (t_done - t_launch)
            for k, v in (("raw", t_raw), ("done", t_done)):
                marks[f"{k}_first"].append(np.nanmin(v))
                marks[f"{k}_median"].append(np.nanmedian(v))
                marks[f"{k}_last"].append(np.nanmax(v))
            leads.append(np.nanmedian(t_done - t_raw))
        extras["chunked"] = {"workload": "weight_sync_bf16_1GiB", "chunk_bytes": cb, "chunks": chunks,
                             "ms": round(ch_ms, 4), "GBps": gbps(nbytes, ch_ms), "ratio": round(csize / nbytes, 4),
                             "hbm_frac": frac(nbytes + csize, ch_ms),
                             "chunks_decompress_ms": round(cd_ms, 4), "chunks_decompress_GBps": gbps(nbytes, cd_ms),
                             "chunks_decompress_frac": frac(nbytes + csize, cd_ms),
                             "flags_seen_by_host_us": {k: round(float(np.median(v)), 1) for k, v in marks.items()},
                             "raw_ready_lead_over_done_us_median": round(float(np.median(leads)), 1)}
        log(f"[bench] chunked producer {ch_ms:.3f} ms, its 256 chunk streams decoded in one launch {cd_ms:.3f} ms; "
            f"flags seen by the host (us after launch): {extras['chunked']['flags_seen_by_host_us']}")
        # the workload as defined (4 MiB chunks with ready flags, decoded by
        # the receiver) beside the whole-stream step
        roofline["split_send_compress_frac"] = extras["chunked"]["hbm_frac"]
        roofline["split_send_decompress_frac"] = extras["chunked"]["chunks_decompress_frac"]
        del cout, cws

        # ------------- 4 MiB bf16 N(0, 0.02), 64 KiB blocks (after a cache flush) -------------
        mark("normal_bf16_4MiB")
        x1h = W.normal_bf16()
        x1 = torch.from_numpy(x1h.view(np.int16)).to(dev)
        n1 = x1h.size
        o1 = torch.empty(uz.uzip_max_compressed_size(uz.BF16, n1, bb), dtype=torch.uint8, device=dev)
        w1 = torch.empty(uz.uzip_workspace_size(uz.OP_COMPRESS, uz.BF16, n1, bb), dtype=torch.uint8, device=dev)
        y1 = torch.empty_like(x1)
        s1 = uz.compress(x1, bb, dtype="bf16", out=o1, ws=w1)[1]
        torch.cuda.synchronize()
        t1 = int(s1.item())
        c_cold = timed(lambda: uz.compress(x1, bb, dtype="bf16", out=o1, ws=w1), reps, flush)
        d_cold = timed(lambda: uz.decompress(o1, "bf16", n1, out=y1, ws=dws), reps, flush)
        c_warm = timed(lambda: uz.compress(x1, bb, dtype="bf16", out=o1, ws=w1), reps)
        d_warm = timed(lambda: uz.decompress(o1, "bf16", n1, out=y1, ws=dws), reps)
        assert torch.equal(x1, y1)
        cm, dm = float(np.median(c_cold)), float(np.median(d_cold))
        extras["normal_bf16_4MiB"] = {
            "n_elems": n1, "block_bytes": bb, "ratio": round(t1 / (2 * n1), 4),
            "compress_ms_cold": round(cm, 4), "decompress_ms_cold": round(dm, 4),
            "compress_ms_warm": round(float(np.median(c_warm)), 4),
            "decompress_ms_warm": round(float(np.median(d_warm)), 4),
            "compress_GBps": gbps(2 * n1, cm), "decompress_GBps": gbps(2 * n1, dm),
            "compress_frac": frac(2 * n1 + t1, cm), "decompress_frac": frac(2 * n1 + t1, dm)}
        log(f"[bench] 4 MiB bf16: compress {cm * 1e3:.1f} us, decompress {dm * 1e3:.1f} us (cold)")
        del x1, o1, w1, y1

        # ------------- fp32 / fp16 gradients, 256 KiB blocks -------------
        for name, gen, code, e_bytes in (("grad_fp32_1GiB", W.grad_fp32, uz.FP32, 4),
                                         ("grad_fp16_512MiB", W.grad_fp16, uz.FP16, 2)):
            mark(name)
            gh = gen()
            ng = gh.size
            gt = torch.from_numpy(gh.view(np.int32 if e_bytes == 4 else np.int16)).to(dev)
            del gh
            go = torch.empty(uz.uzip_max_compressed_size(code, ng, 262144), dtype=torch.uint8, device=dev)
            gw = torch.empty(uz.uzip_workspace_size(uz.OP_COMPRESS, code, ng, 262144), dtype=torch.uint8, device=dev)
            gy = torch.empty_like(gt)
            gs = uz.compress(gt, 262144, dtype=code, out=go, ws=gw)[1]
            torch.cuda.synchronize()
            gtot = int(gs.item())
            ct = timed(lambda: uz.compress(gt, 262144, dtype=code, out=go, ws=gw), reps)
            dt = timed(lambda: uz.decompress(go, code, ng, out=gy, ws=dws), reps)
            assert torch.equal(gt, gy)
            cm, dm = float(np.mean(ct)), float(np.mean(dt))
            gb = e_bytes * ng
            extras[name] = {"n_elems": ng, "block_bytes": 262144, "ratio": round(gtot / gb, 4),
                            "compress_ms": round(cm, 4), "decompress_ms": round(dm, 4),
                            "compress_GBps": gbps(gb, cm), "decompress_GBps": gbps(gb, dm),
                            "compress_frac": frac(gb + gtot, cm), "decompress_frac": frac(gb + gtot, dm)}
            log(f"[bench] {name}: ratio {gtot / gb:.4f} compress {cm:.3f} ms decompress {dm:.3f} ms")
            del gt, go, gw, gy

        # ------------- the 1 GiB weight buffer in 1 MiB and 4 MiB blocks -------------
        # (few, long blocks: each is one wave's serial chain)
        for lb in (1 << 20, 1 << 22):
            lname = f"weight_sync_bf16_1GiB_{lb >> 20}MiB_blocks"
            mark(lname)
            lo = torch.empty(uz.uzip_max_compressed_size(uz.BF16, n, lb), dtype=torch.uint8, device=dev)
            lw = torch.empty(uz.uzip_workspace_size(uz.OP_COMPRESS, uz.BF16, n, lb), dtype=torch.uint8, device=dev)
            ly = torch.empty_like(x)
            ltot = int(uz.compress(x, lb, dtype=uz.BF16, out=lo, ws=lw)[1].item())
            lreps = max(2, reps // 2)
            ct = timed(lambda: uz.compress(x, lb, dtype=uz.BF16, out=lo, ws=lw), lreps)
            dt = timed(lambda: uz.decompress(lo, uz.BF16, n, out=ly, ws=dws), lreps)
            assert torch.equal(x, ly)
            cm, dm = float(np.mean(ct)), float(np.mean(dt))
            extras[lname] = {"block_bytes": lb, "ratio": round(ltot / nbytes, 4),
                             "compress_ms": round(cm, 4), "decompress_ms": round(dm, 4),
                             "compress_frac": frac(nbytes + ltot, cm), "decompress_frac": frac(nbytes + ltot, dm)}
            log(f"[bench] {lname}: ratio {ltot / nbytes:.4f} compress {cm:.3f} ms decompress {dm:.3f} ms")
            del lo, lw, ly

        # ------------- 2 GiB bf16 KV cache, 1 MiB chunks -------------
        mark("kv_chunked")
        kh = W.kv_cache()
        nk = kh.size
        kt = torch.from_numpy(kh.view(np.int16)).to(dev)
        del kh
        kcb = 1 << 20
        kchunks = (2 * nk + kcb - 1) // kcb
        kflags = torch.zeros(2 * kchunks, dtype=torch.int32).pin_memory()
        kslot = (uz.uzip_max_compressed_size(uz.BF16, kcb // 2, bb) + 255) // 256 * 256
        kout = torch.empty(kslot * kchunks, dtype=torch.uint8, device=dev)
        kws = torch.empty(uz.uzip_workspace_size(uz.OP_CHUNKED, uz.BF16, nk, bb, kcb), dtype=torch.uint8, device=dev)
        kep = [0]

        def kproduce():
            kep[0] += 1
            return uz.compress_chunked(kt, bb, kcb, dtype="bf16", epoch=kep[0], flags=kflags, out=kout, ws=kws)

        kt_ms = timed(kproduce, reps)
        ksizes = uz.compress_chunked(kt, bb, kcb, dtype="bf16", epoch=kep[0] + 1, flags=kflags, out=kout, ws=kws)[2]
        torch.cuda.synchronize()
        ktot = int(ksizes.sum().item())
        # a receiver that decodes each 1 MiB chunk stream on its own: one
        # call per chunk on one stream (each call runs the chunk's 16 blocks
        # alone, so its time is one block's sequential decode)
        ky = torch.empty_like(kt)
        kce = kcb // 2
        kst = torch.zeros(1, dtype=torch.int32, device=dev)
        s_ptr = stream.cuda_stream

        def kdecode():
            for c in range(kchunks):
                uz.uzip_decompress(kout.data_ptr() + c * kslot, kslot, uz.BF16, kce, ky.data_ptr() + 2 * c * kce,
                                   2 * kce, kst.data_ptr(), None, 0, s_ptr)

        mark("kv_chunk_decode_calls")
        kd_ms = timed(kdecode, 3)
        assert int(kst.item()) == 0 and torch.equal(kt, ky)
        # the same chunk streams, all decoded in one launch
        mark("kv_chunk_decode_batched")
        ky.zero_()
        kb_ms = timed(lambda: uz.uzip_decompress_chunked(kout.data_ptr(), kslot, 0, kchunks, uz.BF16, nk, bb, kcb,
                                                         ky.data_ptr(), 2 * nk, kst.data_ptr(), s_ptr), reps)
        assert int(kst.item()) == 0 and torch.equal(kt, ky)
        del kout, kws, ky
        # the same tensor as one stream (one launch each way)
        mark("kv_whole_stream")
        ko = torch.empty(uz.uzip_max_compressed_size(uz.BF16, nk, bb), dtype=torch.uint8, device=dev)
        kw = torch.empty(uz.uzip_workspace_size(uz.OP_COMPRESS, uz.BF16, nk, bb), dtype=torch.uint8, device=dev)
        ky2 = torch.empty_like(kt)
        kwh_c = timed(lambda: uz.compress(kt, bb, dtype="bf16", out=ko, ws=kw), 3)
        kwh_d = timed(lambda: uz.decompress(ko, "bf16", nk, out=ky2, ws=dws), 3)
        assert torch.equal(kt, ky2)
        kc, kd, kbd = float(np.mean(kt_ms)), float(np.mean(kd_ms)), float(np.mean(kb_ms))
        kb = 2 * nk
        extras["kv_cache_bf16_2GiB"] = {
            "n_elems": nk, "block_bytes": bb, "chunk_bytes": kcb, "chunks": kchunks, "ratio": round(ktot / kb, 4),
            "chunked_compress_ms": round(kc, 4), "chunked_compress_GBps": gbps(kb, kc),
            "chunked_compress_frac": frac(kb + ktot, kc),
            "chunks_decompress_ms": round(kbd, 4), "chunks_decompress_GBps": gbps(kb, kbd),
            "chunks_decompress_frac": frac(kb + ktot, kbd),
            "per_chunk_calls_decompress_ms": round(kd, 4), "per_chunk_calls_decompress_GBps": gbps(kb, kd),
            "whole_stream_compress_ms": round(float(np.mean(kwh_c)), 4),
            "whole_stream_decompress_ms": round(float(np.mean(kwh_d)), 4),
            "whole_stream_decompress_frac": frac(kb + ktot, float(np.mean(kwh_d)))}
        log(f"[bench] kv 2 GiB: ratio {ktot / kb:.4f} chunked compress {kc:.3f} ms, all chunks decompressed in "
            f"one launch {kbd:.3f} ms, {kchunks} decompress calls {kd:.3f} ms")
        del kt, ko, kw, ky2

        # ------------- fused reduce: 8 compressed bf16 shares [1024 x 8192] -------------
        mark("reduce_inputs")
        shares = W.reduce_slices()
        rn = shares[0].size
        streams = []
        for s in shares:
            st, sz = uz.compress(torch.from_numpy(s.view(np.int16)).to(dev), bb, dtype="bf16")
            streams.append(st[:int(sz.item())].clone())
        in_bytes = [t.numel() for t in streams]
        rcap = uz.uzip_max_compressed_size(uz.BF16, rn, bb)
        rout = torch.empty(rcap, dtype=torch.uint8, device=dev)
        rws = torch.empty(uz.uzip_workspace_size(uz.OP_REDUCE, uz.BF16, rn, bb, 8), dtype=torch.uint8, device=dev)
        res = {}

        def reduce_call():
            res["r"] = uz.reduce_fused(streams, "bf16", rn, bb, out=rout, ws=rws)

        # the inputs (~90 MB) fit the 256 MB Infinity Cache: warm runs, and
        # cold ones each after a 512 MiB write that evicts them
        mark("reduce_8x16MiB")
        times = timed(reduce_call, reps)
        cold = timed(reduce_call, reps, flush)
        _, rsz, raw, rst = res["r"]
        assert int(rst.item()) == 0
        r_ms = float(np.mean(times))
        rc_ms = float(np.median(cold))
        moved = sum(in_bytes) + int(rsz.item()) + 2 * rn
        extras["reduce"] = {"n_in": 8, "share_elems": rn, "ms": round(r_ms, 4),
                            "ms_cold_median": round(rc_ms, 4), "ms_cold_min": round(float(np.min(cold)), 4),
                            "hbm_frac_cold": frac(moved, rc_ms),
                            "input_GBps_uncompressed": gbps(8 * 2 * rn, r_ms),
                            "hbm_frac": frac(moved, r_ms),
                            "ratio_in": round(sum(in_bytes) / (8 * 2 * rn), 4),
                            "ratio_out": round(int(rsz.item()) / (2 * rn), 4)}
        log(f"[bench] fused reduce {r_ms:.3f} ms (after a cache flush: {rc_ms:.3f} ms)")
        del rout, rws, streams

        if not args.no_reduce_full:
            # the other reading of the activation slices: each input is the
            # whole [8192 x 8192] tensor (128 MiB), 2048 blocks per input
            mark("reduce_full_inputs")
            fshares = W.reduce_slices(tokens=8192)
            fn_ = fshares[0].size
            fstreams = []
            for s_ in fshares:
                st, sz = uz.compress(torch.from_numpy(s_.view(np.int16)).to(dev), bb, dtype="bf16")
                fstreams.append(st[:int(sz.item())].clone())
            del fshares
            f_in = sum(t.numel() for t in fstreams)
            fout = torch.empty(uz.uzip_max_compressed_size(uz.BF16, fn_, bb), dtype=torch.uint8, device=dev)
            fws = torch.empty(uz.uzip_workspace_size(uz.OP_REDUCE, uz.BF16, fn_, bb, 8), dtype=torch.uint8,
                              device=dev)

            def freduce():
                res["f"] = uz.reduce_fused(fstreams, "bf16", fn_, bb, out=fout, ws=fws)

            mark("reduce_full_tensor")
            times = timed(freduce, reps)
            _, fsz, fraw, fst = res["f"]
            assert int(fst.item()) == 0
            # the output stream decodes to the reduced tensor the call returned
            fy, fyst = uz.decompress(fout, "bf16", fn_)
            torch.cuda.synchronize()
            assert int(fyst.item()) == 0 and torch.equal(fy.view(torch.int16), fraw.view(torch.int16))
            f_ms = float(np.mean(times))
            f_moved = f_in + int(fsz.item()) + 2 * fn_
            extras["reduce_full_tensor"] = {
                "n_in": 8, "elems_per_input": fn_, "ms": round(f_ms, 4),
                "input_GBps_uncompressed": gbps(8 * 2 * fn_, f_ms),
                "hbm_frac": frac(f_moved, f_ms), "ratio_in": round(f_in / (8 * 2 * fn_), 4)}
            log(f"[bench] fused reduce, full-tensor reading (8 x 128 MiB) {f_ms:.3f} ms")
            del fstreams, fout, fws, fy, fraw
            res.clear()

        # ------------- stream-wide tables: the same buffer, one table per stream -------------
        mark("tables")
        tws = torch.empty(uz.uzip_workspace_size(uz.OP_COMPRESS_TABLE, uz.BF16, n, bb), dtype=torch.uint8, device=dev)
        tout = torch.empty(cap + uz.TABLE_BYTES, dtype=torch.uint8, device=dev)
        ty = torch.empty_like(x)
        tab = uz.build_table(x, dtype="bf16")
        for mode in ("sampled", "external"):
            tabarg = tab if mode == "external" else None
            for _ in range(2):
                _, tsz = uz.compress_table(x, bb, mode, tabarg, dtype="bf16", out=tout, ws=tws)
                _, tst = uz.decompress_table(tout, "bf16", n, tabarg, out=ty, ws=dws)
            torch.cuda.synchronize()
            if int(tst.item()) != 0 or not torch.equal(x, ty):
                log(f"[bench] table mode {mode}: round trip is NOT lossless")
                return 1
            tsize = int(tsz.item())
            ct = timed(lambda: uz.compress_table(x, bb, mode, tabarg, dtype="bf16", out=tout, ws=tws), reps)
            dt_ = timed(lambda: uz.decompress_table(tout, "bf16", n, tabarg, out=ty, ws=dws), reps)
            fc, fd = float(np.mean(ct)), float(np.mean(dt_))
            moved = nbytes + tsize
            extras[f"table_{mode}"] = {"ratio": round(tsize / nbytes, 5),
                                       "ratio_cost_vs_per_block": round(tsize / total - 1, 4),
                                       "compress_ms": round(fc, 4), "decompress_ms": round(fd, 4),
                                       "compress_frac": frac(moved, fc), "decompress_frac": frac(moved, fd)}
            log(f"[bench] table {mode}: ratio {tsize / nbytes:.4f} compress {fc:.3f} ms decompress {fd:.3f} ms")
        del tws, tout, ty
        # split-send producer with a table per 4 MiB chunk (sampled from the chunk's first 256 KiB)
        mark("chunked_sampled_tables")
        cws2 = torch.empty(uz.uzip_workspace_size(uz.OP_CHUNKED_TABLE, uz.BF16, n, bb, cb), dtype=torch.uint8,
                           device=dev)
        slot2 = (uz.uzip_max_compressed_size(uz.BF16, cb // 2, bb) + uz.TABLE_BYTES + 255) // 256 * 256
        cout2 = torch.empty(slot2 * chunks, dtype=torch.uint8, device=dev)

        def produce2():
            epoch[0] += 1
            res["c2"] = uz.compress_chunked_table(x, bb, cb, "sampled", dtype="bf16", epoch=epoch[0], flags=flags,
                                                  out=cout2, ws=cws2)

        times = timed(produce2, reps)
        assert bool((flags == epoch[0]).all())
        c2 = int(res["c2"][2].sum().item())
        extras["chunked_sampled_tables"] = {"chunk_bytes": cb, "ms": round(float(np.mean(times)), 4),
                                            "ratio": round(c2 / nbytes, 5),
                                            "ratio_cost_vs_per_block": round(c2 / total - 1, 4)}
        log(f"[bench] chunked, sampled table per chunk: ratio {c2 / nbytes:.4f} {np.mean(times):.3f} ms")
        del cws2, cout2, res

        # ------------- FP8 pairs: 1 GiB of e4m3fn / e5m2 values N(0, 1) -------------
        for fmt, code in (("e4m3fn", uz.E4M3FN), ("e5m2", uz.E5M2)):
            mark(f"fp8_{fmt}")
            f8 = torch.from_numpy(W.normal_fp8_pairs(n, fmt).view(np.int16)).to(dev)
            fout = torch.empty(uz.uzip_max_compressed_size(code, n, bb), dtype=torch.uint8, device=dev)
            fws = torch.empty(uz.uzip_workspace_size(uz.OP_COMPRESS, code, n, bb), dtype=torch.uint8, device=dev)
            fy = torch.empty_like(f8)
            fsz = uz.compress(f8, bb, dtype=fmt, out=fout, ws=fws)[1]
            ct = timed(lambda: uz.compress(f8, bb, dtype=fmt, out=fout, ws=fws), reps)
            dt_ = timed(lambda: uz.decompress(fout, fmt, n, out=fy, ws=dws), reps)
            if not torch.equal(f8, fy):
                log(f"[bench] {fmt} round trip is NOT lossless")
                return 1
            fsize = int(fsz.item())
            fc, fd = float(np.mean(ct)), float(np.mean(dt_))
            moved = nbytes + fsize
            extras[f"fp8_{fmt}"] = {"workload": f"normal_{fmt}_pairs_1GiB", "pairs": n, "ratio": round(fsize / nbytes, 4),
                                    "compress_ms": round(fc, 4), "decompress_ms": round(fd, 4),
                                    "compress_frac": frac(moved, fc), "decompress_frac": frac(moved, fd)}
            log(f"[bench] {fmt}: ratio {fsize / nbytes:.4f} compress {fc:.3f} ms decompress {fd:.3f} ms")
            del f8, fout, fws, fy
        del flush_buf

    if args.calibrate_copy:
        # a plain device copy of known size, for scaling the HBM counters
        mark("calibration_copy")
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    mark(None)
    cpu = None
    if not args.no_cpu_baseline:
        # the oracle as it stands, on independent 4 MiB chunks of the same
        # buffer (every 16th of its 256 chunks): compress + decompress of each
        # (ctypes releases the GIL, so threads run the C oracle in parallel)
        from concurrent.futures import ThreadPoolExecutor
        from oracle import ref
        ce = 2 << 20
        picks = list(range(0, n // ce, 16))

        def roundtrip(c):
            xs = x_host[c * ce:(c + 1) * ce]
            s_ = ref.compress(xs, "bf16", bb)
            yy = ref.decompress(s_, "bf16", xs.size)
            assert yy is not None and np.array_equal(yy, xs)

        def run(nthreads, chunk_list):
            t0_ = time.perf_counter()
            with ThreadPoolExecutor(nthreads) as ex_:
                list(ex_.map(roundtrip, chunk_list))
            return time.perf_counter() - t0_

        threads = host_threads()
        one = [run(1, picks[:8]) for _ in range(3)]
        all_list = [picks[i % len(picks)] for i in range(4 * threads)]
        allt = [run(threads, all_list) for _ in range(3)]
        g1 = 2 * ce * 8 / float(np.median(one)) / 1e9
        ga = 2 * ce * len(all_list) / float(np.median(allt)) / 1e9
        cpu = {"value": round(ga, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
               "sample": f"compress + decompress round trips of 4 MiB chunks of the weight-sync buffer (every 16th "
                         f"chunk; 8 on one thread, 4 per thread on all: {len(all_list)} chunks on {threads} threads), C oracle, median of 3",
               "single_thread_GBps": round(g1, 4), "host_cpus": os.cpu_count(), "cpu_model": cpu_model(),
               "seconds": round(float(np.sum(one) + np.sum(allt)), 2)}
        log(f"[bench] cpu oracle: {g1:.3f} GB/s on 1 thread, {ga:.3f} GB/s on {threads} threads "
            f"({os.cpu_count()} CPUs, {cpu['cpu_model']})")

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "preheat": {"ms": PREHEAT_MS, "untimed_steps": pre_steps},
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": "weight_sync_bf16_1GiB", "elem_dtype": "bf16", "n_elems": n,
                   "block_bytes": bb, "step": "uzip_compress + uzip_decompress of the whole buffer"},
        "compress_GBps": round(comp_gbps, 1), "decompress_GBps": round(dec_gbps, 1),
        "compress_ms": round(c_ms, 4), "decompress_ms": round(d_ms, 4),
        "compress_ms_median": round(float(np.median(comp_ms)), 4), "compress_ms_min": round(float(np.min(comp_ms)), 4),
        "decompress_ms_median": round(float(np.median(dec_ms)), 4),
        "decompress_ms_min": round(float(np.min(dec_ms)), 4),
        "ratio": round(total / nbytes, 5), "compressed_bytes": total,
        "roofline": roofline, "cpu_baseline": cpu, **extras,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
