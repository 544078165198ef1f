#!/usr/bin/env python3
"""Benchmark: 1080p frames/s, encode + decode, on one MI355X, fp16 and int16 paths.

One step = one frame of the 1920x1088 P-frame sequence (C = 256 at 1/8
scale, 8 + 8 DC blocks) encoded by one context and decoded by another; all
frames are resident in HBM before the timed region starts.  ``value`` is the
fp16 path's frames/s (encode + decode of each frame); the int16 path is
measured in the same run and reported under ``"int16"``.

After the timed region an instrumented pass over the same frames records
HIP events around every kernel on the codec's stream; the dominant kernel's
average duration gives ``roofline.achieved``.  The CPU oracle is timed on a
bounded spatial sample of the same workload for ``cpu_baseline``.

Usage: python bench.py [--steps K] [--warmup W] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import statistics
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "1080p frames/sec encode and decode on 1 MI355X (fp16 and int path)"
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0
MFMA_I8_PEAK_TOPS = 5000.0


def workload_model(H, W, C, ne, nd, block="lrelu"):
    """Algorithmic flops and HBM bytes per launch of each kernel kind (weights excluded).
    The DC block's pointwise pair is C -> 2C -> C (LeakyReLU form) or C -> 2C, C -> C
    (gated form: 6 C^2 flops per pixel instead of 8 C^2)."""
    P8 = (H // 8) * (W // 8)
    P16 = P8 // 4
    fmap = P8 * C * 2
    lat = P16 * C * 2
    frame = 3 * H * W * 2
    k = {
        "embed": (2 * P8 * C * 192, frame + fmap),
        "fuse": (2 * P8 * C * 2 * C, 3 * fmap),
        "dcblock": (P8 * ((8 if block == "lrelu" else 6) * C * C + 18 * C), 2 * fmap),
        "down": (2 * P16 * C * 4 * C, fmap + lat),
        "prior_enc": (2 * P16 * 2 * C * C, 4 * lat),
        "prior_dec": (2 * P16 * C * C, 3 * lat),
        "up": (2 * P16 * 4 * C * C, lat + fmap),
        "recon": (2 * P8 * 192 * C, fmap + frame),
    }
    enc = ["embed", "fuse"] + ["dcblock"] * ne + ["down", "prior_enc", "up", "fuse"] + ["dcblock"] * nd
    dec = ["prior_dec", "up", "fuse"] + ["dcblock"] * nd + ["recon"]
    return k, enc, dec


def roofline_seconds(kinds, names, flop_peak):
    t = 0.0
    for n in names:
        fl, by = kinds[n]
        t += max(fl / flop_peak, by / (HBM_PEAK_GBS * 1e9))
    return t


def macs_per_frame(H, W, C, ne, nd):
    kinds, enc, dec = workload_model(H, W, C, ne, nd)
    return sum(kinds[n][0] for n in enc) / 2, sum(kinds[n][0] for n in dec) / 2


def cpu_baseline(pre, weights, strip_rows, path="fp16"):
    """Oracle (NumPy, float64 or exact integers) encode and decode of a horizontal strip
    of the first frame, timed separately."""
    import numpy as np

    import oracle
    import synth
    from oracle import codec_float as cf
    from oracle import codec_int as ci

    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=os.cpu_count())
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    p = oracle.unpack(weights, pre.channels, pre.n_enc, pre.n_dec)
    x = next(synth.frame_sequence(pre, 1))[:, :strip_rows, :]
    if path == "int16":
        m, p = ci, ci.integerize(p)
    else:
        m = cf
    st = m.zero_state(p, strip_rows, pre.width)
    t0 = time.perf_counter()
    r = m.encode_frame(p, x, st)
    t1 = time.perf_counter()
    m.decode_frame(p, r.q, st)
    t2 = time.perf_counter()
    frac = strip_rows / pre.height
    kind = "float64 NumPy" if path == "fp16" else "exact-integer NumPy"
    return {"value": frac / (t2 - t0), "unit": "frames/s", "cores": int(threads), "kind": "oracle",
            "encode_fps": frac / (t1 - t0), "decode_fps": frac / (t2 - t1),
            "sample": f"{path}-path oracle ({kind}) encode + decode of the top {strip_rows} of {pre.height} rows "
                      f"of 1080p frame 0 ({t2 - t0:.1f} s), scaled by {frac:.3f}; host cpu_count={os.cpu_count()}"}


TRAFFIC_PROFILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "dcblock_hd1080_hbm_traffic.md")
CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2502_20762_amd", "csrc")
SOURCES = {"k_dcchain128_f16<false>": ["kernels_f16_dc128.hip", "common.hpp", "internal.hpp"],
           "k_dcblock128_f16<false>": ["kernels_f16_dc128.hip", "common.hpp", "internal.hpp"],
           "k_dcchain128_i16": ["kernels_i16_dc128.hip", "common.hpp", "internal.hpp"],
           "k_dcblock128_i16": ["kernels_i16_dc128.hip", "common.hpp", "internal.hpp"]}


def counted_traffic(kernel):
    """HBM bytes per launch from the committed counter summary (FETCH_SIZE and WRITE_SIZE
    passes scaled by a plain copy), or None if it is missing or the kernel sources changed
    since the counters were taken."""
    import hashlib
    try:
        text = open(TRAFFIC_PROFILE).read()
        h = hashlib.sha256()
        for f in SOURCES[kernel]:
            h.update(open(os.path.join(CSRC, f), "rb").read())
    except (OSError, KeyError):
        return None
    for line in text.splitlines():
        parts = line.split()
        if len(parts) >= 4 and parts[0] == "traffic" and parts[1] == kernel.replace(" ", ""):
            fields = dict(p.split("=", 1) for p in parts[2:])
            if fields.get("sources_sha256") == h.hexdigest():
                return int(fields["bytes_per_launch"])
    return None


def timed_loop(enc, dec, gframes, qbuf, bits, xout, steps, warmup, torch):
    """Encode then decode `steps` frames; per-frame event stamps on the codec stream."""
    stream = torch.cuda.current_stream()
    nfr = len(gframes)
    ev_e = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev_d = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev_e[0].record(stream)
    for k in range(steps):
        enc.encode(gframes[(warmup + k) % nfr], q_out=qbuf[k], bits_out=bits[k])
        ev_e[k + 1].record(stream)
    ev_d[0].record(stream)
    for k in range(steps):
        dec.decode(qbuf[k], out=xout)
        ev_d[k + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fe = [ev_e[k].elapsed_time(ev_e[k + 1]) for k in range(steps)]
    fd = [ev_d[k].elapsed_time(ev_d[k + 1]) for k in range(steps)]
    return {"enc_ms": sum(fe), "dec_ms": sum(fd), "wall_s": wall,
            "enc_median_ms": statistics.median(fe), "dec_median_ms": statistics.median(fd)}


def coded_loop(enc, dec, gframes, steps, warmup, xout, torch, parallel=False):
    """Encode each frame into a container and decode it from the container
    (Fig. 4 "AE" / "AD" on the GPU); per-frame event stamps; the decoder is given
    the buffer capacity as the container size (the header holds the lengths).
    parallel: the coder overlaps the decoder part of the encode on a second
    stream (Fig. 6, supplementary "Parallel Coding")."""
    stream = torch.cuda.current_stream()
    enc.parallel_coding(parallel)
    dec.parallel_coding(parallel)
    nfr = len(gframes)
    cap = enc.stream_capacity()
    sbuf = [torch.empty(cap, dtype=torch.uint8, device="cuda") for _ in range(2)]
    # one byte count and status per container: three (z, y^1, y^2) with the
    # two-step entropy model
    nsec = (3,) if enc.hyperprior else ()
    nbytes = torch.zeros((steps,) + nsec, dtype=torch.int64, device="cuda")
    status = torch.zeros((steps,) + nsec, dtype=torch.int32, device="cuda")
    bits = torch.zeros(steps, dtype=torch.float64, device="cuda")
    enc.reset()
    dec.reset()
    for i in range(warmup):
        enc.encode_coded(gframes[i % nfr], stream=sbuf[0], nbytes_out=nbytes[0])
        dec.decode_coded(sbuf[0], cap, out=xout, status_out=status[0])
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    for k in range(steps):
        b = sbuf[k % 2]
        ev[k][0].record(stream)
        enc.encode_coded(gframes[(warmup + k) % nfr], stream=b, nbytes_out=nbytes[k], bits_out=bits[k])
        ev[k][1].record(stream)
        dec.decode_coded(b, cap, out=xout, status_out=status[k])
        ev[k][2].record(stream)
    torch.cuda.synchronize()
    enc_ms = [e[0].elapsed_time(e[1]) for e in ev]
    dec_ms = [e[1].elapsed_time(e[2]) for e in ev]
    # the same loop without the coder (encode with bits, decode from the symbols),
    # for the coder's share at equal loop structure
    qk = torch.empty(enc.q_shape, dtype=torch.int16, device="cuda")
    enc.reset()
    dec.reset()
    for i in range(warmup):
        enc.encode(gframes[i % nfr], q_out=qk, bits_out=bits[0])
        dec.decode(qk, out=xout)
    pv = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    for k in range(steps):
        pv[k][0].record(stream)
        enc.encode(gframes[(warmup + k) % nfr], q_out=qk, bits_out=bits[k])
        pv[k][1].record(stream)
        dec.decode(qk, out=xout)
        pv[k][2].record(stream)
    torch.cuda.synchronize()
    plain_enc = sum(e[0].elapsed_time(e[1]) for e in pv)
    plain_dec = sum(e[1].elapsed_time(e[2]) for e in pv)
    per_frame = nbytes.reshape(steps, -1).sum(dim=1).double()
    res = {"encode_fps": steps / (sum(enc_ms) * 1e-3), "decode_fps": steps / (sum(dec_ms) * 1e-3),
           "value": steps / ((sum(enc_ms) + sum(dec_ms)) * 1e-3),
           "uncoded_same_loop": {"encode_fps": steps / (plain_enc * 1e-3), "decode_fps": steps / (plain_dec * 1e-3)},
           "bytes_per_frame": float(per_frame[1:].mean().item()) if steps > 1 else float(per_frame[0].item()),
           "estimated_bytes_per_frame": float(bits[1:].mean().item()) / 8.0 if steps > 1 else float(bits[0].item()) / 8.0}
    if enc.hyperprior:
        # the scale indices of y depend on the frame's z and y^1: no coder-alone timing
        enc.parallel_coding(False)
        dec.parallel_coding(False)
        res["decoded_ok"] = bool((status == 0).all().item())
        return res
    # the coder alone, on the last frame's symbols: container in, container out
    q = torch.empty(enc.q_shape, dtype=torch.int16, device="cuda")
    k_idx = enc.scale_indices()
    enc.encode(gframes[0], q_out=q)
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    reps = 8
    out_q = torch.empty_like(q)
    e0.record(stream)
    for _ in range(reps):
        enc.rans_encode(q, k_idx, stream=sbuf[0], nbytes_out=nbytes[0])
    e1.record(stream)
    for _ in range(reps):
        enc.rans_decode(sbuf[0], cap, k_idx, out=out_q, status_out=status[0])
    e2.record(stream)
    torch.cuda.synchronize()
    enc.parallel_coding(False)
    dec.parallel_coding(False)
    ok = bool((status == 0).all().item()) and bool(torch.equal(out_q, q))
    res.update({"rans_encode_us": 1e3 * e0.elapsed_time(e1) / reps, "rans_decode_us": 1e3 * e1.elapsed_time(e2) / reps,
                "decoded_ok": ok})
    return res


def run_path(path, pre, weights, gframes, steps, warmup, torch, Codec):
    H, W, C, ne, nd = pre.height, pre.width, pre.channels, pre.n_enc, pre.n_dec
    enc = Codec(H, W, C, ne, nd, path, weights)
    dec = Codec(H, W, C, ne, nd, path, weights)
    odt = torch.int16 if path == "int16" else torch.float16
    qbuf = [torch.empty(enc.q_shape, dtype=torch.int16, device="cuda") for _ in range(steps)]
    bits = torch.zeros(steps, dtype=torch.float64, device="cuda")
    xout = torch.empty(enc.frame_shape, dtype=odt, device="cuda")
    nfr = len(gframes)

    def warm():
        enc.reset()
        dec.reset()
        for i in range(warmup):
            q, _ = enc.encode(gframes[i % nfr])
            dec.decode(q, out=xout)
        torch.cuda.synchronize()

    # direct launches (the library default), then the same frames as hipGraph replays
    warm()
    r = timed_loop(enc, dec, gframes, qbuf, bits, xout, steps, warmup, torch)
    enc.graphs(True)
    dec.graphs(True)
    warm()
    graph = timed_loop(enc, dec, gframes, qbuf, bits, xout, steps, warmup, torch)
    enc.graphs(False)
    dec.graphs(False)

    # instrumented pass: events around every kernel, same frames (always direct launches)
    enc.reset()
    dec.reset()
    enc.timing(True)
    dec.timing(True)
    for k in range(steps):
        enc.encode(gframes[(warmup + k) % nfr], q_out=qbuf[k], bits_out=bits[k])
        dec.decode(qbuf[k], out=xout)
    te, td = enc.timing_read(), dec.timing_read()
    enc.timing(False)
    dec.timing(False)
    kern = {}
    for src in (te, td):
        for kind, (n, ms) in src.items():
            a = kern.setdefault(kind, [0, 0.0])
            a[0] += n
            a[1] += ms
    coded = coded_loop(enc, dec, gframes, steps, warmup, xout, torch)
    coded["parallel_coding"] = {k: v for k, v in coded_loop(enc, dec, gframes, steps, warmup, xout, torch,
                                                            parallel=True).items()
                                if k in ("encode_fps", "decode_fps", "value", "decoded_ok", "uncoded_same_loop")}
    r.update({
        "graph": graph,
        "coded": coded,
        "bits_per_frame": float(bits.mean().item()),
        "kernels": {k: {"launches": n, "avg_us": 1e3 * ms / n, "total_ms": ms} for k, (n, ms) in kern.items()},
        "kernels_per_frame": [enc.kernels_per_frame(False), dec.kernels_per_frame(True)],
        "block_chains": bool(enc.block_chain_status()[0]),
        "chain_timeouts": enc.block_chain_status()[1] + dec.block_chain_status()[1],
    })
    return r


def run_gated(path, pre, gframes, steps, warmup, torch, Codec):
    """The gated DC-block form (Supp. B.1, WSiLU + Chunk) on the same frames:
    frames/s and the per-kernel event times of its launches."""
    import synth
    H, W, C, ne, nd = pre.height, pre.width, pre.channels, pre.n_enc, pre.n_dec
    weights = synth.make_weights(C, ne, nd, block="gated")
    enc = Codec(H, W, C, ne, nd, path, weights, block="gated")
    dec = Codec(H, W, C, ne, nd, path, weights, block="gated")
    odt = torch.int16 if path == "int16" else torch.float16
    qbuf = [torch.empty(enc.q_shape, dtype=torch.int16, device="cuda") for _ in range(steps)]
    bits = torch.zeros(steps, dtype=torch.float64, device="cuda")
    xout = torch.empty(enc.frame_shape, dtype=odt, device="cuda")
    nfr = len(gframes)
    for i in range(warmup):
        q, _ = enc.encode(gframes[i % nfr])
        dec.decode(q, out=xout)
    enc.reset()
    dec.reset()
    torch.cuda.synchronize()
    r = timed_loop(enc, dec, gframes, qbuf, bits, xout, steps, warmup, torch)
    enc.reset()
    dec.reset()
    enc.timing(True)
    dec.timing(True)
    for k in range(steps):
        enc.encode(gframes[(warmup + k) % nfr], q_out=qbuf[k], bits_out=bits[k])
        dec.decode(qbuf[k], out=xout)
    kern = {}
    te, td = enc.timing_read(), dec.timing_read()
    enc.timing(False)
    dec.timing(False)
    for src in (te, td):
        for kind, (n, ms) in src.items():
            a = kern.setdefault(kind, [0, 0.0])
            a[0] += n
            a[1] += ms
    K = steps
    return {"value": K / ((r["enc_ms"] + r["dec_ms"]) * 1e-3), "encode_fps": K / (r["enc_ms"] * 1e-3),
            "decode_fps": K / (r["dec_ms"] * 1e-3),
            "kernels_us": {k: round(1e3 * ms / n, 2) for k, (n, ms) in kern.items()},
            "kernels_per_frame": [enc.kernels_per_frame(False), dec.kernels_per_frame(True)]}


SWEEP = [  # (label, H, W, C, N_e, N_d, N_f, N_r, block, two-step entropy model):
    # resolution, width, depth, modules, form
    ("720p", 720, 1280, 256, 8, 8, 0, 0, "lrelu", False),
    ("1080p C=64", 1088, 1920, 64, 8, 8, 0, 0, "lrelu", False),
    ("1080p C=128", 1088, 1920, 128, 8, 8, 0, 0, "lrelu", False),
    ("1080p", 1088, 1920, 256, 8, 8, 0, 0, "lrelu", False),
    ("1080p gated blocks", 1088, 1920, 256, 8, 8, 0, 0, "gated", False),
    ("1080p 16+16 blocks", 1088, 1920, 256, 16, 16, 0, 0, "lrelu", False),
    ("1080p 32+32 blocks", 1088, 1920, 256, 32, 32, 0, 0, "lrelu", False),
    ("1080p + feature extractor (2 blocks), reconstruction generation (2 blocks), qp banks",
     1088, 1920, 256, 8, 8, 2, 2, "lrelu", False),
    ("1080p + two-step entropy model with hyperprior", 1088, 1920, 256, 8, 8, 0, 0, "lrelu", True),
    ("1080p, all modules: feature extractor, reconstruction generation, qp banks, two-step entropy model",
     1088, 1920, 256, 8, 8, 2, 2, "lrelu", True),
    ("4K", 2176, 3840, 256, 8, 8, 0, 0, "lrelu", False),
    ("1080p C=384 (wide blocks)", 1088, 1920, 384, 8, 8, 0, 0, "lrelu", False),
    ("1080p C=512 (wide blocks, a Large model's width)", 1088, 1920, 512, 8, 8, 0, 0, "lrelu", False),
    ("1080p C=512 16+16 blocks (a Large model's width and depth)", 1088, 1920, 512, 16, 16, 0, 0, "lrelu", False),
    ("1080p C=512 gated blocks (wide blocks, the paper's block form)", 1088, 1920, 512, 8, 8, 0, 0, "gated", False),
]


def sweep(paths, steps, warmup, torch, Codec, match=""):
    """Frames/s and the DC block's MFMA fraction across resolutions, widths and
    depths (random-init weights, seeded random frames); one JSON line each."""
    import synth
    for label, H, W, C, ne, nd, nfe, nrg, block, hyper in SWEEP:
        if match not in label:
            continue
        frames = [torch.from_numpy(synth.random_frame(H, W, seed=90 + i)).to("cuda") for i in range(4)]
        banks = nfe + nrg > 0
        weights = synth.make_weights(C, ne, nd, block=block, n_fe=nfe, n_rg=nrg, banks=banks, hyper=hyper)
        kinds, enc_list, dec_list = workload_model(H, W, C, ne, nd, block)
        enc_list = ["dcblock"] * nfe + enc_list
        dec_list = ["dcblock"] * (nfe + nrg) + dec_list
        for path in paths:
            kw = dict(block=block, n_fe_blocks=nfe, n_rg_blocks=nrg, qp_banks=banks, hyperprior=hyper)
            enc = Codec(H, W, C, ne, nd, path, weights, **kw)
            dec = Codec(H, W, C, ne, nd, path, weights, **kw)
            odt = torch.int16 if path == "int16" else torch.float16
            qbuf = [torch.empty(enc.q_shape, dtype=torch.int16, device="cuda") for _ in range(steps)]
            bits = torch.zeros(steps, dtype=torch.float64, device="cuda")
            xout = torch.empty(enc.frame_shape, dtype=odt, device="cuda")
            for i in range(warmup):
                q, _ = enc.encode(frames[i % 4])
                dec.decode(q, out=xout)
            enc.reset()
            dec.reset()
            torch.cuda.synchronize()
            r = timed_loop(enc, dec, frames, qbuf, bits, xout, steps, warmup, torch)
            enc.reset()
            enc.timing(True)
            for k in range(min(steps, 4)):
                enc.encode(frames[k % 4], q_out=qbuf[k], bits_out=bits[k])
            t = enc.timing_read()
            enc.timing(False)
            n, ms = t.get("dcblock", (0, 0.0))
            if not n and "dcblock_dw" in t:  # a wide block (C > 256) is three launches
                n = t["dcblock_dw"][0]
                ms = sum(v[1] for k, v in t.items() if k.startswith("dcblock_"))
            peak, scale = (MFMA_F16_PEAK_TFLOPS, 1) if path == "fp16" else (MFMA_I8_PEAK_TOPS, 4)
            frac = scale * kinds["dcblock"][0] / (ms * 1e-3 / n) / 1e12 / peak if n else None
            t_roof = roofline_seconds(kinds, enc_list + dec_list, peak * 1e12 / scale)
            value = steps / ((r["enc_ms"] + r["dec_ms"]) * 1e-3)
            coded = None
            if hyper:  # three containers per frame (z, y^1, y^2)
                c = coded_loop(enc, dec, frames, steps, warmup, xout, torch)
                coded = {k: c[k] for k in ("encode_fps", "decode_fps", "value", "bytes_per_frame",
                                           "estimated_bytes_per_frame", "decoded_ok")}
            print(json.dumps({"sweep": label, "path": path, "height": H, "width": W, "channels": C,
                              "n_enc_blocks": ne, "n_dec_blocks": nd, "n_fe_blocks": nfe, "n_rg_blocks": nrg,
                              "block": block, "two_step_entropy_model": hyper, "coded": coded,
                              "frames_per_s": value,
                              "encode_fps": steps / (r["enc_ms"] * 1e-3), "decode_fps": steps / (r["dec_ms"] * 1e-3),
                              "dcblock_us": 1e3 * ms / n if n else None, "dcblock_mfma_frac": frac,
                              "encode_kernels_us": {k: round(1e3 * v[1] / v[0], 2) for k, v in t.items()},
                              "frame_roofline_fps": 1.0 / t_roof, "frac_of_frame_roofline": value * t_roof}),
                  flush=True)
            del enc, dec, qbuf, xout
            torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--paths", default="fp16,int16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gated", action="store_true", help="skip the gated DC-block form")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the 1080p line: one line per resolution / width / depth of the sweep table")
    ap.add_argument("--sweep-match", default="", help="only the sweep rows whose label contains this text")
    ap.add_argument("--cpu-strip-rows", type=int, default=1088)
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="first run a plain device copy of this many MiB (3 times), as the reference "
                         "kernel for scaling hardware byte counters")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the per-frame transform runs on a single MI355X "
              "(frames of one stream are sequential); --gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    from paper_2502_20762_amd.ncodec import Codec

    if args.sweep:
        sweep(args.paths.split(","), args.steps, args.warmup, torch, Codec, args.sweep_match)
        return

    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    pre = synth.PRESETS["hd1080"]
    H, W, C, ne, nd = pre.height, pre.width, pre.channels, pre.n_enc, pre.n_dec
    weights = synth.make_weights(C, ne, nd)
    nfr = min(args.steps + args.warmup, pre.n_frames)
    frames = list(synth.frame_sequence(pre, nfr))
    gframes = [torch.from_numpy(f).to("cuda") for f in frames]
    torch.cuda.synchronize()

    kinds, enc_list, dec_list = workload_model(H, W, C, ne, nd)
    res = {}
    for path in args.paths.split(","):
        res[path] = run_path(path, pre, weights, gframes, args.steps, args.warmup, torch, Codec)

    def summary(path, r, peak_tflops, op_scale, unit):
        # the dominant kernel: one DC block per launch, or (at C = 256) one
        # chain of a transform's blocks per launch; the timing log counts
        # blocks either way
        chained = r["block_chains"]
        bpl = min(ne, nd, 16) if chained else 1
        kname = ("k_dcchain128_f16<false>" if chained else "k_dcblock128_f16<false>") if path == "fp16" \
            else ("k_dcchain128_i16" if chained else "k_dcblock128_i16")
        traffic = counted_traffic(kname)
        K = args.steps
        fl, by = kinds["dcblock"]
        if chained:  # a chain's algorithmic HBM bytes: its input and its output, once
            fl, by = bpl * fl, by
        kd = r["kernels"]["dcblock"]
        launch_us = kd["avg_us"] * bpl
        achieved = op_scale * fl / (launch_us * 1e-6) / 1e12
        t_roof = roofline_seconds(kinds, enc_list + dec_list, peak_tflops * 1e12 / op_scale)
        step_ms = (r["enc_ms"] + r["dec_ms"]) / K
        ga = r["graph"]
        return {
            "value": K / ((r["enc_ms"] + r["dec_ms"]) * 1e-3),
            "ms_per_step": step_ms,
            "encode_fps": K / (r["enc_ms"] * 1e-3),
            "decode_fps": K / (r["dec_ms"] * 1e-3),
            "encode_fps_median": 1e3 / r["enc_median_ms"],
            "decode_fps_median": 1e3 / r["dec_median_ms"],
            "graph_replay": {"value": K / ((ga["enc_ms"] + ga["dec_ms"]) * 1e-3),
                             "encode_fps": K / (ga["enc_ms"] * 1e-3), "decode_fps": K / (ga["dec_ms"] * 1e-3)},
            "roofline": {"kernel": kname, "bound": "mfma", "achieved": achieved, "peak": peak_tflops,
                         "unit": unit, "frac": achieved / peak_tflops, "traffic": traffic,
                         "per_launch": {"algorithmic_ops": op_scale * fl, "algorithmic_bytes": by,
                                        "avg_us": launch_us, "launches": kd["launches"] // bpl,
                                        "blocks_per_launch": bpl, "per_block_us": kd["avg_us"]}},
            "chain_timeouts": r["chain_timeouts"],
            "frame_roofline_fps": 1.0 / t_roof,
            "frac_of_frame_roofline": K / ((r["enc_ms"] + r["dec_ms"]) * 1e-3) * t_roof,
            "encode_frac_of_roofline": roofline_seconds(kinds, enc_list, peak_tflops * 1e12 / op_scale)
                                       / (r["enc_ms"] * 1e-3 / K),
            "decode_frac_of_roofline": roofline_seconds(kinds, dec_list, peak_tflops * 1e12 / op_scale)
                                       / (r["dec_ms"] * 1e-3 / K),
            "kernels_us": {k: round(v["avg_us"], 2) for k, v in r["kernels"].items()},
            "kernels_per_frame": r["kernels_per_frame"],
            "bits_per_frame": r["bits_per_frame"],
            "coded": r["coded"],
        }

    out = {"metric": METRIC}
    main_path = "fp16" if "fp16" in res else next(iter(res))
    s_main = summary(main_path, res[main_path], *(
        (MFMA_F16_PEAK_TFLOPS, 1, "TFLOP/s") if main_path == "fp16" else (MFMA_I8_PEAK_TOPS, 4, "TOP/s")))
    out.update({
        "value": s_main["value"], "unit": "frames/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": s_main["ms_per_step"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16" if main_path == "fp16" else "int16", "data": "synthetic",
        "config": {"workload": "1080p P-frame sequence, 1920x1088 (padded), C=256 at 1/8 scale (240x136), "
                               "8+8 DC blocks, latent 120x68x256; one step = encode + decode of one frame",
                   "height": H, "width": W, "channels": C, "n_enc_blocks": ne, "n_dec_blocks": nd,
                   "path": main_path},
        "encode_fps": s_main["encode_fps"], "decode_fps": s_main["decode_fps"],
        "encode_fps_median": s_main["encode_fps_median"], "decode_fps_median": s_main["decode_fps_median"],
        "launch_mode": "direct", "graph_replay": s_main["graph_replay"],
        "roofline": s_main["roofline"],
        "frame_roofline_fps": s_main["frame_roofline_fps"],
        "frac_of_frame_roofline": s_main["frac_of_frame_roofline"],
        "encode_frac_of_roofline": s_main["encode_frac_of_roofline"],
        "decode_frac_of_roofline": s_main["decode_frac_of_roofline"],
        "kernels_us": s_main["kernels_us"], "kernels_per_frame": s_main["kernels_per_frame"],
        "coded": s_main["coded"],
    })
    if "int16" in res and main_path != "int16":
        out["int16"] = summary("int16", res["int16"], MFMA_I8_PEAK_TOPS, 4, "TOP/s")
    if not args.no_gated:
        out["gated_block"] = {p: run_gated(p, pre, gframes, args.steps, args.warmup, torch, Codec)
                              for p in args.paths.split(",")}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(pre, weights, args.cpu_strip_rows, main_path)
        if "int16" in out:
            out["int16"]["cpu_baseline"] = cpu_baseline(pre, weights, args.cpu_strip_rows, "int16")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
