#!/usr/bin/env python3
"""Benchmark of the attention hot path on one MI355X.

Default workload: one mixed prefill/decode step with handoff (28 query heads,
4 KV heads, d 128, bf16):

  split-K paged decode of 192 requests, context lognormal(2048, 0.7) clipped
  to [64, 16384] -> varlen causal prefill over 8 x 512 fresh tokens -> paged
  KV write of those 4096 tokens -> handoff pack of the 8 prefilled requests
  (1 layer), in order on one stream (``--order prefill-first`` runs the
  decode after the write; ``--streams 2`` puts it on a second stream)

A "step" is one such launch set; K timed steps run back to back after W
warm-up steps.  Every kernel is bracketed by HIP events on the stream it runs
on.  The headline value is decode attention HBM throughput (algorithmic bytes /
decode kernel time); prefill TFLOP/s and the write/pack bandwidths are
reported beside it.  ``--workload`` selects the single-kernel workloads
(decode MHA 7B-shaped, varlen prefill + write, GQA decode 70B-shaped, chunked
prefill over the paged cache, the P->D handoff) for the per-workload tables;
``--kv fp8`` runs the decode workloads over E4M3 KV pages.

Prints ONE JSON line.
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

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = ("paper_2511_20982_amd/csrc/dopd_attn.hip",
                  "paper_2511_20982_amd/csrc/kernels/common.hpp",
                  "paper_2511_20982_amd/csrc/kernels/decode_bf16.hpp",
                  "paper_2511_20982_amd/csrc/kernels/prefill_bf16.hpp",
                  "paper_2511_20982_amd/csrc/kernels/kv_write.hpp",
                  "paper_2511_20982_amd/csrc/kernels/kv_pack.hpp",
                  "paper_2511_20982_amd/csrc/kernels/kv_unpack.hpp")
# Kernels behind each timed call (the decode call is a split kernel plus, when
# some context exceeds one split, a merge kernel; a chunk call with key splits
# adds the prefill merge kernel).
CALL_KERNELS = {"decode": ("decode_split_kernel", "decode_merge_kernel"),
                "prefill": ("prefill_bf16_kernel<128, false>", "prefill_bf16_kernel<64, false>"),
                "prefill_chunked": ("prefill_bf16_kernel<128, true>", "prefill_bf16_kernel<64, true>",
                                    "prefill_split_merge_kernel"),
                "kv_write": ("kv_write_kernel",),
                "pack": ("kv_pack_kernel",), "unpack": ("kv_unpack_kernel",)}

WORKLOADS = {
    "mixed": ("mixed P/D step + handoff: prefill 8x512, decode 192 req ctx lognormal(2048,0.7) "
              "[64,16384], 28/4 heads, d128, bf16, pack 8 req x 1 layer", 5),
    "decode_mha": ("decode, MHA 7B-shaped: B64, 32 heads, d128, bf16, ctx lognormal(1024,0.8) "
                   "[16,4096]", 2),
    "prefill": ("varlen causal prefill + paged write: 16 prompts lognormal(1500,1.0) [32,8192], "
                "32/32 heads, d128, bf16", 3),
    "decode_gqa": ("decode, GQA 70B-shaped: B256, 64/8 heads, d128, bf16, ctx 80% U[100,500] + "
                   "20% U[4096,16384]", 4),
    "chunked": ("chunked prefill over the paged cache: the 16 prompts of the varlen prefill "
                "workload (lognormal(1500,1.0) [32,8192], 32/32 heads, d128, bf16) in chunks of "
                "--chunk tokens, calls filled to --budget tokens, each chunk attending to its "
                "cached prefix", 3),
    "handoff": ("P->D handoff on one GPU: pack 8 prefilled requests x 512 tokens from the P pool, "
                "unpack into a D pool with another page order; 28/4 heads, d128, bf16, "
                "--pack-layers layers", 5),
}


# ------------------------------------------------------------------ algorithmic work
def decode_bytes(ctx, hq, hkv, d, s=2, kv_s=None):
    """K and V once (kv_s bytes per element), q and out (s bytes), page ids, lengths."""
    ctx = np.asarray(ctx, np.int64)
    b = len(ctx)
    kv_s = s if kv_s is None else kv_s
    return int((2 * hkv * d * ctx * kv_s).sum() + b * hq * d * 2 * s +
               (4 * ((ctx + 15) // 16)).sum() + 4 * b)


def prefill_flops(lens, hq, d):
    lens = np.asarray(lens, np.int64)
    return int((4 * d * hq * lens * (lens + 1) // 2).sum())


def write_bytes(lens, hkv, d, s=2, out_s=None):
    """K and V read (s bytes per element) and written (out_s bytes), page ids, lengths."""
    lens = np.asarray(lens, np.int64)
    t = int(lens.sum())
    out_s = s if out_s is None else out_s
    return int(2 * t * hkv * d * (s + out_s) + 4 * ((lens + 15) // 16).sum() + 8 * len(lens))


def pack_bytes(lens, layers, hkv, d, s=2):
    lens = np.asarray(lens, np.int64)
    return int(2 * (layers * 2 * hkv * lens * d * s).sum())


# ------------------------------------------------------------------ helpers
def source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def repeat_timed(fn, min_seconds):
    """Calls fn until at least min_seconds have passed (once at least); returns
    (first result, passes, seconds)."""
    t0 = time.time()
    res = fn()
    n = 1
    while time.time() - t0 < min_seconds:
        fn()
        n += 1
    return res, n, time.time() - t0


def load_traffic(workload, call):
    """HBM bytes per call from committed counter summaries, if the kernels are unchanged."""
    path = os.path.join(PROFILES, f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_hash") != source_hash() or call not in t.get("calls", {}):
        return None
    return t["calls"][call]["hbm_bytes_per_call"]


def summarize(args):
    """Turns rocprofv3 CSV output into the markdown/JSON summaries kept in profiles/."""
    import csv
    import glob
    from collections import defaultdict
    out = []
    stats = sorted(glob.glob(os.path.join(args.summarize, "**", "*kernel_stats.csv"), recursive=True))
    if stats:
        out.append(f"# rocprofv3 kernel statistics: {args.label}\n")
        out.append(f"Command: `{args.command}`\n")
        out.append("| kernel | calls | avg us | min us | max us | share |")
        out.append("|---|---|---|---|---|---|")
        for row in csv.DictReader(open(stats[0])):
            name = row["Name"][:90].replace("|", "/")
            out.append(f"| {name} | {row['Calls']} | {float(row['AverageNs']) / 1e3:.2f} | "
                       f"{float(row['MinNs']) / 1e3:.2f} | {float(row['MaxNs']) / 1e3:.2f} | "
                       f"{float(row['Percentage']):.1f}% |")
    pmc = sorted(glob.glob(os.path.join(args.summarize, "**", "*counter_collection.csv"),
                           recursive=True))
    if pmc:
        # per kernel name: list of per-dispatch counter sums
        per = defaultdict(lambda: defaultdict(list))
        for f in pmc:
            acc = defaultdict(float)
            names = {}
            for r in csv.DictReader(open(f)):
                key = (r["Dispatch_Id"], r["Counter_Name"])
                acc[key] += float(r["Counter_Value"])
                names[r["Dispatch_Id"]] = r["Kernel_Name"]
            for (disp, ctr), v in acc.items():
                per[names[disp]][ctr].append(v)
        copy_mib = args.copy_calib_mib
        factors = {}
        for kname, ctrs in per.items():
            if "neg_kernel" in kname:
                for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
                    if ctr in ctrs:
                        measured = float(np.median(ctrs[ctr]))  # KiB per dispatch
                        factors[ctr] = copy_mib * 1024.0 / measured if measured > 0 else None
        out.append(f"\n# rocprofv3 HBM counters (KiB per dispatch, median): {args.label}\n")
        out.append(f"`--pmc FETCH_SIZE` and `--pmc WRITE_SIZE` in separate runs.  Calibration: one "
                   f"elementwise kernel reading and writing {copy_mib} MiB in the same run; scale = "
                   f"known bytes / counter = {json.dumps(factors)}.\n")
        out.append("| kernel | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB |")
        out.append("|---|---|---|---|")
        calls = {}
        for kname, ctrs in sorted(per.items()):
            f_k = float(np.median(ctrs["FETCH_SIZE"])) if "FETCH_SIZE" in ctrs else float("nan")
            w_k = float(np.median(ctrs["WRITE_SIZE"])) if "WRITE_SIZE" in ctrs else float("nan")
            n = max(len(ctrs.get("FETCH_SIZE", [])), len(ctrs.get("WRITE_SIZE", [])))
            out.append(f"| {kname[:90]} | {n} | {f_k:.0f} | {w_k:.0f} |")
            for call, kernels in CALL_KERNELS.items():
                if any(k in kname for k in kernels):
                    c = calls.setdefault(call, {"fetch_kib": 0.0, "write_kib": 0.0, "kernels": []})
                    c["fetch_kib"] += f_k
                    c["write_kib"] += w_k
                    c["kernels"].append(kname)
        for call, c in calls.items():
            ff, fw = factors.get("FETCH_SIZE") or 1.0, factors.get("WRITE_SIZE") or 1.0
            c["hbm_bytes_per_call"] = int(1024 * (c["fetch_kib"] * ff + c["write_kib"] * fw))
        tr = {"workload": args.label, "source_hash": source_hash(), "copy_factors": factors,
              "calls": calls, "command": args.command}
        with open(os.path.join(args.traffic_dir, f"traffic_{args.label}.json"), "w") as f:
            json.dump(tr, f, indent=1)
        out.append("\nHBM bytes per call (scaled): " +
                   ", ".join(f"{k}: {v['hbm_bytes_per_call'] / 1e6:.1f} MB" for k, v in calls.items()))
    text = "\n".join(out) + "\n"
    with open(args.summary_out, "w") as f:
        f.write(text)
    print(text)


def cpu_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model


class Timer:
    """HIP events around a call on a given stream, accumulated over steps."""

    def __init__(self, torch, stream):
        self.torch, self.stream, self.pairs = torch, stream, []

    def __enter__(self):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record(self.stream)
        self.pairs.append([e, None])
        return self

    def __exit__(self, *exc):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record(self.stream)
        self.pairs[-1][1] = e

    def avg_us(self, skip=0):
        ts = [a.elapsed_time(b) * 1e3 for a, b in self.pairs[skip:]]
        return float(np.mean(ts)) if ts else float("nan")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="mixed")
    ap.add_argument("--pack-layers", type=int, default=1,
                    help="layers packed per handoff in the mixed step (1 = the configured step)")
    ap.add_argument("--split", type=int, default=0, help="decode split tokens (0 = automatic)")
    ap.add_argument("--chunk", type=int, default=512, help="chunked workload: tokens per chunk")
    ap.add_argument("--budget", type=int, default=8192,
                    help="chunked workload: tokens per call (chunks of several prompts)")
    ap.add_argument("--splits", type=int, default=0,
                    help="chunked workload: key splits per call (0 = automatic, 1 = none)")
    ap.add_argument("--order", choices=("decode-first", "prefill-first"), default="decode-first",
                    help="mixed step on one stream: the decode batch before the prefill, write "
                         "and pack (its tokens are the TPOT-bound ones), or after the write")
    ap.add_argument("--streams", type=int, default=1, choices=(1, 2),
                    help="mixed step: 2 = decode on its own stream beside prefill/write/pack, "
                         "1 = everything in order on one stream")
    ap.add_argument("--kv", choices=("bf16", "fp8"), default="bf16",
                    help="KV cache element type (fp8 = E4M3 pages with per-KV-head scales): "
                         "decode workloads read it (written by the fp8 writer before timing), "
                         "the prefill workload writes it")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="after timing, run one device copy of this size (counter calibration)")
    ap.add_argument("--summarize", default=None,
                    help="summarise a rocprofv3 output directory instead of benchmarking")
    ap.add_argument("--label", default="mixed")
    ap.add_argument("--command", default="")
    ap.add_argument("--summary-out", default=None)
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="host time the oracle baseline is timed over (passes repeat)")
    ap.add_argument("--traffic-dir", default=PROFILES,
                    help="where --summarize writes traffic_<label>.json")
    args = ap.parse_args()
    if args.summarize:
        summarize(args)
        return

    if args.kv == "fp8" and args.workload not in ("decode_mha", "decode_gqa", "prefill"):
        print("--kv fp8 applies to the decode_mha, decode_gqa and prefill workloads",
              file=sys.stderr)
        sys.exit(2)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the hot path is measured on a single MI355X; "
              "--gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2511_20982_amd import attn as A
    from paper_2511_20982_amd import inputs as I

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    A.lib()  # fail loudly if the HIP library is not built

    desc, cfg = WORKLOADS[args.workload]
    t0 = time.time()
    w = {5: lambda: I.config5(num_layers=args.pack_layers), 2: I.config2, 3: I.config3,
         4: I.config4}[cfg]()
    gen_s = time.time() - t0
    dev = "cuda"
    shape = A.make_shape(w.hq, w.hkv, w.d, w.dtype, w.scale)
    sA = torch.cuda.current_stream()
    sB = torch.cuda.Stream()  # default priority

    kern = {}
    if args.workload in ("mixed",):
        L = args.pack_layers
        # paged pools: layer 0 is the attention layer; extra layers only widen the pack
        kp_np, vp_np = w.k_pool, w.v_pool
        kp = torch.empty((L,) + kp_np.shape, dtype=torch.bfloat16, device=dev)
        vp = torch.empty((L,) + vp_np.shape, dtype=torch.bfloat16, device=dev)
        kp[0].copy_(A.to_device(kp_np))
        vp[0].copy_(A.to_device(vp_np))
        for layer in range(1, L):
            kp[layer].copy_(kp[0])
            vp[layer].copy_(vp[0])
        pt = A.to_device(w.page_table)
        stride = w.page_table.shape[1]
        pre_pt = pt[w.prefill_rows[0]:]  # rows of the prefill requests
        q, k, v = A.to_device(w.q), A.to_device(w.k), A.to_device(w.v)
        cu = A.to_device(w.cu_seqlens)
        out_p = torch.empty_like(q)
        n_pre = len(w.prefill_lens)
        start = torch.zeros(n_pre, dtype=torch.int32, device=dev)
        n_dec = len(w.context_lens)
        q_dec = A.to_device(w.q_dec)
        ctx = A.to_device(w.context_lens)
        out_d = torch.empty_like(q_dec)
        ws = A.decode_workspace(shape, w.context_lens, n_dec, args.split)
        offs_np = I.handoff_offsets(w.handoff_lens, L, w.hkv, w.d)
        offs = A.to_device(offs_np)
        hreq, hlen = A.to_device(w.handoff_reqs), A.to_device(w.handoff_lens)
        out_h = torch.empty(int(offs_np[-1]), dtype=torch.bfloat16, device=dev)
        T = int(w.cu_seqlens[-1])
        tm = {n: Timer(torch, s) for n, s in
              (("prefill", sA), ("kv_write", sA), ("pack", sA), ("decode", sB))}
        ev_join = torch.cuda.Event()

        sD = sB if args.streams == 2 else sA
        if args.streams == 1:
            tm["decode"] = Timer(torch, sA)

        dec_first = args.streams == 1 and args.order == "decode-first"

        def decode_call():
            with tm["decode"]:
                A.dopd_decode_attn(shape, q_dec, kp[0], vp[0], w.num_pages, pt, stride, ctx,
                                   w.context_lens, n_dec, args.split, out_d, None, ws,
                                   stream=sD)

        def step():
            # Two streams: the prefill is enqueued first, so its large workgroups
            # are dispatched before the decode work items fill the machine.
            if args.streams == 2:
                sB.wait_stream(sA)
            if dec_first:
                decode_call()
            with tm["prefill"]:
                A.dopd_prefill_attn(shape, q, k, v, out_p, None, cu, w.cu_seqlens, n_pre, stream=sA)
            if args.streams == 2:
                decode_call()
            with tm["kv_write"]:
                A.dopd_kv_write(shape, k, v, kp[0], vp[0], w.num_pages, pre_pt, stride, cu, start,
                                n_pre, T, sA)
            if args.streams == 1 and not dec_first:
                decode_call()
            with tm["pack"]:
                A.dopd_kv_pack_for_handoff(shape, L, kp, vp, w.num_pages, pt, stride, hreq, hlen,
                                           w.handoff_lens, offs, n_pre, out_h, sA)
            if args.streams == 2:
                ev_join.record(sB)
                sA.wait_event(ev_join)

        work = {
            "decode": ("GB/s", decode_bytes(w.context_lens, w.hq, w.hkv, w.d)),
            "prefill": ("TFLOP/s", prefill_flops(w.prefill_lens, w.hq, w.d)),
            "kv_write": ("GB/s", write_bytes(w.prefill_lens, w.hkv, w.d)),
            "pack": ("GB/s", pack_bytes(w.handoff_lens, L, w.hkv, w.d)),
        }
        dominant = "decode"
    elif args.workload in ("decode_mha", "decode_gqa"):
        kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
        pt = A.to_device(w.page_table)
        q_dec = A.to_device(w.q_dec)
        ctx = A.to_device(w.context_lens)
        out_d = torch.empty_like(q_dec)
        n_dec = len(w.context_lens)
        ws = A.decode_workspace(shape, w.context_lens, n_dec, args.split)
        tm = {"decode": Timer(torch, sA)}
        if args.kv == "fp8":
            # The cache as a prefill would leave it: token-major K/V of every
            # cached token (gathered from the bf16 pools), one scale per KV head
            # from its absolute maximum, written by the fp8 writer (untimed).
            shape8 = A.make_shape(w.hq, w.hkv, w.d, "fp8", w.scale)
            cl = w.context_lens.astype(np.int64)
            r_idx = np.repeat(np.arange(n_dec), cl)
            j = np.arange(int(cl.sum())) - np.repeat(np.cumsum(cl) - cl, cl)
            pg = torch.from_numpy(w.page_table[r_idx, j // 16].astype(np.int64)).to(dev)
            sl = torch.from_numpy((j % 16).astype(np.int64)).to(dev)
            ktok = kp[pg, :, sl, :].contiguous()          # [T][Hkv][d]
            vtok = vp[pg, :, :, sl].contiguous()          # [T][Hkv][d]
            ks = (ktok.abs().amax(dim=(0, 2)).float() / 448.0).contiguous()
            vs = (vtok.abs().amax(dim=(0, 2)).float() / 448.0).contiguous()
            kp8 = torch.full((w.num_pages, w.hkv, 16, w.d), 0x7F, dtype=torch.uint8, device=dev)
            vp8 = torch.full((w.num_pages, w.hkv, w.d, 16), 0x7F, dtype=torch.uint8, device=dev)
            ws = A.decode_workspace(shape8, w.context_lens, n_dec, args.split)
            cu_t = A.to_device(I.cu_from_lens(w.context_lens))
            A.dopd_kv_write_fp8(shape8, ktok, vtok, ks, vs, kp8, vp8, w.num_pages, pt,
                                w.page_table.shape[1], cu_t,
                                torch.zeros(n_dec, dtype=torch.int32, device=dev), n_dec,
                                int(cl.sum()), sA)
            torch.cuda.synchronize()
            del ktok, vtok, kp, vp

            def step():
                with tm["decode"]:
                    A.dopd_decode_attn_fp8(shape8, q_dec, kp8, vp8, ks, vs, w.num_pages, pt,
                                           w.page_table.shape[1], ctx, w.context_lens, n_dec,
                                           args.split, out_d, None, ws, stream=sA)

            work = {"decode": ("GB/s", decode_bytes(w.context_lens, w.hq, w.hkv, w.d, kv_s=1))}
        else:
            def step():
                with tm["decode"]:
                    A.dopd_decode_attn(shape, q_dec, kp, vp, w.num_pages, pt,
                                       w.page_table.shape[1], ctx, w.context_lens, n_dec,
                                       args.split, out_d, None, ws, stream=sA)

            work = {"decode": ("GB/s", decode_bytes(w.context_lens, w.hq, w.hkv, w.d))}
        dominant = "decode"
    elif args.workload == "handoff":
        L = args.pack_layers
        n_dec, n_pre = len(w.context_lens), len(w.prefill_lens)
        kp = torch.empty((L,) + w.k_pool.shape, dtype=torch.bfloat16, device=dev)
        vp = torch.empty((L,) + w.v_pool.shape, dtype=torch.bfloat16, device=dev)
        kp[0].copy_(A.to_device(w.k_pool))
        vp[0].copy_(A.to_device(w.v_pool))
        pt = A.to_device(w.page_table)
        stride = w.page_table.shape[1]
        # fill the prefilled requests' pages (untimed), then replicate the layer
        A.dopd_kv_write(shape, A.to_device(w.k), A.to_device(w.v), kp[0], vp[0], w.num_pages,
                        pt[n_dec:], stride, A.to_device(w.cu_seqlens),
                        torch.zeros(n_pre, dtype=torch.int32, device=dev), n_pre,
                        int(w.cu_seqlens[-1]))
        for layer in range(1, L):
            kp[layer].copy_(kp[0])
            vp[layer].copy_(vp[0])
        # receiving pool: same requests, another random page order
        pt_d_np, pages_d = I.allocate_pages(np.random.default_rng(w.seed + 1000), w.handoff_lens)
        kd = torch.zeros((L, pages_d, w.hkv, 16, w.d), dtype=torch.bfloat16, device=dev)
        vd = torch.zeros((L, pages_d, w.hkv, w.d, 16), dtype=torch.bfloat16, device=dev)
        pt_d = A.to_device(pt_d_np)
        offs_np = I.handoff_offsets(w.handoff_lens, L, w.hkv, w.d)
        offs = A.to_device(offs_np)
        hreq, hlen = A.to_device(w.handoff_reqs), A.to_device(w.handoff_lens)
        dreq = torch.arange(n_pre, dtype=torch.int32, device=dev)
        buf = torch.empty(int(offs_np[-1]), dtype=torch.bfloat16, device=dev)
        tm = {"pack": Timer(torch, sA), "unpack": Timer(torch, sA)}

        def step():
            with tm["pack"]:
                A.dopd_kv_pack_for_handoff(shape, L, kp, vp, w.num_pages, pt, stride, hreq, hlen,
                                           w.handoff_lens, offs, n_pre, buf, sA)
            with tm["unpack"]:
                A.dopd_kv_unpack_from_handoff(shape, L, buf, offs, dreq, hlen, w.handoff_lens,
                                              n_pre, kd, vd, pages_d, pt_d, pt_d_np.shape[1], sA)

        work = {"pack": ("GB/s", pack_bytes(w.handoff_lens, L, w.hkv, w.d)),
                "unpack": ("GB/s", pack_bytes(w.handoff_lens, L, w.hkv, w.d))}
        dominant = "unpack"
    elif args.workload == "chunked":
        # All K/V go into the paged cache first (one timed write).  Then the
        # prompts are prefilled in chunks of C tokens, each attending to its
        # cached prefix: a call takes the next chunk of the prompts in turn until
        # it holds `budget` tokens (a chunked-prefill batch), calls back to back.
        C, B = args.chunk, args.budget
        lens = w.prefill_lens.astype(np.int64)
        k, v = A.to_device(w.k), A.to_device(w.v)
        cu = A.to_device(w.cu_seqlens)
        kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
        pt_np = w.page_table
        stride = pt_np.shape[1]
        n_pre = len(lens)
        start = torch.zeros(n_pre, dtype=torch.int32, device=dev)
        T = int(w.cu_seqlens[-1])
        q_all = A.to_device(w.q)
        out_all = torch.empty_like(q_all)
        pos = np.zeros(n_pre, np.int64)
        chunks = []
        while (pos < lens).any():
            sel = []  # (request, start, n)
            budget = B
            for r in np.argsort(-(lens - pos), kind="stable"):
                if budget <= 0:
                    break
                n = int(min(C, lens[r] - pos[r], budget))
                if n > 0:
                    sel.append((int(r), int(pos[r]), n))
                    pos[r] += n
                    budget -= n
            n_arr = np.array([x[2] for x in sel], np.int32)
            pre = np.array([x[1] for x in sel], np.int32)
            rows = np.concatenate([w.cu_seqlens[r] + s0 + np.arange(n) for r, s0, n in sel])
            rows_d = torch.from_numpy(rows.astype(np.int64)).to(dev)
            cu_c = I.cu_from_lens(n_arr)
            pt_c = np.ascontiguousarray(pt_np[[x[0] for x in sel]])
            chunks.append(dict(q=q_all.index_select(0, rows_d).contiguous(), rows=rows_d,
                               out=torch.empty((len(rows), w.hq, w.d), dtype=torch.bfloat16,
                                               device=dev),
                               cu=A.to_device(cu_c), cu_h=cu_c, pre=A.to_device(pre), pre_h=pre,
                               pt=A.to_device(pt_c), n=len(sel)))
        pt = A.to_device(pt_np)
        # One workspace serves every call (they run in order on one stream);
        # thin calls split their keys over several workgroups.
        ws_bytes = max(A.dopd_prefill_paged_workspace_size(shape, ch["cu_h"], ch["pre_h"], ch["n"],
                                                           args.splits) for ch in chunks)
        ws_buf = torch.empty(ws_bytes + 256, dtype=torch.uint8, device=dev)
        ws = ws_buf[(-ws_buf.data_ptr()) % 256:][:ws_bytes]
        tm = {"prefill_chunked": Timer(torch, sA), "kv_write": Timer(torch, sA)}

        def step():
            with tm["kv_write"]:
                A.dopd_kv_write(shape, k, v, kp, vp, w.num_pages, pt, stride, cu, start, n_pre, T,
                                sA)
            with tm["prefill_chunked"]:
                for ch in chunks:
                    A.dopd_prefill_paged_attn_split(shape, ch["q"], kp, vp, w.num_pages,
                                                    ch["pt"], stride, ch["cu"], ch["cu_h"],
                                                    ch["pre"], ch["pre_h"], ch["n"], args.splits,
                                                    ch["out"], None, ws, ws_bytes, sA)

        def gather_out():
            for ch in chunks:
                out_all.index_copy_(0, ch["rows"], ch["out"])
            return out_all

        work = {"prefill_chunked": ("TFLOP/s", prefill_flops(w.prefill_lens, w.hq, w.d)),
                "kv_write": ("GB/s", write_bytes(w.prefill_lens, w.hkv, w.d))}
        dominant = "prefill_chunked"
    else:  # prefill + write
        q, k, v = A.to_device(w.q), A.to_device(w.k), A.to_device(w.v)
        cu = A.to_device(w.cu_seqlens)
        out_p = torch.empty_like(q)
        kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
        pt = A.to_device(w.page_table)
        n_pre = len(w.prefill_lens)
        start = torch.zeros(n_pre, dtype=torch.int32, device=dev)
        T = int(w.cu_seqlens[-1])
        tm = {"prefill": Timer(torch, sA), "kv_write": Timer(torch, sA)}
        if args.kv == "fp8":
            # The prompts' K/V go to an E4M3 cache (scales from each head's
            # absolute maximum over the batch).
            shape8 = A.make_shape(w.hq, w.hkv, w.d, "fp8", w.scale)
            ks = (k.abs().amax(dim=(0, 2)).float() / 448.0).contiguous()
            vs = (v.abs().amax(dim=(0, 2)).float() / 448.0).contiguous()
            kp = torch.full((w.num_pages, w.hkv, 16, w.d), 0x7F, dtype=torch.uint8, device=dev)
            vp = torch.full((w.num_pages, w.hkv, w.d, 16), 0x7F, dtype=torch.uint8, device=dev)

            def write():
                A.dopd_kv_write_fp8(shape8, k, v, ks, vs, kp, vp, w.num_pages, pt,
                                    w.page_table.shape[1], cu, start, n_pre, T, sA)
            wbytes = write_bytes(w.prefill_lens, w.hkv, w.d, out_s=1)
        else:
            def write():
                A.dopd_kv_write(shape, k, v, kp, vp, w.num_pages, pt, w.page_table.shape[1], cu,
                                start, n_pre, T, sA)
            wbytes = write_bytes(w.prefill_lens, w.hkv, w.d)

        def step():
            with tm["prefill"]:
                A.dopd_prefill_attn(shape, q, k, v, out_p, None, cu, w.cu_seqlens, n_pre, stream=sA)
            with tm["kv_write"]:
                write()

        work = {"prefill": ("TFLOP/s", prefill_flops(w.prefill_lens, w.hq, w.d)),
                "kv_write": ("GB/s", wbytes)}
        dominant = "prefill"

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    for t in tm.values():
        t.pairs.clear()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(sA)
    for _ in range(args.steps):
        step()
    ev1.record(sA)
    torch.cuda.synchronize()
    ms_step = ev0.elapsed_time(ev1) / args.steps

    for name, t in tm.items():
        unit, amount = work[name]
        us = t.avg_us()
        rate = amount / (us * 1e-6) / (1e12 if unit == "TFLOP/s" else 1e9)
        peak = BF16_PEAK_TFLOPS if unit == "TFLOP/s" else HBM_PEAK_GBS
        kern[name] = {"avg_us": round(us, 2), "rate": round(rate, 2), "unit": unit,
                      "frac": round(rate / peak, 4),
                      ("flops" if unit == "TFLOP/s" else "bytes"): amount}

    if args.copy_calib_mib:
        # A shader kernel of known traffic (reads and writes N MiB once), used to
        # scale the HBM counters; a plain device copy would go to a DMA engine.
        src = torch.ones(args.copy_calib_mib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    dk = kern[dominant]
    roofline = {"kernel": dominant, "kernels": list(CALL_KERNELS[dominant]),
                "bound": "mfma" if dk["unit"] == "TFLOP/s" else "hbm",
                "achieved": dk["rate"], "peak": BF16_PEAK_TFLOPS if dk["unit"] == "TFLOP/s" else HBM_PEAK_GBS,
                "unit": dk["unit"], "frac": dk["frac"],
                "traffic": load_traffic(args.workload + ("_fp8" if args.kv == "fp8" else ""),
                                        dominant)}

    # ---- CPU baseline: the fp64 oracle on host cores, plus a parity spot check
    cpu = None
    parity = None
    if not args.no_cpu_baseline and args.workload != "handoff":
        import oracle
        threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
        os.environ.setdefault("OMP_NUM_THREADS", str(threads))
        if dominant == "decode" and args.kv == "fp8":
            # The oracle quantises the bf16 cache itself (same scales, its own
            # encoder) and decodes the whole batch over its codes.
            ks_h, vs_h = ks.cpu().numpy(), vs.cpu().numpy()
            P, hkv, d = w.num_pages, w.hkv, w.d
            kq = oracle.e4m3_quantize(w.k_pool.transpose(0, 2, 1, 3).reshape(-1, hkv, d), ks_h)
            vq = oracle.e4m3_quantize(w.v_pool.transpose(0, 3, 1, 2).reshape(-1, hkv, d), vs_h)
            kq = kq.reshape(P, 16, hkv, d).transpose(0, 2, 1, 3).copy()
            vq = vq.reshape(P, 16, hkv, d).transpose(0, 2, 3, 1).copy()
            (ref, _), n, dt = repeat_timed(
                lambda: oracle.decode_e4m3(w.q_dec, kq, vq, ks_h, vs_h, w.page_table,
                                           w.context_lens, w.scale), args.cpu_seconds)
            amount = work["decode"][1]
            cpu = {"value": round(n * amount / dt / 1e9, 4), "unit": "GB/s", "cores": threads,
                   "kind": "oracle", "cpu": cpu_info(), "seconds": round(dt, 2),
                   "sample": f"fp64 oracle decode over E4M3 pages of the whole batch "
                             f"({len(w.context_lens)} requests, {amount / 1e9:.3f} GB algorithmic), "
                             f"{n} passes"}
            gotf = I.bf16_bits_to_f32(A.to_host(out_d)).astype(np.float64)
            parity = {"decode_max_abs_err": float(np.max(np.abs(gotf - ref))),
                      "decode_rows": int(ref.shape[0] * ref.shape[1]),
                      "kv": "fp8 pages from the GPU writer; oracle quantised the same bf16 cache"}
        elif dominant == "decode":
            # The whole decode batch of the step (about a second of host work).
            (ref, _), n, dt = repeat_timed(
                lambda: oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table,
                                      w.context_lens, w.scale), args.cpu_seconds)
            amount = decode_bytes(w.context_lens, w.hq, w.hkv, w.d)
            cpu = {"value": round(n * amount / dt / 1e9, 4), "unit": "GB/s", "cores": threads,
                   "kind": "oracle", "cpu": cpu_info(), "seconds": round(dt, 2),
                   "sample": f"fp64 oracle decode of the whole batch ({len(w.context_lens)} "
                             f"requests, {amount / 1e9:.3f} GB algorithmic), {n} passes"}
            gotf = I.bf16_bits_to_f32(A.to_host(out_d)).astype(np.float64)
            parity = {"decode_max_abs_err": float(np.max(np.abs(gotf - ref))),
                      "decode_rows": int(ref.shape[0] * ref.shape[1])}
            if "prefill" in kern:
                (ref_p, _), n_p, dtp = repeat_timed(
                    lambda: oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale),
                    args.cpu_seconds)
                cpu["prefill_tflops"] = round(n_p * work["prefill"][1] / dtp / 1e12, 6)
                cpu["prefill_seconds"] = round(dtp, 2)
                cpu["sample"] += (f"; fp64 oracle prefill of the whole prefill batch, {n_p} passes "
                                  f"({dtp:.1f} s)")
                gotp = I.bf16_bits_to_f32(A.to_host(out_p)).astype(np.float64)
                parity["prefill_max_abs_err"] = float(np.max(np.abs(gotp - ref_p)))
        else:
            # Bounded sample: the last 4 rows of every prompt (the longest rows), per head.
            rows_tok = np.concatenate([w.cu_seqlens[1:] - 1 - i for i in range(4)])
            rows_tok = np.repeat(rows_tok, 4)
            heads = (np.arange(len(rows_tok)) * 7) % w.hq
            (ref, _), n, dt = repeat_timed(
                lambda: oracle.prefill_rows(w.q, w.k, w.v, w.cu_seqlens, w.scale, rows_tok, heads),
                args.cpu_seconds)
            req_of = np.searchsorted(w.cu_seqlens, rows_tok, side="right") - 1
            pos = rows_tok - w.cu_seqlens[req_of]
            flops = int((4 * w.d * (pos + 1)).sum())
            cpu = {"value": round(n * flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": threads,
                   "kind": "oracle", "cpu": cpu_info(), "seconds": round(dt, 2),
                   "sample": f"fp64 oracle prefill of {len(rows_tok)} sampled rows (the last 4 "
                             f"rows of every prompt, 4 heads each; {flops / 1e9:.2f} GFLOP), "
                             f"{n} passes"
                             + ("; chunked output checked against the one-shot oracle rows"
                                if args.workload == "chunked" else "")}
            out_rows = gather_out() if args.workload == "chunked" else out_p
            gotf = I.bf16_bits_to_f32(A.to_host(out_rows)[rows_tok, heads]).astype(np.float64)
            parity = {"prefill_max_abs_err": float(np.max(np.abs(gotf - ref))),
                      "prefill_rows": int(len(rows_tok))}

    value = kern[dominant]["rate"]
    line = {
        "metric": "decode attn HBM GB/s (% peak) + prefill attn TFLOP/s (% MFMA peak)",
        "value": value,
        "unit": kern[dominant]["unit"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": desc + (", KV cache E4M3 with per-KV-head scales"
                                       if args.kv == "fp8" else ""),
                   "seed": int(w.seed), "split_tokens": args.split, "kv": args.kv,
                   "streams": args.streams if args.workload == "mixed" else 1,
                   "order": args.order if args.workload == "mixed" and args.streams == 1 else None,
                   "pack_layers": args.pack_layers if args.workload in ("mixed", "handoff") else None,
                   "chunk": args.chunk if args.workload == "chunked" else None,
                   "budget": args.budget if args.workload == "chunked" else None},
        "roofline": roofline,
        "kernels": kern,
        "cpu_baseline": cpu,
        "parity": parity,
        "input_gen_s": round(gen_s, 1),
    }
    if "prefill" in kern and dominant != "prefill":
        line["prefill_tflops"] = kern["prefill"]["rate"]
        line["prefill_mfma_frac"] = kern["prefill"]["frac"]
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
