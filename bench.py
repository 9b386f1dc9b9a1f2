#!/usr/bin/env python3
"""Benchmark of the attention hot path on one MI355X.

Headline workload: one mixed prefill/decode step with handoff (28 query heads,
4 KV heads, d 128, bf16), in order on one stream:

  split-K paged decode of 192 requests, context lognormal(2048, 0.7) clipped
  to [64, 16384] -> varlen causal prefill over 8 x 512 fresh tokens -> paged
  KV write of those 4096 tokens -> handoff pack of the 8 prefilled requests
  (1 layer)  (``--order prefill-first`` runs the decode after the write)

A "step" is one such launch set.  W warm-up steps, then K timed steps back to
back (ms_per_step), then --reps cold reps, each after a flush of L2 and the
MALL (write 1 GiB, read another 1 GiB; outside the timed region), and as many
warm reps.  Every C-ABI call is bracketed by HIP events on the stream it runs
on; the per-call tables give median, p10 and p90.  The headline value is the
decode call's algorithmic HBM bytes over its cold median.  After the headline,
the same step as one PD-aggregated launch (``pd_step``), the step's write and
pack as separate calls and as one pass (``write_pack``), and the decode MHA
7B-shaped, varlen prefill + paged write and GQA 70B-shaped decode workloads
are measured the same way (``configs``), each with its own oracle baseline on
the host cores.  ``--workload`` selects any single workload
(also the chunked prefill over the paged cache and the P->D handoff);
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
                  "paper_2511_20982_amd/csrc/plan.hpp",
                  "paper_2511_20982_amd/csrc/kernels/kv_write_pack.hpp",
                  "paper_2511_20982_amd/csrc/kernels/pd_step.hpp",
                  "paper_2511_20982_amd/csrc/kernels/common.hpp",
                  "paper_2511_20982_amd/csrc/kernels/attn_f32.hpp",
                  "paper_2511_20982_amd/csrc/kernels/decode_bf16.hpp",
                  "paper_2511_20982_amd/csrc/kernels/prefill_bf16.hpp",
                  "paper_2511_20982_amd/csrc/kernels/kv_write.hpp",
                  "paper_2511_20982_amd/csrc/kernels/kv_pack.hpp",
                  "paper_2511_20982_amd/csrc/kernels/kv_unpack.hpp")
# Kernels behind each timed call (the decode call is a split kernel plus, when
# some (request, KV head) spans two slices, one of the two merge kernels; a
# chunk call with key splits adds the prefill merge kernel).
CALL_KERNELS = {"decode": ("decode_split_kernel", "decode_merge_list_kernel",
                           "decode_merge_kernel"),
                "prefill": ("prefill_bf16_kernel<128, false, false>",
                            "prefill_bf16_kernel<64, false, false>"),
                "prefill_chunked": ("prefill_bf16_kernel<128, true, false>",
                                    "prefill_bf16_kernel<64, true, false>",
                                    "prefill_split_merge_kernel"),
                "prefill_chunked_fp8": ("prefill_bf16_kernel<128, true, true>",
                                        "prefill_bf16_kernel<64, true, true>",
                                        "prefill_split_merge_kernel"),
                "kv_write": ("kv_write_kernel",), "kv_write_fp8": ("kv_write_e4m3_kernel",),
                "plain_copy": ("bitwise_not_kernel",),
                "pack": ("kv_pack_kernel",), "unpack": ("kv_unpack_kernel",),
                "pd_step": ("pd_step_kernel", "decode_merge_list_kernel",
                            "decode_merge_kernel"),
                "kv_write_pack": ("kv_write_pack_kernel",)}

WORKLOADS = {
    "mixed": ("mixed P/D step + handoff: prefill 8x512, decode 192 req ctx lognormal(2048,0.7) "
              "[64,16384], 28/4 heads, d128, bf16, pack 8 req x 1 layer", "mixed_step"),
    "decode_mha": ("decode, MHA 7B-shaped: B64, 32 heads, d128, bf16, ctx lognormal(1024,0.8) "
                   "[16,4096]", "decode_mha_7b"),
    "prefill": ("varlen causal prefill + paged write: 16 prompts lognormal(1500,1.0) [32,8192], "
                "32/32 heads, d128, bf16", "varlen_prefill"),
    "decode_gqa": ("decode, GQA 70B-shaped: B256, 64/8 heads, d128, bf16, ctx 80% U[100,500] + "
                   "20% U[4096,16384]", "decode_gqa_70b"),
    "chunked": ("chunked prefill over the paged cache: the 16 prompts of the varlen prefill "
                "workload (lognormal(1500,1.0) [32,8192], 32/32 heads, d128, bf16) in chunks of "
                "--chunk tokens, calls filled to --budget tokens, each chunk attending to its "
                "cached prefix; --kv fp8: the prompts written to an E4M3 cache and the chunks "
                "read from it", "varlen_prefill"),
    "pd_step": ("the mixed P/D step + handoff of the mixed workload as one PD-aggregated launch "
                "(dopd_pd_step: decode slices, prefill items and write+pack workgroups in one "
                "grid, then the decode merge); --kv fp8: over E4M3 pages (dopd_pd_step_fp8)",
                "mixed_step"),
    "write_pack": ("paged write + handoff pack of the mixed step's 8 x 512 fresh prompts (28/4 "
                   "heads, d128, bf16, 1 layer): the separate write and pack calls, then the "
                   "one-pass write+pack (dopd_kv_write_pack_for_handoff), and a plain "
                   "elementwise kernel moving the pack's bytes (the floor at this size)",
                   "mixed_step"),
    "handoff": ("P->D handoff on one GPU: pack 8 prefilled requests x 512 tokens from the P pool, "
                "unpack into a D pool with another page order; 28/4 heads, d128, bf16, "
                "--pack-layers layers", "mixed_step"),
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


def write_pack_bytes(lens, hkv, d, s=2):
    """K and V read once, written to the pages and to the handoff buffer; page ids, lengths."""
    lens = np.asarray(lens, np.int64)
    t = int(lens.sum())
    return int(2 * t * hkv * d * 3 * s + 4 * ((lens + 15) // 16).sum() + 8 * len(lens) +
               8 * len(lens))


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
def e4m3_head_scales(x) -> np.ndarray:
    """One E4M3 scale per KV head of bf16 x[T][Hkv][d]: its absolute maximum
    over the tokens and dims / 448 (the largest finite E4M3 value), in fp32."""
    a = np.abs((np.asarray(x, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32))
    a = a.max(axis=(0, 2))
    return (a / np.float32(448)).astype(np.float32)


def json_safe(x):
    """The record with non-finite floats as null (strict JSON)."""
    if isinstance(x, dict):
        return {k: json_safe(v) for k, v in x.items()}
    if isinstance(x, (list, tuple)):
        return [json_safe(v) for v in x]
    if isinstance(x, float) and not np.isfinite(x):
        return None
    return x


def mean_or_none(xs):
    """Mean of a list of times in us (None when empty: no back-to-back steps)."""
    return round(float(np.mean(xs)), 2) if len(xs) else None


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
        out.append(f"Kernel sources: {source_hash()}\n")
        out.append("| kernel | calls | avg us | min us | max us | share |")
        out.append("|---|---|---|---|---|---|")
        rows = list(csv.DictReader(open(stats[0])))
        for row in rows:
            name = row["Name"][:90].replace("|", "/")
            out.append(f"| {name} | {row['Calls']} | {float(row['AverageNs']) / 1e3:.2f} | "
                       f"{float(row['MinNs']) / 1e3:.2f} | {float(row['MaxNs']) / 1e3:.2f} | "
                       f"{float(row['Percentage']):.1f}% |")
        # Kernel time per C-ABI call: the kernels of the call, each weighted by
        # its launches per launch of the call's first kernel.
        kcalls = {}
        for call, kernels in CALL_KERNELS.items():
            # a call is present when its first kernel ran (the others it may add
            # are shared with other calls: the decode merge kernel)
            if not any(kernels[0] in r["Name"] for r in rows):
                continue
            match = [r for r in rows if any(k in r["Name"] for k in kernels)]
            first = next(r for k in kernels for r in match if k in r["Name"])
            n_calls = float(first["Calls"])
            us = sum(float(r["AverageNs"]) * float(r["Calls"]) for r in match) / n_calls / 1e3
            kcalls[call] = {"avg_us": round(us, 3), "calls": int(n_calls),
                            "kernels": [r["Name"][:90] for r in match]}
        os.makedirs(args.traffic_dir, exist_ok=True)
        with open(os.path.join(args.traffic_dir, f"kernels_{args.label}.json"), "w") as f:
            json.dump({"workload": args.label, "source_hash": source_hash(), "calls": kcalls,
                       "command": args.command}, f, indent=1)
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
        present = {call for call, kernels in CALL_KERNELS.items()
                   if any(kernels[0] in kname for kname in per)}
        for kname, ctrs in sorted(per.items()):
            f_k = float(np.median(ctrs["FETCH_SIZE"])) if "FETCH_SIZE" in ctrs else float("nan")
            w_k = float(np.median(ctrs["WRITE_SIZE"])) if "WRITE_SIZE" in ctrs else float("nan")
            n = max(len(ctrs.get("FETCH_SIZE", [])), len(ctrs.get("WRITE_SIZE", [])))
            out.append(f"| {kname[:90]} | {n} | {f_k:.0f} | {w_k:.0f} |")
            for call, kernels in CALL_KERNELS.items():
                if call in present and any(k in kname for k in kernels):
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


class Flush:
    """Evicts L2 and the MALL between timed reps, outside the timed region:
    writes a 1 GiB scratch buffer, then reads another 1 GiB one, so that no
    dirty line of the flush is left for the timed call to write back."""

    def __init__(self, torch, nbytes=1 << 30):
        self.torch = torch
        self.w = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        self.r = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
        self.acc = torch.empty((), dtype=torch.float32, device="cuda")
        self.i = 0

    def __call__(self):
        self.i += 1
        self.w.fill_(self.i & 255)
        self.torch.sum(self.r, dim=0, out=self.acc)


def stats_us(samples):
    a = np.asarray(samples, np.float64)
    return {"median": round(float(np.median(a)), 2), "p10": round(float(np.percentile(a, 10)), 2),
            "p90": round(float(np.percentile(a, 90)), 2), "mean": round(float(a.mean()), 2),
            "n": int(a.size)}


def time_calls(torch, calls, stream, reps, flush=None):
    """Runs the calls in order `reps` times, each call bracketed by HIP events
    on `stream` (the stream every call is enqueued on); with `flush`, the
    caches are flushed before every rep, outside the events.  Returns
    {call: [us, ...]}."""
    pending = []
    for _ in range(reps):
        if flush is not None:
            flush()
        evs = []
        for name, fn in calls:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            evs.append((name, e0, e1))
        pending.append(evs)
    torch.cuda.synchronize()
    out = {name: [] for name, _ in calls}
    for evs in pending:
        for name, e0, e1 in evs:
            out[name].append(e0.elapsed_time(e1) * 1e3)
    return out


def load_kernel_times(label):
    """rocprofv3 average kernel durations (us) per call of a workload from the
    committed summary, if the kernel sources are unchanged since."""
    path = os.path.join(PROFILES, f"kernels_{label}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_hash") != source_hash():
        return None
    return t.get("calls")


class Workload:
    """One benchmark workload: its calls in step order (each enqueues one C-ABI
    call on the stream), their algorithmic work, the dominant call and the
    oracle baseline / parity check."""

    def __init__(self, name, desc, seed, calls, work, dominant, cpu, label=None, extra=None):
        self.name, self.desc, self.seed = name, desc, seed
        self.calls, self.work, self.dominant, self.cpu = calls, work, dominant, cpu
        self.label = label or name
        self.extra = extra or {}


def build_workload(name, args, torch, A, I, sA):
    """Allocates and fills the device inputs of workload `name` (untimed)."""
    desc, inputs = WORKLOADS[name]  # the inputs module's builder of its seeded inputs
    dev = "cuda"
    w = (I.mixed_step(num_layers=args.pack_layers) if inputs == "mixed_step"
         else getattr(I, inputs)())
    shape = A.make_shape(w.hq, w.hkv, w.d, w.dtype, w.scale)
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    os.environ.setdefault("OMP_NUM_THREADS", str(threads))

    def cpu_entry(value, unit, amount, n, dt, sample):
        return {"value": value, "unit": unit, "cores": threads, "kind": "oracle",
                "cpu": cpu_info(), "seconds": round(dt, 2), "passes": n, "sample": sample}

    def widen(t):
        return I.bf16_bits_to_f32(A.to_host(t)).astype(np.float64)

    def err_block(got, ref):
        err = np.abs(got - ref)
        rms = np.sqrt(np.mean(ref ** 2, axis=-1))
        return {"max_abs_err": float(err.max()),
                "max_norm_err": float((err.max(axis=-1) / np.maximum(rms, 1e-30)).max()),
                "rows": int(np.prod(ref.shape[:-1]))}

    if name == "mixed":
        L = args.pack_layers
        kp = torch.empty((L,) + w.k_pool.shape, dtype=torch.bfloat16, device=dev)
        vp = torch.empty((L,) + w.v_pool.shape, dtype=torch.bfloat16, device=dev)
        kp[0].copy_(A.to_device(w.k_pool))
        vp[0].copy_(A.to_device(w.v_pool))
        for layer in range(1, L):  # extra layers only widen the pack
            kp[layer].copy_(kp[0])
            vp[layer].copy_(vp[0])
        pt = A.to_device(w.page_table)
        stride = w.page_table.shape[1]
        pre_pt = pt[w.prefill_rows[0]:]
        q, k, v = A.to_device(w.q), A.to_device(w.k), A.to_device(w.v)
        cu = A.to_device(w.cu_seqlens)
        out_p = torch.empty_like(q)
        n_pre, n_dec = len(w.prefill_lens), len(w.context_lens)
        start = torch.zeros(n_pre, dtype=torch.int32, device=dev)
        q_dec, ctx = A.to_device(w.q_dec), A.to_device(w.context_lens)
        out_d = torch.empty_like(q_dec)
        ws = A.decode_workspace(shape, w.context_lens, n_dec, args.split)
        offs_np = I.handoff_offsets(w.handoff_lens, L, w.hkv, w.d)
        offs = A.to_device(offs_np)
        hreq, hlen = A.to_device(w.handoff_reqs), A.to_device(w.handoff_lens)
        out_h = torch.empty(int(offs_np[-1]), dtype=torch.bfloat16, device=dev)
        T = int(w.cu_seqlens[-1])

        def decode():
            A.dopd_decode_attn(shape, q_dec, kp[0], vp[0], w.num_pages, pt, stride, ctx,
                               w.context_lens, n_dec, args.split, out_d, None, ws, stream=sA)

        def prefill():
            A.dopd_prefill_attn(shape, q, k, v, out_p, None, cu, w.cu_seqlens, n_pre, stream=sA)

        def write():
            A.dopd_kv_write(shape, k, v, kp[0], vp[0], w.num_pages, pre_pt, stride, cu, start,
                            n_pre, T, sA)

        def pack():
            A.dopd_kv_pack_for_handoff(shape, L, kp, vp, w.num_pages, pt, stride, hreq, hlen,
                                       w.handoff_lens, offs, n_pre, out_h, sA)

        order = [("prefill", prefill), ("kv_write", write)]
        order = ([("decode", decode)] + order if args.order == "decode-first"
                 else order + [("decode", decode)])
        calls = order + [("pack", pack)]
        work = {"decode": ("GB/s", decode_bytes(w.context_lens, w.hq, w.hkv, w.d)),
                "prefill": ("TFLOP/s", prefill_flops(w.prefill_lens, w.hq, w.d)),
                "kv_write": ("GB/s", write_bytes(w.prefill_lens, w.hkv, w.d)),
                "pack": ("GB/s", pack_bytes(w.handoff_lens, L, w.hkv, w.d))}

        def cpu():
            import oracle
            (ref, _), n, dt = repeat_timed(
                lambda: oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table,
                                      w.context_lens, w.scale), args.cpu_seconds)
            amount = work["decode"][1]
            base = cpu_entry(round(n * amount / dt / 1e9, 4), "GB/s", amount, n, dt,
                             f"fp64 oracle decode of the whole batch ({n_dec} requests, "
                             f"{amount / 1e9:.3f} GB algorithmic), {n} passes")
            (ref_p, _), n_p, dtp = repeat_timed(
                lambda: oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale), args.cpu_seconds)
            base["prefill_tflops"] = round(n_p * work["prefill"][1] / dtp / 1e12, 6)
            base["prefill_seconds"] = round(dtp, 2)
            base["sample"] += f"; fp64 oracle prefill of the whole prefill batch, {n_p} passes"
            parity = {"decode": err_block(widen(out_d), ref),
                      "prefill": err_block(widen(out_p), ref_p)}
            if L == 1:
                rk, rv = oracle.kv_write(w.k, w.v, w.k_pool, w.v_pool,
                                         w.page_table[w.prefill_rows[0]:], w.cu_seqlens,
                                         np.zeros(n_pre, np.int32))
                ref_h = oracle.pack(rk, rv, 1, w.page_table, w.handoff_reqs, w.handoff_lens,
                                    offs_np)
                parity["kv_write_bit_exact"] = bool(
                    np.array_equal(A.to_host(kp[0]), rk) and np.array_equal(A.to_host(vp[0]), rv))
                parity["pack_bit_exact"] = bool(np.array_equal(A.to_host(out_h), ref_h))
            return base, parity

        return Workload(name, desc, w.seed, calls, work, "decode", cpu,
                        extra={"order": args.order, "pack_layers": L})

    if name == "pd_step":
        n_pre, n_dec = len(w.prefill_lens), len(w.context_lens)
        kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
        pt = A.to_device(w.page_table)
        stride = w.page_table.shape[1]
        q, k, v = A.to_device(w.q), A.to_device(w.k), A.to_device(w.v)
        cu, ctx = A.to_device(w.cu_seqlens), A.to_device(w.context_lens)
        out_p = torch.empty_like(q)
        q_dec = A.to_device(w.q_dec)
        out_d = torch.empty_like(q_dec)
        offs_np = I.handoff_offsets(w.prefill_lens, 1, w.hkv, w.d)
        offs = A.to_device(offs_np)
        out_h = torch.empty(int(offs_np[-1]), dtype=torch.bfloat16, device=dev)
        ws = A.pd_step_workspace(shape, w.context_lens, n_dec, args.schedule)
        fp8 = args.kv == "fp8"
        if fp8:
            # The decode requests' cache as E4M3 pages, written by the fp8 writer
            # from their bf16 tokens (untimed); one scale per KV head from the
            # absolute maximum of those tokens.
            shape8 = A.make_shape(w.hq, w.hkv, w.d, "fp8", w.scale)
            cl = w.context_lens.astype(np.int64)
            r_idx = np.repeat(np.arange(n_dec), cl)
            j = np.arange(int(cl.sum())) - np.repeat(np.cumsum(cl) - cl, cl)
            pg = torch.from_numpy(w.page_table[r_idx, j // 16].astype(np.int64)).to(dev)
            sl = torch.from_numpy((j % 16).astype(np.int64)).to(dev)
            ktok = kp[pg, :, sl, :].contiguous()
            vtok = vp[pg, :, :, sl].contiguous()
            ks_h, vs_h = e4m3_head_scales(A.to_host(ktok)), e4m3_head_scales(A.to_host(vtok))
            ks, vs = A.to_device(ks_h), A.to_device(vs_h)
            kp = torch.full((w.num_pages, w.hkv, 16, w.d), 0x7F, dtype=torch.uint8, device=dev)
            vp = torch.full((w.num_pages, w.hkv, w.d, 16), 0x7F, dtype=torch.uint8, device=dev)
            A.dopd_kv_write_fp8(shape8, ktok, vtok, ks, vs, kp, vp, w.num_pages, pt[:n_dec],
                                stride, A.to_device(I.cu_from_lens(w.context_lens)),
                                torch.zeros(n_dec, dtype=torch.int32, device=dev), n_dec,
                                int(cl.sum()), sA)
            torch.cuda.synchronize()
            del ktok, vtok
            out_h = torch.empty(int(offs_np[-1]), dtype=torch.uint8, device=dev)

            def step():
                A.dopd_pd_step_fp8(shape8, q_dec, pt[:n_dec], ctx, w.context_lens, n_dec, out_d,
                                   None, q, k, v, cu, w.cu_seqlens, n_pre, pt[n_dec:], out_p,
                                   None, kp, vp, ks, vs, w.num_pages, stride, offs, out_h,
                                   args.schedule, ws, stream=sA)
        else:
            def step():
                A.dopd_pd_step(shape, q_dec, pt[:n_dec], ctx, w.context_lens, n_dec, out_d,
                               None, q, k, v, cu, w.cu_seqlens, n_pre, pt[n_dec:], out_p, None,
                               kp, vp, w.num_pages, stride, offs, out_h, args.schedule, ws,
                               stream=sA)

        work = {"pd_step": ("step", None)}

        def cpu():
            import oracle
            if fp8:
                # the oracle quantises the same bf16 cache and prompts with the
                # same scales, and decodes / writes / packs the codes
                P, hkv, d = w.num_pages, w.hkv, w.d
                kq = oracle.e4m3_quantize(w.k_pool.transpose(0, 2, 1, 3).reshape(-1, hkv, d), ks_h)
                vq = oracle.e4m3_quantize(w.v_pool.transpose(0, 3, 1, 2).reshape(-1, hkv, d), vs_h)
                k0 = kq.reshape(P, 16, hkv, d).transpose(0, 2, 1, 3).copy()
                v0 = vq.reshape(P, 16, hkv, d).transpose(0, 2, 3, 1).copy()
                ref, _ = oracle.decode_e4m3(w.q_dec, k0, v0, ks_h, vs_h, w.page_table[:n_dec],
                                            w.context_lens, w.scale)
                knew, vnew = oracle.e4m3_quantize(w.k, ks_h), oracle.e4m3_quantize(w.v, vs_h)
            else:
                k0, v0, knew, vnew = w.k_pool, w.v_pool, w.k, w.v
                ref, _ = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table[:n_dec],
                                       w.context_lens, w.scale)
            ref_p, _ = oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale)
            rk, rv = oracle.kv_write(knew, vnew, k0, v0, w.page_table[n_dec:], w.cu_seqlens,
                                     np.zeros(n_pre, np.int32))
            ref_h = oracle.pack(rk, rv, 1, w.page_table[n_dec:],
                                np.arange(n_pre, dtype=np.int32), w.prefill_lens, offs_np)
            return None, {"decode": err_block(widen(out_d), ref),
                          "prefill": err_block(widen(out_p), ref_p),
                          "kv_write_bit_exact": bool(np.array_equal(A.to_host(kp), rk) and
                                                     np.array_equal(A.to_host(vp), rv)),
                          "pack_bit_exact": bool(np.array_equal(A.to_host(out_h), ref_h))}

        return Workload(name, desc, w.seed, [("pd_step", step)], work, "pd_step", cpu,
                        label=name + ("_fp8" if fp8 else ""),
                        extra={"schedule": args.schedule, "kv": args.kv})

    if name == "write_pack":
        n_pre, n_dec = len(w.prefill_lens), len(w.context_lens)
        kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
        pt = A.to_device(w.page_table)
        stride = w.page_table.shape[1]
        k, v = A.to_device(w.k), A.to_device(w.v)
        cu = A.to_device(w.cu_seqlens)
        start = torch.zeros(n_pre, dtype=torch.int32, device=dev)
        offs_np = I.handoff_offsets(w.prefill_lens, 1, w.hkv, w.d)
        offs = A.to_device(offs_np)
        hreq, hlen = A.to_device(w.handoff_reqs), A.to_device(w.handoff_lens)
        out_h = torch.empty(int(offs_np[-1]), dtype=torch.bfloat16, device=dev)
        out_h2 = torch.empty_like(out_h)
        T = int(w.cu_seqlens[-1])

        def write():
            A.dopd_kv_write(shape, k, v, kp, vp, w.num_pages, pt[n_dec:], stride, cu, start,
                            n_pre, T, sA)

        def pack():
            A.dopd_kv_pack_for_handoff(shape, 1, kp, vp, w.num_pages, pt, stride, hreq, hlen,
                                       w.handoff_lens, offs, n_pre, out_h, sA)

        def write_pack():
            A.dopd_kv_write_pack_for_handoff(shape, k, v, kp, vp, w.num_pages, pt[n_dec:],
                                             stride, cu, w.cu_seqlens, n_pre, offs, out_h2, sA)

        # The floor at this size: a plain elementwise kernel that reads and
        # writes as many bytes as the pack does.
        nb = pack_bytes(w.handoff_lens, 1, w.hkv, w.d) // 2
        src16 = torch.zeros(nb // 2, dtype=torch.int16, device=dev)
        dst16 = torch.empty_like(src16)

        def plain_copy():
            torch.bitwise_not(src16, out=dst16)

        work = {"kv_write": ("GB/s", write_bytes(w.prefill_lens, w.hkv, w.d)),
                "pack": ("GB/s", pack_bytes(w.handoff_lens, 1, w.hkv, w.d)),
                "kv_write_pack": ("GB/s", write_pack_bytes(w.prefill_lens, w.hkv, w.d)),
                "plain_copy": ("GB/s", 2 * nb)}

        def cpu():
            import oracle
            rk, rv = oracle.kv_write(w.k, w.v, w.k_pool, w.v_pool, w.page_table[n_dec:],
                                     w.cu_seqlens, np.zeros(n_pre, np.int32))
            ref_h = oracle.pack(rk, rv, 1, w.page_table, w.handoff_reqs, w.handoff_lens, offs_np)
            return None, {"kv_write_bit_exact": bool(np.array_equal(A.to_host(kp), rk) and
                                                     np.array_equal(A.to_host(vp), rv)),
                          "pack_bit_exact": bool(np.array_equal(A.to_host(out_h), ref_h)),
                          "write_pack_bit_exact": bool(np.array_equal(A.to_host(out_h2), ref_h))}

        return Workload(name, desc, w.seed, [("kv_write", write), ("pack", pack),
                                             ("kv_write_pack", write_pack),
                                             ("plain_copy", plain_copy)], work,
                        "kv_write_pack", cpu)

    if name in ("decode_mha", "decode_gqa"):
        kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
        pt = A.to_device(w.page_table)
        q_dec, ctx = A.to_device(w.q_dec), A.to_device(w.context_lens)
        out_d = torch.empty_like(q_dec)
        n_dec = len(w.context_lens)
        stride = w.page_table.shape[1]
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
            ktok = kp[pg, :, sl, :].contiguous()
            vtok = vp[pg, :, :, sl].contiguous()
            ks = (ktok.abs().amax(dim=(0, 2)).float() / 448.0).contiguous()
            vs = (vtok.abs().amax(dim=(0, 2)).float() / 448.0).contiguous()
            kp8 = torch.full((w.num_pages, w.hkv, 16, w.d), 0x7F, dtype=torch.uint8, device=dev)
            vp8 = torch.full((w.num_pages, w.hkv, w.d, 16), 0x7F, dtype=torch.uint8, device=dev)
            ws = A.decode_workspace(shape8, w.context_lens, n_dec, args.split)
            cu_t = A.to_device(I.cu_from_lens(w.context_lens))
            A.dopd_kv_write_fp8(shape8, ktok, vtok, ks, vs, kp8, vp8, w.num_pages, pt, stride,
                                cu_t, torch.zeros(n_dec, dtype=torch.int32, device=dev), n_dec,
                                int(cl.sum()), sA)
            torch.cuda.synchronize()
            del ktok, vtok, kp, vp

            def decode():
                A.dopd_decode_attn_fp8(shape8, q_dec, kp8, vp8, ks, vs, w.num_pages, pt, stride,
                                       ctx, w.context_lens, n_dec, args.split, out_d, None, ws,
                                       stream=sA)

            work = {"decode": ("GB/s", decode_bytes(w.context_lens, w.hq, w.hkv, w.d, kv_s=1))}
        else:
            ws = A.decode_workspace(shape, w.context_lens, n_dec, args.split)

            def decode():
                A.dopd_decode_attn(shape, q_dec, kp, vp, w.num_pages, pt, stride, ctx,
                                   w.context_lens, n_dec, args.split, out_d, None, ws, stream=sA)

            work = {"decode": ("GB/s", decode_bytes(w.context_lens, w.hq, w.hkv, w.d))}

        def cpu():
            import oracle
            amount = work["decode"][1]
            if args.kv == "fp8":
                # the oracle quantises the same bf16 cache with the same scales
                ks_h, vs_h = ks.cpu().numpy(), vs.cpu().numpy()
                P, hkv, d = w.num_pages, w.hkv, w.d
                kq = oracle.e4m3_quantize(w.k_pool.transpose(0, 2, 1, 3).reshape(-1, hkv, d), ks_h)
                vq = oracle.e4m3_quantize(w.v_pool.transpose(0, 3, 1, 2).reshape(-1, hkv, d), vs_h)
                kq = kq.reshape(P, 16, hkv, d).transpose(0, 2, 1, 3).copy()
                vq = vq.reshape(P, 16, hkv, d).transpose(0, 2, 3, 1).copy()
                (ref, _), n, dt = repeat_timed(
                    lambda: oracle.decode_e4m3(w.q_dec, kq, vq, ks_h, vs_h, w.page_table,
                                               w.context_lens, w.scale), args.cpu_seconds)
                what = "fp64 oracle decode over E4M3 pages"
                # the format's own error: the GPU's E4M3 decode against the exact
                # decode over the bf16 cache it was quantised from (reported, not a gate)
                ref_bf16, _ = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table,
                                            w.context_lens, w.scale)
            else:
                (ref, _), n, dt = repeat_timed(
                    lambda: oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table,
                                          w.context_lens, w.scale), args.cpu_seconds)
                what = "fp64 oracle decode"
            base = cpu_entry(round(n * amount / dt / 1e9, 4), "GB/s", amount, n, dt,
                             f"{what} of the whole batch ({n_dec} requests, "
                             f"{amount / 1e9:.3f} GB algorithmic), {n} passes")
            got = widen(out_d)
            par = {"decode": err_block(got, ref)}
            if args.kv == "fp8":
                par["e4m3_quantisation_error_vs_bf16_cache"] = err_block(got, ref_bf16)
            return base, par

        return Workload(name, desc, w.seed, [("decode", decode)], work, "decode", cpu,
                        label=name + ("_fp8" if args.kv == "fp8" else ""),
                        extra={"kv": args.kv})

    if name == "handoff":
        L = args.pack_layers
        n_dec, n_pre = len(w.context_lens), len(w.prefill_lens)
        kp = torch.empty((L,) + w.k_pool.shape, dtype=torch.bfloat16, device=dev)
        vp = torch.empty((L,) + w.v_pool.shape, dtype=torch.bfloat16, device=dev)
        kp[0].copy_(A.to_device(w.k_pool))
        vp[0].copy_(A.to_device(w.v_pool))
        pt = A.to_device(w.page_table)
        stride = w.page_table.shape[1]
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

        def pack():
            A.dopd_kv_pack_for_handoff(shape, L, kp, vp, w.num_pages, pt, stride, hreq, hlen,
                                       w.handoff_lens, offs, n_pre, buf, sA)

        def unpack():
            A.dopd_kv_unpack_from_handoff(shape, L, buf, offs, dreq, hlen, w.handoff_lens, n_pre,
                                          kd, vd, pages_d, pt_d, pt_d_np.shape[1], sA)

        work = {"pack": ("GB/s", pack_bytes(w.handoff_lens, L, w.hkv, w.d)),
                "unpack": ("GB/s", pack_bytes(w.handoff_lens, L, w.hkv, w.d))}
        return Workload(name, desc, w.seed, [("pack", pack), ("unpack", unpack)], work, "unpack",
                        None, extra={"pack_layers": L})

    # varlen prefill (+ paged write), one-shot or chunked over the paged cache
    q, k, v = A.to_device(w.q), A.to_device(w.k), A.to_device(w.v)
    cu = A.to_device(w.cu_seqlens)
    kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
    pt = A.to_device(w.page_table)
    stride = w.page_table.shape[1]
    n_pre = len(w.prefill_lens)
    start = torch.zeros(n_pre, dtype=torch.int32, device=dev)
    T = int(w.cu_seqlens[-1])
    out_p = torch.empty_like(q)
    if name == "chunked":
        # The prompts are prefilled in chunks of C tokens, each attending to its
        # cached prefix: a call takes the next chunk of the prompts in turn until
        # it holds `budget` tokens (a chunked-prefill batch), calls back to back.
        C, B = args.chunk, args.budget
        lens = w.prefill_lens.astype(np.int64)
        pos = np.zeros(n_pre, np.int64)
        chunks = []
        while (pos < lens).any():
            sel, budget = [], B
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
            pt_c = np.ascontiguousarray(w.page_table[[x[0] for x in sel]])
            chunks.append(dict(q=q.index_select(0, rows_d).contiguous(), rows=rows_d,
                               out=torch.empty((len(rows), w.hq, w.d), dtype=torch.bfloat16,
                                               device=dev),
                               cu=A.to_device(cu_c), cu_h=cu_c, pre=A.to_device(pre), pre_h=pre,
                               pt=A.to_device(pt_c), n=len(sel)))
        fp8 = args.kv == "fp8"
        wsize = (A.dopd_prefill_paged_fp8_workspace_size if fp8 else
                 A.dopd_prefill_paged_workspace_size)
        shape_c = A.make_shape(w.hq, w.hkv, w.d, "fp8", w.scale) if fp8 else shape
        ws_bytes = max(wsize(shape_c, ch["cu_h"], ch["pre_h"], ch["n"], args.splits)
                       for ch in chunks)
        ws_buf = torch.empty(ws_bytes + 256, dtype=torch.uint8, device=dev)
        ws = ws_buf[(-ws_buf.data_ptr()) % 256:][:ws_bytes]

        def result():
            for ch in chunks:
                out_p.index_copy_(0, ch["rows"], ch["out"])
            return out_p

        if fp8:
            ks_h, vs_h = e4m3_head_scales(w.k), e4m3_head_scales(w.v)
            ks, vs = A.to_device(ks_h), A.to_device(vs_h)
            kp = torch.full((w.num_pages, w.hkv, 16, w.d), 0x7F, dtype=torch.uint8, device=dev)
            vp = torch.full((w.num_pages, w.hkv, w.d, 16), 0x7F, dtype=torch.uint8, device=dev)

            def write():
                A.dopd_kv_write_fp8(shape_c, k, v, ks, vs, kp, vp, w.num_pages, pt, stride, cu,
                                    start, n_pre, T, sA)

            def chunked():
                for ch in chunks:
                    A.dopd_prefill_paged_attn_fp8(shape_c, ch["q"], kp, vp, ks, vs, w.num_pages,
                                                  ch["pt"], stride, ch["cu"], ch["cu_h"],
                                                  ch["pre"], ch["pre_h"], ch["n"], args.splits,
                                                  ch["out"], None, ws, ws_bytes, sA)

            calls = [("kv_write_fp8", write), ("prefill_chunked_fp8", chunked)]
            work = {"prefill_chunked_fp8": ("TFLOP/s",
                                            prefill_flops(w.prefill_lens, w.hq, w.d)),
                    "kv_write_fp8": ("GB/s", write_bytes(w.prefill_lens, w.hkv, w.d, out_s=1))}
            dominant = "prefill_chunked_fp8"
        else:
            def write():
                A.dopd_kv_write(shape, k, v, kp, vp, w.num_pages, pt, stride, cu, start, n_pre, T,
                                sA)

            def chunked():
                for ch in chunks:
                    A.dopd_prefill_paged_attn_split(shape, ch["q"], kp, vp, w.num_pages,
                                                    ch["pt"], stride, ch["cu"], ch["cu_h"],
                                                    ch["pre"], ch["pre_h"], ch["n"], args.splits,
                                                    ch["out"], None, ws, ws_bytes, sA)

            calls = [("kv_write", write), ("prefill_chunked", chunked)]
            work = {"prefill_chunked": ("TFLOP/s", prefill_flops(w.prefill_lens, w.hq, w.d)),
                    "kv_write": ("GB/s", write_bytes(w.prefill_lens, w.hkv, w.d))}
            dominant = "prefill_chunked"
        extra = {"chunk": C, "budget": B, "calls_per_pass": len(chunks), "kv": args.kv}
    else:
        if args.kv == "fp8":
            # the prompts' K/V go to an E4M3 cache (scales from each head's
            # absolute maximum over the batch)
            shape8 = A.make_shape(w.hq, w.hkv, w.d, "fp8", w.scale)
            ks = (k.abs().amax(dim=(0, 2)).float() / 448.0).contiguous()
            vs = (v.abs().amax(dim=(0, 2)).float() / 448.0).contiguous()
            kp = torch.full((w.num_pages, w.hkv, 16, w.d), 0x7F, dtype=torch.uint8, device=dev)
            vp = torch.full((w.num_pages, w.hkv, w.d, 16), 0x7F, dtype=torch.uint8, device=dev)

            def write():
                A.dopd_kv_write_fp8(shape8, k, v, ks, vs, kp, vp, w.num_pages, pt, stride, cu,
                                    start, n_pre, T, sA)
            wbytes = write_bytes(w.prefill_lens, w.hkv, w.d, out_s=1)
        else:
            def write():
                A.dopd_kv_write(shape, k, v, kp, vp, w.num_pages, pt, stride, cu, start, n_pre,
                                T, sA)
            wbytes = write_bytes(w.prefill_lens, w.hkv, w.d)

        def prefill():
            A.dopd_prefill_attn(shape, q, k, v, out_p, None, cu, w.cu_seqlens, n_pre, stream=sA)

        def result():
            return out_p

        calls = [("prefill", prefill), ("kv_write", write)]
        work = {"prefill": ("TFLOP/s", prefill_flops(w.prefill_lens, w.hq, w.d)),
                "kv_write": ("GB/s", wbytes)}
        dominant = "prefill"
        extra = {"kv": args.kv}

    def cpu():
        # Bounded sample: the last 4 rows of every prompt (the longest rows),
        # 4 heads each; the GPU tests compare every row.
        import oracle
        rows_tok = np.repeat(np.concatenate([w.cu_seqlens[1:] - 1 - i for i in range(4)]), 4)
        heads = (np.arange(len(rows_tok)) * 7) % w.hq
        if name == "chunked" and args.kv == "fp8":
            # the oracle quantises the prompts with the same scales into pools
            # of its own and reads them as one chunk per prompt
            ks_h, vs_h = e4m3_head_scales(w.k), e4m3_head_scales(w.v)
            k8 = np.full((w.num_pages, w.hkv, 16, w.d), 0x7F, np.uint8)
            v8 = np.full((w.num_pages, w.hkv, w.d, 16), 0x7F, np.uint8)
            zeros = np.zeros(n_pre, np.int32)
            k8, v8 = oracle.kv_write(oracle.e4m3_quantize(w.k, ks_h),
                                     oracle.e4m3_quantize(w.v, vs_h), k8, v8,
                                     w.page_table[w.prefill_rows], w.cu_seqlens, zeros)

            def run():
                return oracle.prefill_paged_e4m3(w.q, k8, v8, ks_h, vs_h,
                                                 w.page_table[w.prefill_rows], w.cu_seqlens,
                                                 zeros, w.scale, rows_tok, heads)
            what = "fp64 oracle chunk prefill over E4M3 pages"
        else:
            def run():
                return oracle.prefill_rows(w.q, w.k, w.v, w.cu_seqlens, w.scale, rows_tok, heads)
            what = "fp64 oracle prefill"
        (ref, _), n, dt = repeat_timed(run, args.cpu_seconds)
        req_of = np.searchsorted(w.cu_seqlens, rows_tok, side="right") - 1
        flops = int((4 * w.d * (rows_tok - w.cu_seqlens[req_of] + 1)).sum())
        base = cpu_entry(round(n * flops / dt / 1e12, 6), "TFLOP/s", flops, n, dt,
                         f"{what} of {len(rows_tok)} sampled rows (the last 4 rows "
                         f"of every prompt, 4 heads each; {flops / 1e9:.2f} GFLOP), {n} passes")
        got = widen(result())[rows_tok, heads]
        return base, {dominant: err_block(got, ref)}

    return Workload(name, desc, w.seed, calls, work, dominant, cpu,
                    label=name + ("_fp8" if args.kv == "fp8" else ""), extra=extra)


def run_workload(wl, args, torch, sA, flush, steps, warmup, reps):
    """Warm-up, the K back-to-back timed steps (ms per step), then `reps`
    cold reps (caches flushed before each) and `reps` warm reps, every call
    bracketed by HIP events.  Returns the workload's record."""
    for _ in range(warmup):
        for _, fn in wl.calls:
            fn()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(sA)
    step_us = time_calls(torch, wl.calls, sA, steps)
    ev1.record(sA)
    torch.cuda.synchronize()
    ms_step = ev0.elapsed_time(ev1) / max(1, steps)
    cold = time_calls(torch, wl.calls, sA, reps, flush)
    warm = time_calls(torch, wl.calls, sA, reps)
    ktimes = load_kernel_times(wl.label) or {}
    calls = {}
    for name, _ in wl.calls:
        unit, amount = wl.work[name]
        if amount is None:  # a whole step: times only
            calls[name] = {"unit": unit, "cold_us": stats_us(cold[name]),
                           "warm_us": stats_us(warm[name]),
                           "step_mean_us": mean_or_none(step_us[name])}
            continue
        scale = 1e12 if unit == "TFLOP/s" else 1e9
        peak = BF16_PEAK_TFLOPS if unit == "TFLOP/s" else HBM_PEAK_GBS
        c, wm = stats_us(cold[name]), stats_us(warm[name])
        rec = {"unit": unit, ("flops" if unit == "TFLOP/s" else "bytes"): amount,
               "cold_us": c, "warm_us": wm,
               "rate": round(amount / (c["median"] * 1e-6) / scale, 2),
               "frac": round(amount / (c["median"] * 1e-6) / scale / peak, 4),
               "warm_rate": round(amount / (wm["median"] * 1e-6) / scale, 2),
               "warm_frac": round(amount / (wm["median"] * 1e-6) / scale / peak, 4),
               "step_mean_us": mean_or_none(step_us[name])}
        kt = ktimes.get(name)
        if kt:  # rocprofv3 kernel time (no event or launch overhead)
            rec["kernel_us_rocprof"] = kt["avg_us"]
            rec["kernel_frac_rocprof"] = round(amount / (kt["avg_us"] * 1e-6) / scale / peak, 4)
        calls[name] = rec
    rec = {"workload": wl.desc, "seed": int(wl.seed), "ms_per_step": round(ms_step, 4),
           "calls": calls, "dominant": wl.dominant, **wl.extra}
    if wl.cpu is not None and not args.no_cpu_baseline:
        base, rec["parity"] = wl.cpu()
        if base is not None:
            rec["cpu_baseline"] = base
    return rec


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--reps", type=int, default=50,
                    help="timed reps per call with the caches flushed before each (and as many "
                         "warm reps)")
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="mixed")
    ap.add_argument("--no-configs", action="store_true",
                    help="with the mixed workload: skip the pd_step, write_pack, decode_mha, "
                         "prefill and decode_gqa workloads measured after it")
    ap.add_argument("--pack-layers", type=int, default=1,
                    help="layers packed per handoff in the mixed step (1 = the configured step)")
    ap.add_argument("--split", type=int, default=0, help="decode split tokens (0 = automatic)")
    ap.add_argument("--chunk", type=int, default=512, help="chunked workload: tokens per chunk")
    ap.add_argument("--budget", type=int, default=8192,
                    help="chunked workload: tokens per call (chunks of several prompts)")
    ap.add_argument("--splits", type=int, default=0,
                    help="chunked workload: key splits per call (0 = automatic, 1 = none)")
    ap.add_argument("--order", choices=("decode-first", "prefill-first"), default="decode-first",
                    help="mixed step: the decode batch before the prefill, write and pack (its "
                         "tokens are the TPOT-bound ones), or after the write")
    ap.add_argument("--schedule", type=int, default=0, choices=(0, 1, 2, 3),
                    help="pd_step workload: block order of the single launch (0 = automatic, "
                         "1 = prefill first, 2 = decode first with one decode slice per CU, "
                         "3 = decode first with three slices per two CUs)")
    ap.add_argument("--kv", choices=("bf16", "fp8"), default="bf16",
                    help="KV cache element type (fp8 = E4M3 pages with per-KV-head scales): "
                         "decode workloads read it (written by the fp8 writer before timing), "
                         "the prefill workload writes it, the chunked workload writes it "
                         "and its chunk calls read it, the fused step reads and writes it")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="after timing, run one elementwise kernel over this many MiB "
                         "(counter calibration)")
    ap.add_argument("--summarize", default=None,
                    help="summarise a rocprofv3 output directory instead of benchmarking")
    ap.add_argument("--label", default="mixed")
    ap.add_argument("--command", default="")
    ap.add_argument("--summary-out", default=None)
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="host time the oracle baseline of the headline workload is timed over "
                         "(passes repeat); the other workloads take half")
    ap.add_argument("--traffic-dir", default=PROFILES,
                    help="where --summarize writes traffic_<label>.json and kernels_<label>.json")
    args = ap.parse_args()
    if args.summarize:
        summarize(args)
        return

    if args.kv == "fp8" and args.workload not in ("decode_mha", "decode_gqa", "prefill",
                                                  "chunked", "pd_step"):
        print("--kv fp8 applies to the decode_mha, decode_gqa, prefill, chunked and pd_step "
              "workloads",
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
    sA = torch.cuda.current_stream()
    flush = Flush(torch)
    props = torch.cuda.get_device_properties(0)

    t0 = time.time()
    wl = build_workload(args.workload, args, torch, A, I, sA)
    gen_s = time.time() - t0
    head = run_workload(wl, args, torch, sA, flush, args.steps, args.warmup, args.reps)
    print(f"[bench] {args.workload}: {head['ms_per_step']} ms/step", file=sys.stderr, flush=True)
    del wl
    torch.cuda.empty_cache()

    if args.copy_calib_mib:
        # A shader kernel of known traffic (reads and writes N MiB once), used to
        # scale the HBM counters; a plain device copy would go to a DMA engine.
        src = torch.ones(args.copy_calib_mib << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    configs = {}
    if args.workload == "mixed" and not args.no_configs:
        sub = argparse.Namespace(**vars(args))
        sub.cpu_seconds = args.cpu_seconds / 2
        for name in ("pd_step", "write_pack", "decode_mha", "prefill", "decode_gqa"):
            wl2 = build_workload(name, sub, torch, A, I, sA)
            configs[name] = run_workload(wl2, sub, torch, sA, flush, 0, args.warmup, args.reps)
            configs[name].pop("ms_per_step")
            print(f"[bench] {name} done", file=sys.stderr, flush=True)
            del wl2
            torch.cuda.empty_cache()

    dom = head["calls"][head["dominant"]]
    unit = dom["unit"]
    if "rate" not in dom:  # a whole-step workload (pd_step): its time is the figure
        line = {"metric": "mixed P/D step time (single PD-aggregated launch)",
                "value": dom["cold_us"]["median"], "unit": "us", "n_gpus": 1,
                "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
                "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
                "dtype": "bf16", "data": "synthetic",
                "config": {"workload": wl_desc(args), "seed": head["seed"],
                           "schedule": head.get("schedule")},
                "calls": head["calls"], "parity": head.get("parity"),
                "device": {"name": props.name, "cus": props.multi_processor_count}}
        print(json.dumps(json_safe(line), allow_nan=False), flush=True)
        return
    roofline = {"kernel": head["dominant"], "kernels": list(CALL_KERNELS[head["dominant"]]),
                "bound": "mfma" if unit == "TFLOP/s" else "hbm",
                "achieved": round((dom.get("flops") or dom.get("bytes")) /
                                  (dom["cold_us"]["mean"] * 1e-6) /
                                  (1e12 if unit == "TFLOP/s" else 1e9), 2),
                "peak": BF16_PEAK_TFLOPS if unit == "TFLOP/s" else HBM_PEAK_GBS,
                "unit": unit,
                "traffic": load_traffic(args.workload + ("_fp8" if args.kv == "fp8" else ""),
                                        head["dominant"]),
                "timing": "mean of the cold reps (caches flushed before each), HIP events on "
                          "the call's stream"}
    roofline["frac"] = round(roofline["achieved"] / roofline["peak"], 4)
    line = {
        "metric": "decode attn HBM GB/s (% peak) + prefill attn TFLOP/s (% MFMA peak)",
        "value": dom["rate"],
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl_desc(args), "seed": head["seed"], "split_tokens": args.split,
                   "kv": args.kv, "order": head.get("order"),
                   "pack_layers": head.get("pack_layers"), "chunk": head.get("chunk"),
                   "budget": head.get("budget")},
        "value_timing": "median of the cold reps of the dominant call",
        "roofline": roofline,
        "calls": head["calls"],
        "cpu_baseline": head.get("cpu_baseline"),
        "parity": head.get("parity"),
        "configs": configs,
        "device": {"name": props.name, "cus": props.multi_processor_count},
        "flush": "write 1 GiB, then read another 1 GiB, before every cold rep",
        "input_gen_s": round(gen_s, 1),
    }
    print(json.dumps(json_safe(line), allow_nan=False), flush=True)


def wl_desc(args):
    desc = WORKLOADS[args.workload][0]
    return desc + (", KV cache E4M3 with per-KV-head scales" if args.kv == "fp8" else "")


if __name__ == "__main__":
    main()
