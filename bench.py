#!/usr/bin/env python3
"""Benchmark of MARche's cache-aware decode step on one MI355X.

A bench step is one MAR decoding step of the whole batch (all layers: decoder
input, full-attention layers up to the selection layer with the score pass,
refresh top-k, cache-aware layers).  Steps cycle through the 64-step schedule;
the default --warmup 64 --steps 64 times exactly one complete generation.

Printed (one JSON line on stdout):
  value         images/s of the timed steps = batch * steps / 64 / wall seconds
                (inputs, weights and every step's index lists already resident
                in HBM; the timed region is bracketed by device syncs);
  step_us       median step latency by step type;
  full_recompute  the same kernels with every token active in every step;
  roofline      the kernel with the most time in the timed steps, timed live
                with HIP events on the launch stream, against MI355X peak;
  kernels       every kernel class with its achieved rate;
  cpu_baseline  the fp64 oracle on a bounded sample (one image, the first
                steps of its schedule) on this host's cores, extrapolated.

Workload: seeded synthetic MAR-shaped tensors (no dataset or trained weights).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MAR-L-shape step latency (µs), images/s, MFMA/HBM % of peak vs full recompute"
PEAK_BF16_TFLOPS = 2500.0
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
HBM_BOUND = {"gather_ln", "attention_q32", "attention_q64", "attn_scores", "select_topk",
             "decoder_input", "row_map", "fill_zero"}
KERNEL_SOURCES = {
    "gemm": "paper_2506_12035_amd/csrc/k_gemm.hip",
    "attention": "paper_2506_12035_amd/csrc/k_attn.hip",
    "select": "paper_2506_12035_amd/csrc/k_select.hip",
    "elementwise": "paper_2506_12035_amd/csrc/k_elementwise.hip",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_hash(kernel: str) -> str:
    if kernel.startswith("attention") or kernel == "attn_scores":
        fam = "attention"
    elif kernel.startswith("gemm"):
        fam = "gemm"
    elif kernel == "select_topk":
        fam = "select"
    else:
        fam = "elementwise"
    with open(os.path.join(ROOT, KERNEL_SOURCES[fam])) as f:
        return hashlib.sha256(code_only(f.read()).encode()).hexdigest()[:16]


def code_only(src: str) -> str:
    """A source file's code with its comments and blank space removed, so
    that a change to the comments leaves the hash of the kernels unchanged."""
    out, i, n = [], 0, len(src)
    while i < n:
        if src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
        elif src[i] == '"':  # string literal: copied whole
            j = i + 1
            while j < n and src[j] != '"':
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        else:
            out.append(src[i])
            i += 1
    return " ".join("".join(out).split())


def traffic_for(kernel: str, workload: str):
    """HBM bytes per launch of a timing class from committed rocprofv3 counter
    runs, if they were taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    e = rec.get(workload, {}).get("classes", {}).get(kernel)
    if not e or e.get("source_sha") != source_hash(kernel):
        return None
    return e.get("bytes_per_launch")


def counter_class(name: str):
    """Timing class of a kernel symbol as rocprofv3 prints it (mangled or not),
    before the split into full and cache-aware layers."""
    tile = ("t256" if ("gemm_bf16_big_kernel" in name or "gemm_bf16_big8_kernel" in name) else
            "t320" if "gemm_bf16_t320_kernel" in name else
            "t64x128" if "gemm_bf16_small_kernel" in name else
            "t128" if "gemm_bf16_mid_kernel" in name else "t128x256")
    if "gemm_bf16" in name:
        for key, cls in (("EpiResidILi1E", "fc2"), ("EpiResid<1>", "fc2"), ("EpiResidILi0E", "o"),
                         ("EpiResid<0>", "o"), ("EpiGelu", "fc1"), ("EpiQkv", "qkv")):
            if key in name:
                return f"gemm_{cls}_{tile}"
    if "attn_resident_kernel" in name:
        # the last template argument: the score pass of the selection layer
        scores = re.search(r"attn_resident_kernel<[^>]*, true>", name) is not None or \
            "ELb1EEEv" in name
        return "attention_res_scores" if scores else "attention_res"
    if "attn_reg_kernel" in name:
        for qb, q in (("8", "q256"), ("4", "q128"), ("2", "q64"), ("1", "q32")):
            if f"attn_reg_kernelILi{qb}E" in name or f"attn_reg_kernel<{qb}," in name:
                return f"attention_{q}"
    if "attn_mfma_kernel" in name:
        for nw, q in (("4", "q128"), ("2", "q64"), ("1", "q32")):
            if f"ELi{nw}ELb" in name or f"ELi{nw}EEEv" in name or f", {nw}, " in name:
                return f"attention_{q}"
    for key, cls in (("gather_ln_kernel", "gather_ln"), ("attn_scores_kernel", "attn_scores"),
                     ("select_topk_kernel", "select_topk"), ("decoder_input_kernel", "decoder_input"),
                     ("row_map_kernel", "row_map"), ("fill_zero_kernel", "fill_zero")):
        if key in name:
            return cls
    return None


def counter_rows(path: str) -> list:
    """Per-dispatch records of a rocprofv3 --pmc CSV, in dispatch order, each
    with its timing class split by layer kind.  The run is `--steps 1
    --warmup 1` (steps 0 and 1) or `--steps 1 --warmup 0` (step 0): step 0 is a
    full step (every token active in every layer), so the (class, grid) pairs
    it launches are the full-layer launches; any later dispatch with a pair it
    never launched belongs to a cache-aware layer (class + "_ca").  Steps start
    at the decoder-input kernel, launched once per step."""
    import csv
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
    out = []
    for key, r in zip(dispatch_classes(rows), rows):
        if key is not None:
            out.append((key, float(r["Counter_Value"])))
    return out


# Classes that the library never times as cache-aware: the score pass runs at
# the selection layer (every token active), the selection and the decoder
# input outside the step; the row map has the same grid in both kinds of call.
NOT_SPLIT = {"attn_scores", "attention_res_scores", "select_topk", "decoder_input", "fill_zero",
             "row_map"}


def dispatch_classes(rows: list) -> list:
    """Timing class (split by layer kind) of each dispatch record, in order;
    see counter_rows."""
    starts = [i for i, r in enumerate(rows) if "decoder_input_kernel" in r["Kernel_Name"]]
    step0_end = starts[1] if len(starts) > 1 else len(rows)
    full = {(counter_class(r["Kernel_Name"]), r["Grid_Size"]) for r in rows[:step0_end]}
    out = []
    for r in rows:
        c = counter_class(r["Kernel_Name"])
        if c is None or c in NOT_SPLIT or (c, r["Grid_Size"]) in full:
            out.append(c)
        else:
            out.append(c + "_ca")
    return out


def ingest_mfma(path: str, simds: int, xcds: int) -> dict:
    """MFMA utilisation per timing class from a rocprofv3 --pmc run of
    SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE and SQ_BUSY_CU_CYCLES over the
    bench's first steps: per dispatch, MFMA-busy cycles summed over the SIMDs
    / (GPU-active cycles x SIMDs), averaged over the class's dispatches (the
    MfmaUtil metric of rocprofv3).  The CSV sums GRBM_GUI_ACTIVE over the
    XCDs, each of which counts the whole dispatch, so it is divided by their
    number (the metric takes the maximum instead)."""
    import collections
    import csv
    per = collections.defaultdict(dict)
    first = {}
    for r in csv.DictReader(open(path)):
        d = int(r["Dispatch_Id"])
        per[d][r["Counter_Name"]] = float(r["Counter_Value"])
        first.setdefault(d, r)
    order = sorted(per)
    keys = dispatch_classes([first[d] for d in order])
    agg = collections.defaultdict(list)
    for d, key in zip(order, keys):
        c = per[d]
        if key is None or not c.get("GRBM_GUI_ACTIVE"):
            continue
        active = c["GRBM_GUI_ACTIVE"] / xcds
        agg[key].append((c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (active * simds),
                         c.get("SQ_BUSY_CU_CYCLES", 0.0), active))
    out = {}
    for key, v in sorted(agg.items()):
        out[key] = {"mfma_util": sum(u for u, _, _ in v) / len(v), "dispatches": len(v),
                    "gpu_active_cycles": sum(g for _, _, g in v) / len(v),
                    "source_sha": source_hash(key)}
    return out


def ingest_counters(paths: list, commands: dict) -> dict:
    """profiles/traffic.json entries from four rocprofv3 --pmc CSVs: FETCH_SIZE and
    WRITE_SIZE of the bench's first steps (counter_rows), then of the plain copy
    (--calibrate-copy).  Counter KiB per dispatch are scaled by known bytes /
    counter for the copy.  Full-layer classes have one shape in every step,
    so their per-launch bytes are those of every full-layer launch; a
    cache-aware class's bytes are those of step 1's active sets."""
    import collections

    def per_class(path):
        agg = collections.defaultdict(list)
        for key, v in counter_rows(path):
            agg[key].append(v * 1024.0)
        return agg

    def copy_bytes(path):
        import csv
        v = [float(r["Counter_Value"]) * 1024.0 for r in csv.DictReader(open(path))
             if "copyBuffer" in r["Kernel_Name"]]
        return max(v)

    fetch, write = per_class(paths[0]), per_class(paths[1])
    copy_n = commands["copy_bytes"]
    sf, sw = copy_n / copy_bytes(paths[2]), copy_n / copy_bytes(paths[3])
    out = {}
    for c in sorted(set(fetch) | set(write)):
        f = sum(fetch.get(c, [0.0])) / max(1, len(fetch.get(c, [])))
        w = sum(write.get(c, [0.0])) / max(1, len(write.get(c, [])))
        out[c] = {"fetch_bytes": f * sf, "write_bytes": w * sw, "bytes_per_launch": f * sf + w * sw,
                  "dispatches": len(fetch.get(c, [])), "source_sha": source_hash(c)}
    return {"scale": {"fetch": sf, "write": sw}, "classes": out}


def kernel_rates(prof: dict, dtype: str) -> dict:
    out = {}
    peak_mfma = PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_FP32_TFLOPS
    for name, e in prof.items():
        avg_s = e["ms"] * 1e-3 / e["launches"]
        base = name[:-3] if name.endswith("_ca") else name   # cache-aware layers' classes
        # attention of a cache-aware layer: about |A| flop per byte of K/V, far
        # below the ridge point (312), so HBM-bound whatever its query chunk
        ca_attention = name.endswith("_ca") and base.startswith("attention_q")
        if base in HBM_BOUND or e["flops"] == 0 or ca_attention:
            ach = e["bytes"] / e["launches"] / avg_s / 1e9
            out[name] = {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": ach / PEAK_HBM_GBS}
        else:
            ach = e["flops"] / e["launches"] / avg_s / 1e12
            out[name] = {"bound": "mfma", "achieved": ach, "peak": peak_mfma, "unit": "TFLOP/s",
                         "frac": ach / peak_mfma}
        out[name].update({"launches": e["launches"], "avg_us": avg_s * 1e6,
                          "total_ms": e["ms"]})
    return out


def cpu_baseline(cfg, weights, budget_s: float, n_full_sched: int, n_ca_sched: int):
    """Time the fp64 oracle on image 0's first decoding steps until `budget_s`
    seconds have passed (at least one full and one cache-aware step), and
    extrapolate images/s over the whole schedule."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import schedule as osched
    from oracle import step as ostep
    from paper_2506_12035_amd import workload

    p64 = [{k: np.asarray(v, np.float64) for k, v in w.items()} for w in weights]
    emb = workload.embeddings(cfg, 1)
    order = workload.orders(cfg, 1)[0]
    H, N, dh = cfg.n_heads, cfg.n_tokens, cfg.head_dim
    kcs = [np.zeros((H, N, dh)) for _ in p64]
    vcs = [np.zeros((H, N, dh)) for _ in p64]
    t_full, t_ca = [], []
    start = time.perf_counter()
    t = 0
    while t < cfg.n_steps:
        gen = osched.generating_tokens(order, cfg.n_buf, cfg.n_steps, t)
        cache = osched.caching_tokens(order, cfg.n_buf, cfg.n_steps, t)
        known = osched.known_before(order, cfg.n_buf, cfg.n_steps, t)
        full = osched.is_full_step(t, cfg.full_every)
        k = ostep.refresh_count("ratio", cfg.ratio_bp, N, len(gen), len(cache))
        t0 = time.perf_counter()
        x = ostep.decoder_input(emb.cls[0], emb.value[0], emb.mask, emb.pos, known, cfg.n_buf)
        res = ostep.marche_step(p64, x, kcs, vcs, gen, cache, n_heads=H, eps=cfg.ln_eps,
                                sel_layer=cfg.sel_layer, full=full, k_refresh=k)
        (t_full if full else t_ca).append(time.perf_counter() - t0)
        kcs, vcs = res.k_caches, res.v_caches
        t += 1
        log(f"  cpu oracle step {t - 1} ({'full' if full else 'cache-aware'}): "
            f"{(t_full if full else t_ca)[-1]:.2f} s")
        if t_full and t_ca and time.perf_counter() - start > budget_s:
            break
    tf, tc = statistics.mean(t_full), statistics.mean(t_ca)
    per_image = n_full_sched * tf + n_ca_sched * tc
    threads = sum(i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas")
    return {
        "value": 1.0 / per_image,
        "unit": "images/s",
        "cores": threads or len(os.sched_getaffinity(0)),
        "kind": "oracle",
        "sample": (f"fp64 numpy oracle, image 0, steps 0..{t - 1} of the 64-step schedule "
                   f"({len(t_full)} full at {tf:.2f} s, {len(t_ca)} cache-aware at {tc:.2f} s); "
                   f"images/s = 1 / ({n_full_sched} x full + {n_ca_sched} x cache-aware); "
                   f"images are independent, so the batch adds no per-image work"),
    }


def timed(eng, steps, first, T):
    import torch
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(steps):
        eng.step((first + i) % T)
        evs[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = [evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(steps)]
    kinds = [eng.plans[(first + i) % T].full for i in range(steps)]
    return wall, per, kinds


APPB_SIZES = ((32, 256), (64, 256), (128, 256), (32, 512), (32, 1024), (64, 1024),
              (256, 1024), (32, 2048))


def appb_main(args) -> int:
    """Appendix B on MI355X.  Per (n_active, n_cached): inputs resident in HBM
    (several copies rotated so that no call finds them in the 256 MB memory-side
    cache), then
      concat      = concatenate K_A|K_C and V_A|V_C (this library's copy kernel),
                    then attend over one segment;
      torch_cat   = the same with torch.cat as the concatenation;
      two_segment = one pass over the two segments' own buffers (the method);
      resident    = attention over one buffer that already holds both segments
                    (the library's production layout: the QKV epilogue writes the
                    fresh rows into the cache, so no merge step exists at all).
    Each timed with HIP events over 20 calls after 3 warm-up calls."""
    import numpy as np
    import torch

    from paper_2506_12035_amd import binding, workload

    B, H, dh = 128, 16, 64
    D = H * dh
    bf = torch.bfloat16
    stream = torch.cuda.current_stream()
    rows = []
    for na, nc in APPB_SIZES:
        c = workload.segment_case(B, H, dh, na, nc)
        per_copy = 2 * (2 * B * na * D + 2 * B * (na + nc) * D)
        copies = max(2, int(np.ceil(512e6 / per_copy)))
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(bf)
        base = [dev(c.q), dev(c.k_a), dev(c.v_a), dev(c.k_c), dev(c.v_c)]
        sets = [[t.clone() for t in base] for _ in range(copies)]
        resident = [(torch.cat([s_[1], s_[3]], dim=2).contiguous(),
                     torch.cat([s_[2], s_[4]], dim=2).contiguous()) for s_ in sets]
        o = torch.empty(B, na, D, device="cuda", dtype=bf)
        wsb = binding.attention_workspace_bytes(B, H, dh, na, nc, binding.MARCHE_BF16,
                                                binding.MARCHE_ATTN_CONCAT)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")

        def run(kind, i):
            q, ka, va, kc, vc = sets[i % copies]
            if kind == "concat":
                binding.attention_segments(q, o, na, ka, va, na, kc, vc, nc, B, H, dh,
                                           binding.MARCHE_BF16, binding.MARCHE_ATTN_CONCAT, ws, wsb,
                                           stream)
            elif kind == "two_segment":
                binding.attention_segments(q, o, na, ka, va, na, kc, vc, nc, B, H, dh,
                                           binding.MARCHE_BF16, binding.MARCHE_ATTN_TWO_SEGMENT,
                                           None, 0, stream)
            elif kind == "torch_cat":
                kr = torch.cat([ka, kc], dim=2)
                vr = torch.cat([va, vc], dim=2)
                binding.attention_segments(q, o, na, kr, vr, na + nc, None, None, 0, B, H, dh,
                                           binding.MARCHE_BF16, binding.MARCHE_ATTN_TWO_SEGMENT,
                                           None, 0, stream)
            else:
                kr, vr = resident[i % copies]
                binding.attention_segments(q, o, na, kr, vr, na + nc, None, None, 0, B, H, dh,
                                           binding.MARCHE_BF16, binding.MARCHE_ATTN_TWO_SEGMENT,
                                           None, 0, stream)

        res = {}
        for kind in ("concat", "torch_cat", "two_segment", "resident"):
            for i in range(3):
                run(kind, i)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for i in range(20):
                run(kind, i)
            e1.record(stream)
            torch.cuda.synchronize()
            res[kind] = e0.elapsed_time(e1) / 20 * 1e3
        attn_bytes = 2.0 * (2 * B * na * D + 2 * B * (na + nc) * D)
        row = {"n_active": na, "n_cached": nc, "us": {k: round(v, 1) for k, v in res.items()},
               "two_segment_vs_concat": round(1 - res["two_segment"] / res["concat"], 4),
               "two_segment_vs_torch_cat": round(1 - res["two_segment"] / res["torch_cat"], 4),
               "resident_vs_concat": round(1 - res["resident"] / res["concat"], 4),
               "two_segment_hbm_frac": round(attn_bytes / (res["two_segment"] * 1e-6) / 1e9
                                             / PEAK_HBM_GBS, 4)}
        log(f"[appb] {na:4d} / {nc:5d}: concat {res['concat']:8.1f} us, torch.cat+attend "
            f"{res['torch_cat']:8.1f} us, two-segment "
            f"{res['two_segment']:8.1f} us ({100 * row['two_segment_vs_concat']:+.1f}%), resident "
            f"{res['resident']:8.1f} us ({100 * row['resident_vs_concat']:+.1f}%), two-segment at "
            f"{100 * row['two_segment_hbm_frac']:.1f}% of HBM")
        rows.append(row)
        del sets, resident, ws
        torch.cuda.empty_cache()
    print(json.dumps({"appendix_b": rows, "batch": B, "heads": H, "head_dim": dh,
                      "dtype": "bf16"}), flush=True)
    return 0


def e2e_main(args) -> int:
    """Whole MAR generations (encoder, cache-aware decoder, sampler) at MAR-L
    sizes: seconds per image for the paper's schedule and for full recompute of
    the decoder with the same encoder and sampler, with a per-phase split."""
    import torch

    from paper_2506_12035_amd import binding, driver, workload

    mc = workload.MAR_CONFIGS[args.e2e_config]
    log(f"[e2e] {mc.name}: building the engine")
    eng = driver.MarEngine(mc, micro_batches=args.micro_batches)
    B, T = eng.B, mc.dec.n_steps

    def generation():
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        eng.generate()
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    def phases():
        ev = {k: [] for k in ("encoder", "decoder", "sampler")}
        eng.tok.zero_()
        for t in eng.steps:
            e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            e[0].record()
            eng.encode(t)
            e[1].record()
            eng.dec.step(t, build_input=False)
            e[2].record()
            eng.sample(t)
            e[3].record()
            for i, k in enumerate(ev):
                ev[k].append((e[i], e[i + 1]))
        torch.cuda.synchronize()
        return {k: sum(a.elapsed_time(b) for a, b in v) for k, v in ev.items()}

    log("[e2e] warmup generation")
    generation()
    log("[e2e] timed generation")
    wall = generation()
    split = phases()
    log(f"[e2e] {wall / B * 1e3:.2f} ms/image; per generation (ms): {split}")
    binding.profile_reset()
    binding.profile_enable(True)
    eng.generate()
    prof = binding.profile_collect()
    binding.profile_enable(False)
    rates = kernel_rates(prof, mc.dec.dtype)

    eng.dec.set_schedule(1, "ratio", 10000)
    generation()
    fwall = generation()
    fsplit = phases()
    eng.dec.set_schedule(mc.dec.full_every, "ratio", mc.dec.ratio_bp)
    log(f"[e2e] full recompute: {fwall / B * 1e3:.2f} ms/image -> speedup {fwall / wall:.3f}")
    out = {
        "metric": "MAR end-to-end generation latency (encoder + decoder + sampler), s/image",
        "value": wall / B, "unit": "s/image", "higher_is_better": False, "n_gpus": 1,
        "images_per_s": B / wall, "dtype": mc.dec.dtype, "data": "synthetic",
        "config": {"workload": mc.name, "batch": B, "decode_steps": T,
                   "encoder_layers": mc.enc_layers, "decoder_layers": mc.dec.n_layers,
                   "d_model": mc.dec.d_model, "head_blocks": mc.head_blocks,
                   "head_width": mc.head_width, "token_channels": mc.c_tok,
                   "sampling_steps": mc.sample_steps, "refresh_ratio": mc.dec.ratio_bp / 10000,
                   "full_every": mc.dec.full_every, "sel_layer": mc.dec.sel_layer,
                   "micro_batches": args.micro_batches},
        "phase_ms_per_generation": split,
        "full_recompute": {"s_per_image": fwall / B, "phase_ms_per_generation": fsplit},
        "speedup_vs_full_recompute": fwall / wall,
        "kernels": rates,
    }
    print(json.dumps(out), flush=True)
    return 0


def single_block_main(args) -> int:
    """The single-block fp32 case (one pre-LN block, D 768, 12 heads, N 320,
    batch 1, 16 generating + 16 refresh tokens active): one cache-aware step
    with the attention-mass scores, then the top-16 refresh selection over
    the tokens outside A.  Latency per step (both calls), HIP events on the
    launch stream, median of the timed repetitions; the fp64 oracle's same
    step on this host's cores beside it."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    from paper_2506_12035_amd import binding, workload

    cfg = workload.CONFIGS[1]
    case = workload.single_block_case(cfg)
    p = workload.layer_weights(cfg, 0)
    N, D, H, dh, F = cfg.n_tokens, cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_mlp
    dev = "cuda"
    model = binding.make_model(1, D, H, dh, F, N, binding.MARCHE_F32, cfg.ln_eps)
    params = {k: torch.from_numpy(np.ascontiguousarray(v, np.float32)).to(dev) for k, v in p.items()}
    layers = binding.make_layers([params])
    k = torch.from_numpy(case.k_cache.reshape(-1)).to(dev)
    v = torch.from_numpy(case.v_cache.reshape(-1)).to(dev)
    cache = binding.kv_cache_init(model, 1, k, v, k.numel() * 4)
    x0 = torch.from_numpy(case.x).to(dev)
    x = x0.clone()
    act = case.active[0].astype(np.int32)
    a = len(act)
    idx = torch.from_numpy(act).to(dev)
    off = torch.tensor([0, a], dtype=torch.int32, device=dev)
    gen = torch.tensor([case.n_gen], dtype=torch.int32, device=dev)
    scores = torch.empty(1, H, N, device=dev)
    wsb = binding.workspace_bytes(model, 1, a)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    out = torch.empty(case.k_top, dtype=torch.int32, device=dev)
    ooff = torch.zeros(1, dtype=torch.int32, device=dev)
    eoff = torch.tensor([0, a], dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        binding.marche_step(model, layers, cache, 0, 1, 1, x, idx, off, gen, a, a, case.n_gen,
                            scores, 0, ws, wsb, stream=stream)
        binding.select_refresh(scores, H, idx, eoff, 1, N, case.k_top, out, ooff, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    n = max(args.steps, 1)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    ev[0].record(stream)
    for i in range(n):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(n)]
    us = statistics.median(per)
    # the step's kernels alone (library timing hooks), one pass
    binding.profile_reset()
    binding.profile_enable(True)
    step()
    torch.cuda.synchronize()
    binding.profile_enable(False)
    prof = binding.profile_collect()
    kern_us = sum(e["ms"] for e in prof.values()) * 1e3
    log(f"[bench] single block: {us:.1f} us per step (median of {n}), kernels {kern_us:.1f} us")

    # fp64 oracle: the same step on this host
    from oracle import block, select
    p64 = {kk: np.asarray(vv, np.float64) for kk, vv in p.items()}
    cpu = []
    t_end = time.perf_counter() + args.cpu_budget_s
    while not cpu or (time.perf_counter() < t_end and len(cpu) < 50):
        t0 = time.perf_counter()
        r = block.cache_aware_layer(p64, case.x[0], case.k_cache[0], case.v_cache[0], list(act),
                                    list(act[:case.n_gen]), n_heads=H, eps=cfg.ln_eps, score=True)
        select.select_topk(select.total_scores(r.scores), list(act), case.k_top)
        cpu.append(time.perf_counter() - t0)
    threads = sum(i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas")
    weight_bytes = 4.0 * (3 * D * D + D * D + 2 * D * F)
    res = {
        "metric": "single-block cache-aware step + top-16 refresh latency (us)", "value": us,
        "unit": "us", "higher_is_better": False, "n_gpus": 1, "steps": n, "warmup": args.warmup,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": cfg.name, "batch": 1, "n_tokens": N, "d_model": D, "n_heads": H,
                   "active": a, "generating": case.n_gen, "top_k": case.k_top},
        "kernels_us": {kk: vv["ms"] * 1e3 / vv["launches"] for kk, vv in prof.items()},
        "kernel_sum_us": kern_us,
        "weight_stream_bound_us": weight_bytes / (PEAK_HBM_GBS * 1e9) * 1e6,
        "cpu_baseline": {"value": statistics.median(cpu) * 1e6, "unit": "us", "cores": threads,
                         "kind": "oracle",
                         "sample": f"fp64 oracle cache_aware_layer + select_topk, median of {len(cpu)}"},
    }
    print(json.dumps(res), flush=True)
    return 0


def drift_main(args) -> int:
    """A free-running generation of one image against the fp64 oracle (not a
    parity gate): the GPU runs every step of the whole batch with its own
    refresh sets; the oracle runs image 0's steps from the same seeded inputs
    with its own.  Per step: the relative error of z (the last layer's rows
    at the generating tokens) and how many of the oracle's refresh tokens the
    GPU also chose."""
    import numpy as np
    import torch

    from oracle import schedule as osched
    from oracle import step as ostep
    from paper_2506_12035_amd import driver, workload

    cfg = workload.CONFIGS[args.config]
    b = 0
    weights = workload.all_weights(cfg)
    eng = driver.Engine(cfg, weights=weights, micro_batches=args.micro_batches)
    p64 = [{k: np.asarray(v, np.float64) for k, v in w.items()} for w in weights]
    emb = workload.embeddings(cfg)
    order = workload.orders(cfg)[b]
    H, N, dh = cfg.n_heads, cfg.n_tokens, cfg.head_dim
    kcs = [np.zeros((H, N, dh)) for _ in p64]
    vcs = [np.zeros((H, N, dh)) for _ in p64]
    rows = []
    for t in range(cfg.n_steps):
        eng.step(t)
        torch.cuda.synchronize()
        gen = osched.generating_tokens(order, cfg.n_buf, cfg.n_steps, t)
        cache = osched.caching_tokens(order, cfg.n_buf, cfg.n_steps, t)
        known = osched.known_before(order, cfg.n_buf, cfg.n_steps, t)
        full = osched.is_full_step(t, cfg.full_every)
        k = ostep.refresh_count("ratio", cfg.ratio_bp, N, len(gen), len(cache))
        x_in = ostep.decoder_input(emb.cls[b], emb.value[b], emb.mask, emb.pos, known, cfg.n_buf)
        res = ostep.marche_step(p64, x_in, kcs, vcs, gen, cache, n_heads=H, eps=cfg.ln_eps,
                                sel_layer=cfg.sel_layer, full=full, k_refresh=k)
        kcs, vcs = res.k_caches, res.v_caches
        z_gpu = eng.x[b].cpu().numpy().astype(np.float64)[gen]
        z_err = float(np.abs(z_gpu - res.z).max() / np.abs(res.z).max())
        row = {"t": t, "full": full, "z_rel_err": z_err}
        if not full:
            r_gpu = set(int(v) for v in eng.refresh_lists(t)[b])
            r_ora = set(res.refresh)
            row["refresh_agree"] = len(r_gpu & r_ora) / max(len(r_ora), 1)
        rows.append(row)
        log(f"[drift] step {t:2d} {'full' if full else 'cache-aware'}: z rel err {z_err:.2e}"
            + (f", refresh agreement {row['refresh_agree']:.3f}" if not full else ""))
    agree = [r["refresh_agree"] for r in rows if "refresh_agree" in r]
    print(json.dumps({"drift": rows, "workload": cfg.name, "image": b,
                      "mean_refresh_agreement": statistics.mean(agree) if agree else None,
                      "max_z_rel_err": max(r["z_rel_err"] for r in rows)}), flush=True)
    return 0


def trace_summary_main(args) -> int:
    """Markdown summary of a rocprofv3 --kernel-trace run of the default bench
    (kernel_trace.csv and the run's stderr+stdout with its JSON line): per
    timing class, the trace's average duration over the dispatches of the
    instrumented pass (the class's last `launches` dispatches, the pass being
    the last kernels the bench launches) beside the live HIP-event average of
    the same launches, and the whole trace's totals."""
    import csv
    import collections
    trace_csv, log_path = args.trace_summary
    rows = sorted(csv.DictReader(open(trace_csv)), key=lambda r: int(r["Dispatch_Id"]))
    for r in rows:
        r["Grid_Size"] = r["Grid_Size_X"]
    keys = dispatch_classes(rows)
    dur = collections.defaultdict(list)
    for k, r in zip(keys, rows):
        if k is not None:
            dur[k].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    line = [ln for ln in open(log_path) if ln.startswith("{")][-1]
    live = json.loads(line)
    kern = live.get("kernels", {})
    dom = live.get("roofline", {}).get("kernel")
    out = ["| Class | Live launches | Live avg us | Trace avg us (same launches) | Trace dispatches | Trace total ms |",
           "|---|---:|---:|---:|---:|---:|"]
    for k, v in sorted(kern.items(), key=lambda kv: -kv[1]["total_ms"]):
        d = dur.get(k, [])
        n = v["launches"]
        tail = d[-n:] if len(d) >= n else d
        tavg = sum(tail) / len(tail) if tail else float("nan")
        mark = " (dominant)" if k == dom else ""
        out.append(f"| {k}{mark} | {n} | {v['avg_us']:.1f} | {tavg:.1f} | {len(d)} | {sum(d) / 1e3:.2f} |")
    print("\n".join(out))
    return 0


def ingest_main(args) -> int:
    from paper_2506_12035_amd import workload

    cfg = workload.CONFIGS[args.config]
    fcsv, wcsv, cf, cw = args.ingest_counters
    rec = ingest_counters([fcsv, wcsv, cf, cw], {"copy_bytes": 1024 * (1 << 20)})
    path = os.path.join(ROOT, "profiles", "traffic.json")
    allrec = {}
    if os.path.exists(path):
        with open(path) as f:
            allrec = json.load(f)
    allrec[cfg.name] = rec
    with open(path, "w") as f:
        json.dump(allrec, f, indent=1, sort_keys=True)
    print(json.dumps(rec, indent=1))
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=64)
    ap.add_argument("--config", type=int, default=3, help="workload id (2: MAR-B, 3: MAR-L, 4: MAR-H, 5: high-res)")
    ap.add_argument("--batch", type=int, default=None)
    ap.add_argument("--micro-batches", type=int, default=2,
                    help="run every decoding step as this many ranges of consecutive images, "
                         "each on its own HIP stream (default 2; 1: the whole batch in one call)")
    ap.add_argument("--range-sizes", type=str, default=None,
                    help="comma-separated image count of each range (overrides --micro-batches)")
    ap.add_argument("--ratio-bp", type=int, default=None, help="refresh ratio in basis points")
    ap.add_argument("--full-every", type=int, default=None)
    ap.add_argument("--no-full-recompute", action="store_true")
    ap.add_argument("--no-roofline", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=20.0)
    ap.add_argument("--strategy", default="marche",
                    help="active-set construction: marche, low-attention, random, no-caching, "
                         "no-generating")
    ap.add_argument("--schedule-sweep", action="store_true",
                    help="also time one generation per schedule variant: selection layer 1-4, "
                         "full-refresh period 2-7 and off, fixed 64-token budget, and each "
                         "active-set strategy (latency only)")
    ap.add_argument("--ratio-sweep", action="store_true",
                    help="also time one generation at each refresh ratio of the MAR-H sweep "
                         "(0, 5, 10, 25, 100%%)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB five times (the "
                         "reference for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE) and exit")
    ap.add_argument("--appb", action="store_true",
                    help="only run Appendix B's comparison: attention over an active and a cached "
                         "segment, concatenate-then-attend vs the two-segment pass vs one resident "
                         "buffer, MAR-L heads at batch 128, over a sweep of segment lengths")
    ap.add_argument("--e2e", action="store_true",
                    help="only time whole MAR generations: encoder over the known tokens, the "
                         "cache-aware decoder and the sampler (s/image), against full recompute "
                         "of the decoder with the same encoder and sampler")
    ap.add_argument("--e2e-config", default="mar-l-e2e", help="whole-model workload name")
    ap.add_argument("--repeats", type=int, default=5,
                    help="after the timed K steps, time the same K steps this many more times "
                         "and report their median and spread beside the value (0: off)")
    ap.add_argument("--drift", action="store_true",
                    help="only run a free-running generation against the fp64 oracle for image "
                         "0 (relative error of z and refresh-set agreement per step); not a gate")
    ap.add_argument("--trace-summary", nargs=2, default=None, metavar=("TRACE_CSV", "BENCH_LOG"),
                    help="print a markdown table of a rocprofv3 --kernel-trace run of the bench "
                         "against the live timing of the same launches; no GPU needed")
    ap.add_argument("--ingest-mfma", default=None, metavar="MFMA_CSV",
                    help="write profiles/mfma_util.json from a rocprofv3 --pmc run of "
                         "SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE SQ_BUSY_CU_CYCLES over the "
                         "first steps (--steps 1 --warmup 1); no GPU needed")
    ap.add_argument("--ingest-counters", nargs=4, default=None,
                    metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="write profiles/traffic.json from rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE "
                         "CSVs of a run of the first steps (--steps 1 --warmup 1: a full and a "
                         "cache-aware step) and of --calibrate-copy 1024; no GPU needed")
    args = ap.parse_args()
    if args.ingest_counters:
        return ingest_main(args)
    if args.trace_summary:
        return trace_summary_main(args)
    if args.ingest_mfma:
        from paper_2506_12035_amd import workload
        import csv as _csv
        agent = args.ingest_mfma.replace("counter_collection", "agent_info")
        gpu = [r for r in _csv.DictReader(open(agent)) if r["Agent_Type"] == "GPU"][0]
        simds, xcds = int(gpu["Simd_Count"]), int(gpu["Num_Xcc"])
        rec = {"simds": simds, "xcds": xcds,
               "classes": ingest_mfma(args.ingest_mfma, simds, xcds)}
        path = os.path.join(ROOT, "profiles", "mfma_util.json")
        allrec = json.load(open(path)) if os.path.exists(path) else {}
        allrec[workload.CONFIGS[args.config].name] = rec
        with open(path, "w") as f:
            json.dump(allrec, f, indent=1, sort_keys=True)
        print(json.dumps(rec, indent=1))
        return 0

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the decode step shards over images without collectives; this benchmark "
              "measures one GPU's share", file=sys.stderr)
        return 2
    if args.steps < 1 or args.warmup < 0:
        print("--steps must be >= 1 and --warmup >= 0", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2506_12035_amd import binding, driver, schedule, workload

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.appb:
        return appb_main(args)
    if args.e2e:
        return e2e_main(args)
    if args.drift:
        return drift_main(args)
    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.arange(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n * 4, "repeats": 5}), flush=True)
        return 0
    cfg = workload.CONFIGS[args.config]
    if args.config == 1:
        return single_block_main(args)
    if args.ratio_bp is not None:
        cfg = cfg.with_(ratio_bp=args.ratio_bp)
    if args.full_every is not None:
        cfg = cfg.with_(full_every=args.full_every)
    B = cfg.batch if args.batch is None else args.batch
    T = cfg.n_steps

    log(f"[bench] workload {cfg.name}: generating weights")
    weights = workload.all_weights(cfg)
    log("[bench] uploading")
    sizes = [int(v) for v in args.range_sizes.split(",")] if args.range_sizes else None
    eng = driver.Engine(cfg, batch=B, weights=weights, strategy=args.strategy,
                        micro_batches=args.micro_batches, range_sizes=sizes)
    torch.cuda.synchronize()

    log(f"[bench] warmup {args.warmup} steps")
    for i in range(args.warmup):
        eng.step(i % T)
    torch.cuda.synchronize()
    log(f"[bench] timing {args.steps} steps")
    first = args.warmup % T
    wall, per, kinds = timed(eng, args.steps, first, T)
    value = B * args.steps / T / wall
    step_us = {}
    full_us = [p for p, f in zip(per, kinds) if f]
    ca_us = [p for p, f in zip(per, kinds) if not f]
    if full_us:
        step_us["full"] = statistics.median(full_us)
    if ca_us:
        step_us["cache_aware"] = statistics.median(ca_us)
    log(f"[bench] {value:.2f} images/s, {wall / args.steps * 1e3:.3f} ms/step, {step_us}")
    reps = []
    for r_ in range(args.repeats):
        # the same K steps again (the state of each step is rebuilt from its
        # input; the work does not depend on the values)
        rwall, _, _ = timed(eng, args.steps, first, T)
        reps.append(B * args.steps / T / rwall)

    out = {
        "metric": METRIC, "value": value, "unit": "images/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": cfg.name, "batch": B, "n_tokens": cfg.n_tokens,
                   "n_image_tokens": cfg.n_img, "n_layers": cfg.n_layers,
                   "d_model": cfg.d_model, "n_heads": cfg.n_heads, "head_dim": cfg.head_dim,
                   "refresh_ratio": cfg.ratio_bp / 10000, "sel_layer": cfg.sel_layer,
                   "full_every": cfg.full_every, "decode_steps": T, "strategy": args.strategy,
                   "micro_batches": len(eng.ranges),
                   "range_sizes": [n for _, n in eng.ranges],
                   "full_steps_in_schedule": sum(p.full for p in eng.plans)},
        "step_us": step_us,
    }
    if reps:
        out["repeats"] = {"n": len(reps), "median_images_per_s": statistics.median(reps),
                          "min": min(reps), "max": max(reps),
                          "note": "the same timed steps repeated after the value's timing"}
        log(f"[bench] {len(reps)} repeats: median {statistics.median(reps):.2f} images/s "
            f"({min(reps):.2f} - {max(reps):.2f})")

    if not args.no_full_recompute:
        eng.set_schedule(1, "ratio", 10000)
        n = min(args.steps, T)
        for i in range(2):
            eng.step(i)
        log(f"[bench] full recompute: timing {n} steps")
        fwall, fper, _ = timed(eng, n, 0, T)
        fv = B * n / T / fwall
        out["full_recompute"] = {"images_per_s": fv, "step_us": statistics.median(fper)}
        out["speedup_vs_full_recompute"] = value / fv
        log(f"[bench] full recompute {fv:.2f} images/s -> speedup {value / fv:.3f}")
        eng.set_schedule(cfg.full_every, "ratio", cfg.ratio_bp)

    if args.schedule_sweep:
        variants = [dict(sel_layer=s_) for s_ in (1, 2, 3, 4)]
        variants += [dict(full_every=f_) for f_ in (2, 3, 4, 5, 6, 7, 0)]
        variants += [dict(policy="fixed", budget=64)]
        variants += [dict(strategy=st) for st in driver.STRATEGIES]
        base = dict(sel_layer=cfg.sel_layer, full_every=cfg.full_every, policy="ratio",
                    budget=cfg.ratio_bp, strategy=args.strategy)
        rows = []
        for v in variants:
            conf = dict(base, **v)
            eng.configure(**conf)
            for i in range(T):
                eng.step(i)
            swall, sper, skinds = timed(eng, T, 0, T)
            ca = [p for p, f in zip(sper, skinds) if not f]
            rows.append({**v, "images_per_s": B / swall,
                         "cache_aware_step_us": statistics.median(ca) if ca else None,
                         "full_steps": sum(skinds)})
            log(f"[bench] {v}: {B / swall:.2f} images/s")
        out["schedule_sweep"] = rows
        eng.configure(**base)

    if args.ratio_sweep:
        sweep = []
        for bp in workload.MAR_H_RATIO_SWEEP_BP:
            eng.set_schedule(cfg.full_every, "ratio", bp)
            for i in range(T):
                eng.step(i)
            swall, sper, skinds = timed(eng, T, 0, T)
            ca = [p for p, f in zip(sper, skinds) if not f]
            sweep.append({"refresh_ratio": bp / 10000, "images_per_s": B / swall,
                          "cache_aware_step_us": statistics.median(ca) if ca else None,
                          "mean_active": statistics.mean(p.g + p.n + p.k for p in eng.plans if not p.full)})
            log(f"[bench] ratio {bp / 100:.0f}%: {B / swall:.2f} images/s")
        out["ratio_sweep"] = sweep
        eng.set_schedule(cfg.full_every, "ratio", cfg.ratio_bp)

    if not args.no_roofline:
        # the same steps and image ranges, the ranges one after another on one
        # stream, so that each kernel's duration is its own and not stretched
        # by a kernel of another range sharing the GPU
        log(f"[bench] instrumented pass over the same {args.steps} steps "
            f"({len(eng.ranges)} image range(s) in turn on one stream)")
        eng.overlap = False
        for i in range(args.warmup):
            eng.step(i % T)
        torch.cuda.synchronize()
        binding.profile_reset()
        binding.profile_enable(True)
        for i in range(args.steps):
            eng.step((first + i) % T)
        torch.cuda.synchronize()
        binding.profile_enable(False)
        eng.overlap = True
        prof = binding.profile_collect()
        rates = kernel_rates(prof, cfg.dtype)
        dom = max(rates, key=lambda k: rates[k]["total_ms"])
        r = rates[dom]
        tr = traffic_for(dom, cfg.name)
        out["roofline"] = {"kernel": dom, "bound": r["bound"], "achieved": r["achieved"],
                           "peak": r["peak"], "unit": r["unit"], "frac": r["frac"],
                           "traffic": tr, "avg_us": r["avg_us"], "launches": r["launches"]}
        out["kernels"] = {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv)
                              for kk, vv in v.items()} for k, v in
                          sorted(rates.items(), key=lambda kv: -kv[1]["total_ms"])}
        log(f"[bench] dominant kernel {dom}: {r['achieved']:.1f} {r['unit']} ({r['frac']:.1%})")

    del eng
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (fp64 oracle)")
        n_full = sum(schedule.full_step(t, cfg.full_every) for t in range(T))
        out["cpu_baseline"] = cpu_baseline(cfg, weights, args.cpu_budget_s, n_full, T - n_full)

    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
