"""Benchmark of the hybrid weighted sum on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config vgg11] [--no-cpu-baseline]

A step is one fiona_hybrid_linear call over the whole layer (every output,
both polynomials, every limb and coefficient), inputs already resident in HBM.
The default workload is the VGG11-like 3x3 conv layer (N=2^16, L=8, 64 input
ciphertexts, 128 outputs x 64 terms, 53% ternary in groups of 8).  The same
layer is also timed with every term as a PMult (all-PMult), which computes the
identical outputs, for the speedup of the hybrid route.  Layers whose
plaintext table exceeds the per-chunk budget run in output chunks (plaintexts
regenerated on the device between chunks, untimed) and the chunk times add up.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, vendor peak
PROFILE_DIR = os.path.join(ROOT, "profiles")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def strip_comments(src: str) -> str:
    """C++ source without its comments, whitespace runs collapsed (string and
    character literals kept as they are)."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash() -> str:
    """Hash of the hybrid kernel's code (comments excluded), which the committed
    counter records name: a change of code makes them stale, a change of
    comments does not."""
    h = hashlib.sha256()
    for name in ("fiona.hip", "hybrid_kernel.hpp", "modarith.hpp"):
        with open(os.path.join(ROOT, "paper_2609_35352_amd", "csrc", name), encoding="utf-8") as f:
            h.update(strip_comments(f.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, variant: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel source; else None."""
    path = os.path.join(PROFILE_DIR, "hbm_traffic_%s.json" % workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_src_sha") != kernel_source_hash():
        return None
    v = rec.get(variant)
    return None if v is None else float(v["bytes_per_launch"])


def time_layer(layer, dev, steps, warmup, stream, label, flags=0, padded=True):
    """Run every output chunk of `layer` with plans made under `flags`; return
    (sum of per-chunk ms per launch, algorithmic bytes, per-chunk records).
    time_layer.kernels names the kernel instances and time_layer.counts sums
    the plans' operation counts over the chunks."""
    import torch
    import synth
    import synth.gpu
    import paper_2609_35352_amd as fiona

    cfg = layer.cfg
    n_chunks = cfg.chunks_hybrid if layer.pt_const is None else cfg.chunks_allpm
    chunks = synth.output_chunks(layer.n_out, n_chunks)
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    in_t = torch.empty(layer.n_in * 2 * layer.L * layer.N, dtype=torch.int64, device=dev)
    synth.gpu.fill_inputs(layer, in_t)
    subs = [synth.chunk_layer(layer, a, b) for a, b in chunks]
    # plaintext rows at the library's padded pitch (or packed, pitch L*N)
    if padded is True:
        pitch = ctx.pt_pitch_hint()
    elif padded is False:
        pitch = layer.L * layer.N
    else:   # an explicit pad in words
        pitch = layer.L * layer.N + int(padded)
    max_pt = max(max(1, s.n_pt) for s in subs)
    max_out = max(s.n_out for s in subs)
    pt_t = torch.empty((max_pt - 1) * pitch + layer.L * layer.N, dtype=torch.int64, device=dev)
    out_t = torch.empty(max_out * 2 * layer.L * layer.N, dtype=torch.int64, device=dev)
    total_ms = 0.0
    total_bytes = 0
    per_chunk = []
    waves = set()
    counts = {}
    for ci, sub in enumerate(subs):
        synth.gpu.fill_pts(sub, pt_t, pitch)
        plan = fiona.Plan.from_layer(ctx, sub, flags=flags, pt_pitch=pitch)
        sign_t = torch.from_numpy(np.ascontiguousarray(sub.mem_sign)).to(dev) if sub.mem_sign.size else \
            torch.zeros(1, dtype=torch.int8, device=dev)
        scale_t = torch.from_numpy(np.ascontiguousarray(sub.scales.view(np.int64))).to(dev) if sub.scales.size \
            else torch.zeros(1, dtype=torch.int64, device=dev)
        torch.cuda.synchronize()
        for _ in range(warmup):
            fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, out_t, stream=stream)
        torch.cuda.synchronize()
        # one event between consecutive launches: the mean over the steps and
        # each launch's own time (min, median, max) from the same region
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        ev[0].record(stream)
        for i in range(steps):
            fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, out_t, stream=stream)
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[steps]) / steps
        each = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
        nbytes = synth.algorithmic_bytes(sub)
        total_ms += ms
        total_bytes += nbytes
        per_chunk.append({"outputs": sub.n_out, "ms": round(ms, 4), "alg_GBps": round(nbytes / ms / 1e6, 1),
                          "ms_min": round(each[0], 4), "ms_median": round(float(np.median(each)), 4),
                          "ms_max": round(each[-1], 4)})
        st = plan.stats()
        waves.add(st["waves"])
        for key in ("pmult_grouped", "n_use", "addsub_partial", "n_partial", "n_sum_distinct"):
            counts[key] = counts.get(key, 0) + st[key]
        if ci == 0 or ci == len(subs) - 1 or ci % 8 == 0:
            log("[bench] %s chunk %d/%d: %.3f ms/launch, %.1f GB/s algorithmic, plan %s"
                % (label, ci + 1, len(subs), ms, nbytes / ms / 1e6, plan.stats()))
        del plan
    del pt_t, out_t, in_t
    torch.cuda.empty_cache()
    time_layer.kernels = ["hybrid_linear_kernel<%d>" % w for w in sorted(waves)]
    time_layer.pitch = pitch
    time_layer.counts = counts
    return total_ms, total_bytes, per_chunk


def time_plan_variants(layer, dev, steps, warmup, stream, variants, padded=True, rounds=3):
    """Time plans compiled under different flags on the SAME device buffers (one
    allocation per buffer, every chunk's plaintexts filled once), interleaving
    the variants over `rounds` rounds and keeping each one's best round: the
    physical placement of a fresh allocation moves a layer's time by several
    percent, which would otherwise swamp the differences between plans.
    variants: [(name, flags)]; returns {name: (sum of per-chunk ms, summed plan counts)}."""
    import torch
    import synth
    import synth.gpu
    import paper_2609_35352_amd as fiona

    cfg = layer.cfg
    chunks = synth.output_chunks(layer.n_out, cfg.chunks_hybrid if layer.pt_const is None else cfg.chunks_allpm)
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    pitch = ctx.pt_pitch_hint() if padded is True else (layer.L * layer.N if padded is False
                                                        else layer.L * layer.N + int(padded))
    subs = [synth.chunk_layer(layer, a, b) for a, b in chunks]
    in_t = torch.empty(layer.n_in * 2 * layer.L * layer.N, dtype=torch.int64, device=dev)
    synth.gpu.fill_inputs(layer, in_t)
    max_pt = max(max(1, s.n_pt) for s in subs)
    pt_t = torch.empty((max_pt - 1) * pitch + layer.L * layer.N, dtype=torch.int64, device=dev)
    out_t = torch.empty(max(s.n_out for s in subs) * 2 * layer.L * layer.N, dtype=torch.int64, device=dev)
    res = {name: [0.0, {}] for name, _ in variants}
    for ci, sub in enumerate(subs):
        synth.gpu.fill_pts(sub, pt_t, pitch)
        sign_t = torch.from_numpy(np.ascontiguousarray(sub.mem_sign)).to(dev) if sub.mem_sign.size else \
            torch.zeros(1, dtype=torch.int8, device=dev)
        scale_t = torch.from_numpy(np.ascontiguousarray(sub.scales.view(np.int64))).to(dev) if sub.scales.size \
            else torch.zeros(1, dtype=torch.int64, device=dev)
        plans = {name: fiona.Plan.from_layer(ctx, sub, flags=flags, pt_pitch=pitch) for name, flags in variants}
        best = {name: float("inf") for name, _ in variants}
        torch.cuda.synchronize()
        for rd in range(rounds):
            for name, _ in variants:
                for _ in range(warmup if rd == 0 else 1):
                    fiona.hybrid_linear(plans[name], in_t, pt_t, sign_t, scale_t, out_t, stream=stream)
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for _ in range(steps):
                    fiona.hybrid_linear(plans[name], in_t, pt_t, sign_t, scale_t, out_t, stream=stream)
                e1.record(stream)
                torch.cuda.synchronize()
                best[name] = min(best[name], e0.elapsed_time(e1) / steps)
        for name, _ in variants:
            res[name][0] += best[name]
            st = plans[name].stats()
            for key in ("pmult_grouped", "n_use", "addsub_partial", "n_partial", "n_sum_distinct"):
                res[name][1][key] = res[name][1].get(key, 0) + st[key]
        log("[bench] plan variants, chunk %d/%d: %s" % (ci + 1, len(subs),
                                                        ", ".join("%s %.3f ms" % (n, best[n]) for n, _ in variants)))
        del plans
    del pt_t, out_t, in_t
    torch.cuda.empty_cache()
    return {name: (ms, counts) for name, (ms, counts) in res.items()}


def time_rotate(layer, dev, steps, warmup, stream):
    """Time fiona_hoisted_rotate: the layer's n_in - 1 baby-step rotations
    (by 1 .. n_in - 1 slots) of one ciphertext, one call, device-generated
    ciphertext and keys (uniform residues, already in the library's layout)."""
    import torch
    import synth
    import synth.gpu
    import paper_2609_35352_amd as fiona

    N, L = layer.N, layer.L
    primes = synth.ntt_primes(N, L + 1)
    if [int(q) for q in layer.moduli] != primes[:L]:
        raise ValueError("the layer's moduli are not the first L primes of the modulus rule")
    P = primes[L]
    steps_r = list(range(1, layer.n_in))
    galois = [pow(5, r, 2 * N) for r in steps_r]
    n = len(galois)
    ctx = fiona.Ctx(N, L, layer.moduli)
    rot = fiona.Rotator(ctx, P, n)
    kw = rot.key_words()
    ct_t = torch.empty(2 * L * N, dtype=torch.int64, device=dev)
    synth.gpu.fill_cts(layer, ct_t, 1)
    keys_t = torch.empty(n * kw, dtype=torch.int64, device=dev)
    synth.gpu.fill_rows(keys_t, n * kw // N, list(layer.moduli) + [P], N, layer.seed, synth.TAG_KEY)
    out_t = torch.empty(n * 2 * L * N, dtype=torch.int64, device=dev)
    torch.cuda.synchronize()
    for _ in range(warmup):
        fiona.hoisted_rotate(rot, ct_t, galois, keys_t, out_t, stream=stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        fiona.hoisted_rotate(rot, ct_t, galois, keys_t, out_t, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    nbytes = 8 * (2 * L * N + n * kw + n * 2 * L * N)
    log("[bench] %d hoisted rotations (N=%d, L=%d): %.3f ms, %.1f GB/s algorithmic"
        % (n, N, L, ms, nbytes / ms / 1e6))
    del keys_t, out_t, ct_t, rot
    torch.cuda.empty_cache()
    return {"rotations": n, "special_prime": P, "ms": round(ms, 4), "rotations_per_s": round(n / (ms * 1e-3), 1),
            "alg_bytes": nbytes, "alg_GBps": round(nbytes / ms / 1e6, 1),
            "frac_of_hbm_peak": round(nbytes / ms / 1e6 / HBM_PEAK_GBS, 4)}


def time_rescale(layer, dev, steps, warmup, stream):
    """Time fiona_rescale on n_out ciphertexts of the layer's shape (device-generated
    residues), all outputs in one call."""
    import torch
    import synth.gpu
    import paper_2609_35352_amd as fiona

    N, L, n = layer.N, layer.L, layer.n_out
    ctx = fiona.Ctx(N, L, layer.moduli)
    r = fiona.Rescaler(ctx, n)
    in_t = torch.empty(n * 2 * L * N, dtype=torch.int64, device=dev)
    synth.gpu.fill_cts(layer, in_t, n)
    out_t = torch.empty(n * 2 * (L - 1) * N, dtype=torch.int64, device=dev)
    torch.cuda.synchronize()
    for _ in range(warmup):
        fiona.rescale(r, in_t, n, out_t, stream=stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        fiona.rescale(r, in_t, n, out_t, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    nbytes = 8 * n * 2 * N * (L + (L - 1))
    logn = N.bit_length() - 1
    butterflies = n * 2 * L * (N // 2) * logn
    log("[bench] rescale of %d ciphertexts: %.3f ms, %.1f GB/s algorithmic" % (n, ms, nbytes / ms / 1e6))
    return {"ciphertexts": n, "ms": round(ms, 4), "ct_per_s": round(n / (ms * 1e-3), 1),
            "alg_bytes": nbytes, "alg_GBps": round(nbytes / ms / 1e6, 1),
            "frac_of_hbm_peak": round(nbytes / ms / 1e6 / HBM_PEAK_GBS, 4),
            "butterflies_per_s": round(butterflies / (ms * 1e-3), 1),
            "launches": 2 * L}


def cpu_baseline(layer, seconds: float = 10.0):
    """The oracle (test infrastructure, plain C) on a bounded sample of the same layer."""
    import oracle
    import synth

    threads = min(os.cpu_count() or 1, 16)
    S = 2048
    limbs, coeffs = synth.sample_positions(layer.N, layer.L, S, 7)
    x_s = synth.input_values(layer, (limbs, coeffs))
    pt_s = synth.pt_values(layer, (limbs, coeffs))
    n_pos = len(limbs)
    passes, t = 0, 0.0
    while t < seconds and passes < 1000:
        t0 = time.perf_counter()
        oracle.weighted_sum_sampled(layer, limbs, coeffs, x_s, pt_s, n_threads=threads)
        t += time.perf_counter() - t0
        passes += 1
    frac = n_pos / float(layer.L * layer.N)
    value = layer.ct_terms * frac * passes / t
    return {"value": value, "unit": "ct-terms/s", "cores": threads, "kind": "oracle",
            "sample": "%d (limb, coeff) positions of the layer x all %d outputs x %d terms x 2 polys, %d passes "
                      "in %.1f s (inputs generated before timing)" % (n_pos, layer.n_out, layer.cfg.T, passes, t)}


def time_mac_microbench(stream, blocks=2048, chunks=200, reps=5):
    """The register-only rate of the raw route's arithmetic (plaintext words
    per second, each multiplied into both polynomials), on the stream the
    kernels run on."""
    import torch
    import paper_2609_35352_amd as fiona

    sink = torch.empty(blocks * 256, dtype=torch.int64, device="cuda:0")
    words = fiona.mac_microbench(blocks, chunks, sink, stream=stream)   # warm-up
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fiona.mac_microbench(blocks, chunks, sink, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return {"words_per_s": round(words / (ms * 1e-3), 1), "ms_per_launch": round(ms, 4), "words": words,
            "threads": blocks * 256}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="vgg11")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-allpmult", action="store_true", help="time only the hybrid layer")
    ap.add_argument("--only-allpmult", action="store_true", help="time only the all-PMult layer")
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--rotate", action="store_true",
                    help="also time the hoisted baby-step rotations that produce the layer's inputs "
                         "(fiona_hoisted_rotate)")
    ap.add_argument("--rescale", action="store_true",
                    help="also time the rescale epilogue on the layer's outputs (fiona_rescale)")
    ap.add_argument("--ablation", action="store_true",
                    help="also time the layer compiled per-contribution, grouped, grouped+shared (Sec. 6.2)")
    ap.add_argument("--packed-pts", action="store_true",
                    help="plaintext rows packed at pitch L*N instead of the library's padded pitch hint")
    ap.add_argument("--pt-pad", type=int, default=None,
                    help="plaintext pitch L*N + PT_PAD words (overrides the pitch hint)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="only copy 4 GiB device-to-device (torch copy kernel) to calibrate HBM counters")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build measures one GPU only; the hybrid weighted sum has no "
              "multi-GPU path here (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import paper_2609_35352_amd as fiona

    if args.calib_copy:
        n = 1 << 29   # 4 GiB of int64
        a = torch.ones(n, dtype=torch.int64, device="cuda:0")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"calib_copy_bytes_read": n * 8, "calib_copy_bytes_written": n * 8, "launches": 3}))
        return

    if not os.path.exists(fiona.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    fiona.lib()
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=dev)   # default priority
    cfg = synth.CONFIGS[args.config]
    layer = synth.make_layer(cfg, args.seed)
    pad_mode = False if args.packed_pts else (True if args.pt_pad is None else args.pt_pad)
    log("[bench] %s: %s" % (cfg.name, cfg.description))

    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    if args.only_allpmult:
        apl = synth.all_pmult_layer(layer)
        ap_ms, ap_bytes, ap_chunks = time_layer(apl, dev, args.steps, args.warmup, stream, "all-PMult",
                                                padded=pad_mode)
        print(json.dumps({"variant": "all-PMult", "workload": cfg.name, "ms_per_step": round(ap_ms, 4),
                          "value": round(layer.ct_terms / (ap_ms * 1e-3), 1), "unit": "ct-terms/s",
                          "alg_GBps": round(ap_bytes / ap_ms / 1e6, 1), "chunks": ap_chunks}), flush=True)
        return
    hy_ms, hy_bytes, hy_chunks = time_layer(layer, dev, args.steps, args.warmup, stream, "hybrid",
                                            padded=pad_mode)
    hy_kernels = time_layer.kernels
    hy_pitch = time_layer.pitch
    torch.cuda.synchronize()
    hy_value = layer.ct_terms / (hy_ms * 1e-3)
    hy_gbs = hy_bytes / hy_ms / 1e6

    allpm = None
    if not args.no_allpmult:
        apl = synth.all_pmult_layer(layer)
        ap_ms, ap_bytes, ap_chunks = time_layer(apl, dev, args.steps, args.warmup, stream, "all-PMult",
                                                padded=pad_mode)
        allpm = {"value": round(layer.ct_terms / (ap_ms * 1e-3), 1), "ms_per_step": round(ap_ms, 4),
                 "alg_GBps": round(ap_bytes / ap_ms / 1e6, 1), "alg_bytes": ap_bytes,
                 "frac_of_hbm_peak": round(ap_bytes / ap_ms / 1e6 / HBM_PEAK_GBS, 4),
                 "chunks": len(ap_chunks), "speedup_hybrid_vs_allpmult": round(ap_ms / hy_ms, 3)}
    ablation = None
    if args.ablation:
        # the compilations of Sec. 6.2 on the same kernel: every signed term's
        # factor applied on its own, then grouping, then sharing whole sums,
        # then sharing partly overlapping sums as well (the default plan)
        # (all four on the same buffers, interleaved: see time_plan_variants)
        ablation = []
        variants = (("per-contribution", fiona.FIONA_PLAN_PER_CONTRIBUTION),
                    ("+grouping", fiona.FIONA_PLAN_NO_SHARING),
                    ("+sharing", fiona.FIONA_PLAN_NO_PARTIAL_SHARING),
                    ("+partial sharing", 0))
        timed = time_plan_variants(layer, dev, args.steps, args.warmup, stream, variants, padded=pad_mode)
        for name, _ in variants:
            ms, c = timed[name]
            ablation.append({"plan": name, "ms_per_step": round(ms, 4),
                             "value": round(layer.ct_terms / (ms * 1e-3), 1),
                             "scalar_products": c["n_use"], "pmult": c["pmult_grouped"] - c["n_use"],
                             "addsub": c["addsub_partial"], "common_terms": c["n_partial"],
                             "speedup_vs_per_contribution": None})
        for rec in ablation:
            rec["speedup_vs_per_contribution"] = round(ablation[0]["ms_per_step"] / rec["ms_per_step"], 3)
    rescale = None
    if args.rescale:
        rescale = time_rescale(layer, dev, args.steps, args.warmup, stream)
    rotate = None
    if args.rotate:
        rotate = time_rotate(layer, dev, args.steps, args.warmup, stream)
    # the hybrid launch's raw-term multiply-adds against the register-only rate
    mb = time_mac_microbench(stream)
    hy_words = layer.n_pm * cfg.L * cfg.N / (hy_ms * 1e-3)
    mac_rate = {"raw_words_per_s_hybrid": round(hy_words, 1), "raw_words_per_s_register_only": mb["words_per_s"],
                "frac": round(hy_words / mb["words_per_s"], 4), "microbench": mb}
    wall = time.perf_counter() - t_wall0

    traffic = measured_traffic(cfg.name, "hybrid")
    n_launch = len(hy_chunks)
    result = {
        "metric": "ct-terms/sec and achieved HBM GB/s (hybrid vs all-PMult), N=2^16 layers, 1 GPU",
        "value": round(hy_value, 1),
        "unit": "ct-terms/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(hy_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic (seeded counter-based generator, uniform residues; no dataset or weights)",
        "config": {"workload": "%s: %s" % (cfg.name, cfg.description), "N": cfg.N, "L": cfg.L,
                   "n_in": cfg.n_in, "n_out": cfg.n_out, "terms_per_output": cfg.T, "group": cfg.g,
                   "ternary_groups": layer.n_group, "raw_terms": layer.n_pm, "ct_terms": layer.ct_terms,
                   "chunks": n_launch, "seed": args.seed,
                   "pt_pitch_words": hy_pitch, "pt_row_words": cfg.L * cfg.N},
        "achieved_alg_GBps": round(hy_gbs, 1),
        "launch_ms": {"min": round(sum(c["ms_min"] for c in hy_chunks), 4),
                      "median": round(sum(c["ms_median"] for c in hy_chunks), 4),
                      "max": round(sum(c["ms_max"] for c in hy_chunks), 4)},
        "roofline": {"bound": "hbm", "achieved": round(hy_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(hy_gbs / HBM_PEAK_GBS, 4),
                     "traffic": None if traffic is None else round(traffic),
                     "alg_bytes_per_launch": hy_bytes // n_launch,
                     "kernel": " + ".join(hy_kernels)},
        "all_pmult": allpm,
        "hybrid_chunks": hy_chunks if n_launch > 1 else None,
        "ablation": ablation,
        "rescale": rescale,
        "rotate": rotate,
        "mac_rate": mac_rate,
        "gpu_wall_s": round(wall, 2),
    }
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample (about 10 s)")
        result["cpu_baseline"] = cpu_baseline(layer)
        result["cpu_baseline"]["value"] = round(result["cpu_baseline"]["value"], 1)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
