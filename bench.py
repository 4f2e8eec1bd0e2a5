"""Benchmark of the hybrid weighted sum on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--rounds R] [--layers vgg11,vit768,bert_ffn,large4096]
                    [--no-cpu-baseline] [--ablation] [--rescale] [--rotate] [--pipeline] [--config NAME]

The metric is quoted on the four N=2^16 layers, so a default run times all
four, each both ways: the hybrid layer (PMult for raw terms, Add/Sub and one
scalar product per signed sum) and the same layer with every term a PMult
(all-PMult), which computes identical outputs.  The two forms of a layer run
on the same device buffers (one input, plaintext and output allocation per
layer), alternating over R rounds.  Layers whose plaintext table exceeds the
per-chunk budget run in output chunks: the chunk's plaintexts are generated
on the device (untimed), then W untimed and K timed launches follow, one HIP
event between consecutive launches on the kernels' stream.  A layer's step
time is the sum over its chunks of the median launch time (over the K launches
of every round); the mean, minimum and maximum are reported beside it.

The headline record is the largest layer, the 4096x4096 one (16 output chunks
of 8 outputs; each chunk's 77 GiB of plaintexts resident when its launches
run).  Every layer carries its own roofline (algorithmic bytes per launch over
the mean launch time, against 8 TB/s), counter traffic where the committed
counter records match the kernel source, and the hybrid-vs-all-PMult speedup.
Measured read and copy ceilings of the HBM sit beside the 8 TB/s spec.

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
LAYERS = ("vgg11", "vit768", "bert_ffn", "large4096")
METRIC = "ct-terms/sec and achieved HBM GB/s (hybrid vs all-PMult), N=2^16 layers, 1 GPU"


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
    for name in ("fiona.hip", "hybrid_kernel.hpp", "modarith.hpp", "buffer.hpp"):
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


def _dev_signs_scales(sub, dev):
    import torch
    sign_t = torch.from_numpy(np.ascontiguousarray(sub.mem_sign)).to(dev) if sub.mem_sign.size else \
        torch.zeros(1, dtype=torch.int8, device=dev)
    scale_t = torch.from_numpy(np.ascontiguousarray(sub.scales.view(np.int64))).to(dev) if sub.scales.size \
        else torch.zeros(1, dtype=torch.int64, device=dev)
    return sign_t, scale_t


def _pitch(ctx, layer, padded):
    if padded is True:
        return ctx.pt_pitch_hint()
    if padded is False:
        return layer.L * layer.N
    return layer.L * layer.N + int(padded)


def time_layer(name, dev, stream, steps, warmup, rounds, seed=1, padded=True):
    """Both forms of one layer on the same buffers; returns the layer record."""
    import torch
    import synth
    import synth.gpu
    import paper_2609_35352_amd as fiona

    cfg = synth.CONFIGS[name]
    layer = synth.make_layer(cfg, seed)
    forms = {"hybrid": (layer, cfg.chunks_hybrid), "all_pmult": (synth.all_pmult_layer(layer), cfg.chunks_allpm)}
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    pitch = _pitch(ctx, layer, padded)
    LN = layer.L * layer.N
    subs = {f: [synth.chunk_layer(lay, a, b) for a, b in synth.output_chunks(lay.n_out, nc)]
            for f, (lay, nc) in forms.items()}
    max_pt = max(max(1, s.n_pt) for ss in subs.values() for s in ss)
    max_out = max(s.n_out for ss in subs.values() for s in ss)
    in_t = torch.empty(layer.n_in * 2 * LN, dtype=torch.int64, device=dev)
    synth.gpu.fill_inputs(layer, in_t)
    pt_t = torch.empty((max_pt - 1) * pitch + LN, dtype=torch.int64, device=dev)
    out_t = torch.empty(max_out * 2 * LN, dtype=torch.int64, device=dev)
    plans = {f: [fiona.Plan.from_layer(ctx, s, pt_pitch=pitch) for s in ss] for f, ss in subs.items()}
    args = {f: [_dev_signs_scales(s, dev) for s in ss] for f, ss in subs.items()}
    times = {f: [[] for _ in ss] for f, ss in subs.items()}
    torch.cuda.synchronize()
    for rd in range(rounds):
        for f in forms:
            for ci, sub in enumerate(subs[f]):
                synth.gpu.fill_pts(sub, pt_t, pitch)   # untimed; synchronizes
                plan, (sign_t, scale_t) = plans[f][ci], args[f][ci]
                for _ in range(warmup):
                    fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, out_t, stream=stream)
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
                ev[0].record(stream)
                for i in range(steps):
                    fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, out_t, stream=stream)
                    ev[i + 1].record(stream)
                torch.cuda.synchronize()
                times[f][ci] += [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
            n = len(subs[f])
            log("[bench] %s %s round %d/%d: %d chunk(s), %.3f ms (sum of this round's chunk medians)"
                % (name, f, rd + 1, rounds, n, sum(float(np.median(t[-steps:])) for t in times[f])))
    rec = {"layer": name, "description": cfg.description, "N": cfg.N, "L": cfg.L, "n_in": cfg.n_in,
           "n_out": cfg.n_out, "terms_per_output": cfg.T, "group": cfg.g, "ct_terms": layer.ct_terms,
           "pt_pitch_words": pitch, "pt_row_words": LN}
    for f in forms:
        t = times[f]
        med = sum(float(np.median(x)) for x in t)
        mean = sum(float(np.mean(x)) for x in t)
        nbytes = sum(synth.algorithmic_bytes(s) for s in subs[f])
        n = len(t)
        st = [p.stats() for p in plans[f]]
        waves = sorted({s["waves"] for s in st})
        traffic = measured_traffic(name, "hybrid" if f == "hybrid" else "allpm")
        rec[f] = {
            "ms_per_step": round(med, 4), "ms_mean": round(mean, 4),
            "ms_min": round(sum(min(x) for x in t), 4), "ms_max": round(sum(max(x) for x in t), 4),
            "value": round(layer.ct_terms / (med * 1e-3), 1), "unit": "ct-terms/s",
            "chunks": n, "timed_launches_per_chunk": len(t[0]),
            "alg_bytes": nbytes, "alg_GBps": round(nbytes / med / 1e6, 1),
            "roofline": {"bound": "hbm", "achieved": round(nbytes / mean / 1e6, 1), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(nbytes / mean / 1e6 / HBM_PEAK_GBS, 4),
                         "traffic": None if traffic is None else round(traffic),
                         "alg_bytes_per_launch": nbytes // n,
                         "kernel": " + ".join("hybrid_linear_kernel<%d>" % w for w in waves)},
            "plan": {k: sum(s[k] for s in st) for k in ("n_pmult", "n_use", "n_sum_distinct", "addsub_partial",
                                                         "n_partial")},
        }
        if n > 1:
            rec[f]["chunk_ms_median"] = [round(float(np.median(x)), 4) for x in t]
    rec["speedup_hybrid_vs_allpmult"] = round(rec["all_pmult"]["ms_per_step"] / rec["hybrid"]["ms_per_step"], 3)
    rec["raw_words_per_s_hybrid"] = layer.n_pm * LN / (rec["hybrid"]["ms_per_step"] * 1e-3)
    del plans, args, pt_t, out_t, in_t
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


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
    pitch = _pitch(ctx, layer, padded)
    subs = [synth.chunk_layer(layer, a, b) for a, b in chunks]
    in_t = torch.empty(layer.n_in * 2 * layer.L * layer.N, dtype=torch.int64, device=dev)
    synth.gpu.fill_inputs(layer, in_t)
    max_pt = max(max(1, s.n_pt) for s in subs)
    pt_t = torch.empty((max_pt - 1) * pitch + layer.L * layer.N, dtype=torch.int64, device=dev)
    out_t = torch.empty(max(s.n_out for s in subs) * 2 * layer.L * layer.N, dtype=torch.int64, device=dev)
    res = {name: [0.0, {}] for name, _ in variants}
    for ci, sub in enumerate(subs):
        synth.gpu.fill_pts(sub, pt_t, pitch)
        sign_t, scale_t = _dev_signs_scales(sub, dev)
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
            "butterflies_per_s": round(butterflies / (ms * 1e-3), 1)}


def time_pipeline(layer, dev, steps, warmup, stream):
    """One whole layer step on one stream: the n_in - 1 baby-step rotations of
    one ciphertext, written straight into the weighted sum's input array (baby
    step 0 is the ciphertext itself), the hybrid weighted sum, and the rescale
    of its outputs.  Timed eagerly (HIP events between the three stages; per
    stage and per step the median of the timed steps) and as one HIP graph of
    the three stages replayed (the median replay).  Device-generated inputs:
    ciphertext, keys (uniform residues in the library's layout), plaintexts.
    Layers whose plaintexts fit one launch (one hybrid chunk)."""
    import torch
    import synth
    import synth.gpu
    import paper_2609_35352_amd as fiona

    if layer.cfg.chunks_hybrid != 1:
        raise ValueError("the pipeline times layers whose weighted sum is one launch")
    N, L, LN = layer.N, layer.L, layer.L * layer.N
    P = synth.ntt_primes(N, L + 1)[L]
    galois = [pow(5, r, 2 * N) for r in range(1, layer.n_in)]
    n = len(galois)
    ctx = fiona.Ctx(N, L, layer.moduli)
    rot = fiona.Rotator(ctx, P, max(n, 1))
    kw = rot.key_words()
    in_t = torch.empty(layer.n_in * 2 * LN, dtype=torch.int64, device=dev)
    ct_t, rot_t = in_t[: 2 * LN], in_t[2 * LN:]
    synth.gpu.fill_cts(layer, ct_t, 1)
    keys_t = torch.empty(max(n, 1) * kw, dtype=torch.int64, device=dev)
    synth.gpu.fill_rows(keys_t, max(n, 1) * kw // N, list(layer.moduli) + [P], N, layer.seed, synth.TAG_KEY)
    pitch = ctx.pt_pitch_hint()
    plan = fiona.Plan.from_layer(ctx, layer, pt_pitch=pitch)
    pt_t = torch.empty((max(1, layer.n_pt) - 1) * pitch + LN, dtype=torch.int64, device=dev)
    synth.gpu.fill_pts(layer, pt_t, pitch)
    sign_t, scale_t = _dev_signs_scales(layer, dev)
    out_t = torch.empty(layer.n_out * 2 * LN, dtype=torch.int64, device=dev)
    resc = fiona.Rescaler(ctx, layer.n_out)
    res_t = torch.empty(layer.n_out * 2 * (L - 1) * N, dtype=torch.int64, device=dev)

    def step(ev=None):
        if ev:
            ev[0].record(stream)
        if n:
            fiona.hoisted_rotate(rot, ct_t, galois, keys_t, rot_t, stream=stream)
        if ev:
            ev[1].record(stream)
        fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, out_t, stream=stream)
        if ev:
            ev[2].record(stream)
        fiona.rescale(resc, out_t, layer.n_out, res_t, stream=stream)
        if ev:
            ev[3].record(stream)

    torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for ev in evs:
        step(ev)
    torch.cuda.synchronize()
    med = lambda a, b: float(np.median([ev[a].elapsed_time(ev[b]) for ev in evs]))
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        step()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    ge = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ge[0].record(stream)
    with torch.cuda.stream(stream):
        for i in range(steps):
            graph.replay()
            ge[i + 1].record(stream)
    torch.cuda.synchronize()
    g_ms = float(np.median([ge[i].elapsed_time(ge[i + 1]) for i in range(steps)]))
    rec = {"rotations": n, "rotate_ms": round(med(0, 1), 4), "weighted_sum_ms": round(med(1, 2), 4),
           "rescale_ms": round(med(2, 3), 4), "step_ms": round(med(0, 3), 4), "graph_step_ms": round(g_ms, 4),
           "weighted_sum_share": round(med(1, 2) / med(0, 3), 4)}
    log("[bench] layer step (%d rotations, weighted sum, rescale of %d outputs): %.3f ms eager "
        "(%.3f + %.3f + %.3f), %.3f ms as one HIP graph"
        % (n, layer.n_out, rec["step_ms"], rec["rotate_ms"], rec["weighted_sum_ms"], rec["rescale_ms"], g_ms))
    del graph
    return rec


def host_cpu():
    """CPU model, the host's CPU count and the threads this process may use
    (its affinity, capped by OMP_NUM_THREADS where set: a shared multi-GPU
    host gives each GPU's job a share of its cores)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    cap = os.environ.get("OMP_NUM_THREADS")
    threads = min(avail, int(cap)) if cap and cap.isdigit() and int(cap) > 0 else avail
    return model, os.cpu_count() or 1, avail, threads


def cpu_baseline(layer, seconds: float = 10.0, n_pos: int = None):
    """The oracle (test infrastructure, plain C) on a bounded sample of the same
    layer: n_pos (limb, coefficient) positions x every output and term, both
    polynomials, chunk by chunk for a chunked layer, repeated for about
    `seconds`; scaled to the whole layer.  By default n_pos keeps the sampled
    plaintext values (generated in NumPy before timing) near 10^7."""
    import oracle
    import synth

    model, ncpu, avail, threads = host_cpu()
    if n_pos is None:
        n_pos = int(min(2048, max(16, 10_000_000 // max(1, layer.n_pt))))
    limbs, coeffs = synth.sample_positions(layer.N, layer.L, max(0, n_pos - 6), 7)
    x_s = synth.input_values(layer, (limbs, coeffs))
    chunks = [synth.chunk_layer(layer, a, b) for a, b in synth.output_chunks(layer.n_out, layer.cfg.chunks_hybrid)]
    pts = [synth.pt_values(c, (limbs, coeffs)) for c in chunks]
    passes, t = 0, 0.0
    while t < seconds and passes < 1000:
        t0 = time.perf_counter()
        for c, pt_s in zip(chunks, pts):
            oracle.weighted_sum_sampled(c, limbs, coeffs, x_s, pt_s, n_threads=threads)
        t += time.perf_counter() - t0
        passes += 1
    frac = len(limbs) / float(layer.L * layer.N)
    value = layer.ct_terms * frac * passes / t
    return {"value": value, "unit": "ct-terms/s", "cores": threads, "kind": "oracle",
            "cpu_model": model, "host_cpus": ncpu, "cpus_available": avail,
            "sample": "%d (limb, coeff) positions of %s x all %d outputs x %d terms x 2 polys, %d passes in %.1f s "
                      "(per-term __int128 products and %%, inputs generated before timing); scaled by the positions' "
                      "share of the layer" % (len(limbs), layer.cfg.name, layer.n_out, layer.cfg.T, passes, t)}


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


def time_streams(stream, gib=4, reps=5):
    """Measured HBM ceilings: a plain contiguous read, a plain copy and a plain
    write of `gib` GiB (best grid of four), next to the 8 TB/s spec."""
    import torch
    import paper_2609_35352_amd as fiona

    n = (gib << 30) // 8
    src = torch.ones(n, dtype=torch.int64, device="cuda:0")
    dst = torch.empty_like(src)
    sink = torch.empty(1 << 15, dtype=torch.int64, device="cuda:0")
    out = {}
    for kind in ("read", "copy", "write"):
        best = None
        for blocks in (2048, 4096, 8192, 16384):
            run = {"read": lambda: fiona.stream_read(src, blocks, sink, stream=stream),
                   "copy": lambda: fiona.stream_copy(src, dst, blocks, stream=stream),
                   "write": lambda: fiona.stream_write(dst, blocks, stream=stream)}[kind]
            nbytes = run()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                run()
            e1.record(stream)
            torch.cuda.synchronize()
            gbs = nbytes / (e0.elapsed_time(e1) / reps) / 1e6
            if best is None or gbs > best[0]:
                best = (gbs, blocks)
        out[kind] = {"GBps": round(best[0], 1), "frac_of_spec": round(best[0] / HBM_PEAK_GBS, 4),
                     "workgroups": best[1], "bytes": n * 8 * (2 if kind == "copy" else 1)}
    del src, dst, sink
    torch.cuda.empty_cache()
    out["spec_GBps"] = HBM_PEAK_GBS
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--rounds", type=int, default=2, help="rounds of hybrid then all-PMult per layer")
    ap.add_argument("--layers", default=",".join(LAYERS),
                    help="comma-separated layers to time ('none': only the --ablation/--rescale/--rotate steps)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-streams", action="store_true", help="skip the read, copy and write ceilings")
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--config", default="vgg11", help="the layer of --ablation, --rescale and --rotate")
    ap.add_argument("--rotate", action="store_true",
                    help="also time the hoisted baby-step rotations that produce the layer's inputs "
                         "(fiona_hoisted_rotate)")
    ap.add_argument("--rescale", action="store_true",
                    help="also time the rescale epilogue on the layer's outputs (fiona_rescale)")
    ap.add_argument("--pipeline", action="store_true",
                    help="also time one whole layer step of --config: its rotations, weighted sum and rescale "
                         "on one stream, eagerly and as one HIP graph")
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
        print("bench.py: measures one GPU only; the hybrid weighted sum has no "
              "multi-GPU path (run with --gpus 1)", file=sys.stderr)
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
    pad_mode = False if args.packed_pts else (True if args.pt_pad is None else args.pt_pad)
    names = [n for n in args.layers.split(",") if n and n != "none"]
    for n in names:
        if n not in synth.CONFIGS:
            raise SystemExit("unknown layer %s" % n)
    if not names and not (args.ablation or args.rescale or args.rotate or args.pipeline):
        raise SystemExit("nothing to time: --layers none needs --ablation, --rescale, --rotate or --pipeline")

    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    records = []
    for n in names:
        log("[bench] %s: %s" % (n, synth.CONFIGS[n].description))
        records.append(time_layer(n, dev, stream, args.steps, args.warmup, args.rounds, args.seed, pad_mode))
    head = next((r for r in records if r["layer"] == "large4096"), records[-1] if records else None)

    extra = {}
    if args.ablation or args.rescale or args.rotate or args.pipeline:
        layer = synth.make_layer(synth.CONFIGS[args.config], args.seed)
        if args.ablation:
            # the compilations of Sec. 6.2 on the same kernel: every signed term's
            # factor applied on its own, then grouping, then sharing whole sums,
            # then sharing partly overlapping sums as well (the default plan)
            # (all four on the same buffers, interleaved: see time_plan_variants)
            variants = (("per-contribution", fiona.FIONA_PLAN_PER_CONTRIBUTION),
                        ("+grouping", fiona.FIONA_PLAN_NO_SHARING),
                        ("+sharing", fiona.FIONA_PLAN_NO_PARTIAL_SHARING),
                        ("+partial sharing", 0))
            timed = time_plan_variants(layer, dev, args.steps, args.warmup, stream, variants, padded=pad_mode)
            abl = []
            for name, _ in variants:
                ms, c = timed[name]
                abl.append({"plan": name, "ms_per_step": round(ms, 4), "value": round(layer.ct_terms / (ms * 1e-3), 1),
                            "scalar_products": c["n_use"], "pmult": c["pmult_grouped"] - c["n_use"],
                            "addsub": c["addsub_partial"], "common_terms": c["n_partial"]})
            for rec in abl:
                rec["speedup_vs_per_contribution"] = round(abl[0]["ms_per_step"] / rec["ms_per_step"], 3)
            extra["ablation"] = {"layer": args.config, "plans": abl}
        if args.rescale:
            extra["rescale"] = dict(time_rescale(layer, dev, args.steps, args.warmup, stream), layer=args.config)
        if args.rotate:
            extra["rotate"] = dict(time_rotate(layer, dev, args.steps, args.warmup, stream), layer=args.config)
        if args.pipeline:
            extra["pipeline"] = dict(time_pipeline(layer, dev, args.steps, args.warmup, stream), layer=args.config)
    # each layer's raw-term multiply-adds against the register-only rate
    mb = time_mac_microbench(stream)
    for r in records:
        w = r.pop("raw_words_per_s_hybrid")
        r["mac_rate_frac"] = round(w / mb["words_per_s"], 4)
    streams = None if args.no_streams else time_streams(stream)
    wall = time.perf_counter() - t_wall0
    if head is None:   # --layers none: the extra steps only
        print(json.dumps(dict(extra, mac_microbench=mb, streams=streams, gpu_wall_s=round(wall, 2))), flush=True)
        return

    hy = head["hybrid"]
    result = {
        "metric": METRIC,
        "value": hy["value"],
        "unit": "ct-terms/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": hy["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic (seeded counter-based generator, uniform residues; no dataset or weights)",
        "config": {"workload": "%s: %s" % (head["layer"], head["description"]), "N": head["N"], "L": head["L"],
                   "n_in": head["n_in"], "n_out": head["n_out"], "terms_per_output": head["terms_per_output"],
                   "group": head["group"], "ct_terms": head["ct_terms"], "chunks": hy["chunks"],
                   "seed": args.seed, "rounds": args.rounds,
                   "step": "every output chunk once: sum over chunks of the median launch time"},
        "roofline": hy["roofline"],
        "speedup_hybrid_vs_allpmult": head["speedup_hybrid_vs_allpmult"],
        "layers": records,
        "streams": streams,
        "mac_microbench": mb,
        "gpu_wall_s": round(wall, 2),
    }
    result.update(extra)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample of %s (about 10 s)" % head["layer"])
        cb = cpu_baseline(synth.make_layer(synth.CONFIGS[head["layer"]], args.seed))
        cb["value"] = round(cb["value"], 1)
        result["cpu_baseline"] = cb
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
