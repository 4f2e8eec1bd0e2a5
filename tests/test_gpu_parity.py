"""GPU parity: the HIP path against the oracle, through the C ABI.

Small layers are compared element by element (every output, polynomial, limb
and coefficient); the full-size layers run in the same launch configuration
as the benchmark, on device-generated inputs, and are compared at sampled
positions that the oracle computes from the same generator.  Every comparison
is bit-exact.
"""
import os
import sys

import numpy as np
import pytest

import oracle
import random_layers
import synth
import paper_2609_35352_amd as fiona

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    # fail loudly if the native library is missing: there is no other path
    fiona.lib()
    import synth.gpu
    synth.gpu.lib()
    return torch.device("cuda:0")


def _to_dev(a, dtype, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(dtype)).to(dev)


POISON = -1   # all-ones words in the padding between plaintext rows: never a residue


def _run(layer, dev, x=None, pt=None, flags=0, scales=None, signs=None, pitch=0):
    """Run the layer on the GPU; x/pt from host arrays or, if None, filled on the device.
    pitch: words between plaintext rows (0 = packed L*N, "hint" = fiona_pt_pitch_hint);
    the padding between rows holds all-ones words."""
    import torch
    import synth.gpu
    N, L = layer.N, layer.L
    ctx = fiona.Ctx(N, L, layer.moduli)
    if pitch == "hint":
        pitch = ctx.pt_pitch_hint()
    plan = fiona.Plan.from_layer(ctx, layer, flags=flags, pt_pitch=pitch)
    if x is None:
        in_t = torch.empty(layer.n_in * 2 * L * N, dtype=torch.int64, device=dev)
        synth.gpu.fill_inputs(layer, in_t)
    else:
        in_t = _to_dev(x, np.int64, dev)
    P = plan.pt_pitch
    if pt is None:
        pt_t = torch.full((max(1, plan.pt_words()),), POISON, dtype=torch.int64, device=dev)
        synth.gpu.fill_pts(layer, pt_t, P)
    elif not pt.size:
        pt_t = torch.zeros(1, dtype=torch.int64, device=dev)
    else:
        padded = np.full((layer.n_pt, P), np.uint64(2**64 - 1), np.uint64)
        padded[:, : L * N] = np.ascontiguousarray(pt).reshape(layer.n_pt, L * N)
        pt_t = _to_dev(padded.reshape(-1)[: plan.pt_words()], np.int64, dev)
    sg = layer.mem_sign if signs is None else signs
    sign_t = _to_dev(sg, np.int8, dev) if sg.size else torch.zeros(1, dtype=torch.int8, device=dev)
    sc = layer.scales if scales is None else scales
    scale_t = _to_dev(sc, np.int64, dev) if sc.size else torch.zeros(1, dtype=torch.int64, device=dev)
    out_t = torch.full((max(1, layer.n_out * 2 * L * N),), -1, dtype=torch.int64, device=dev)
    fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, out_t)
    torch.cuda.synchronize()
    return out_t, in_t, pt_t, plan


def _host(out_t, layer):
    return out_t.cpu().numpy().view(np.uint64)[: layer.n_out * 2 * layer.L * layer.N].reshape(
        layer.n_out, 2, layer.L, layer.N)


def _assert_equal(got, expect, what):
    bad = np.argwhere(got != expect)
    if bad.size:
        first = tuple(int(v) for v in bad[0])
        raise AssertionError("%s: %d mismatches; first at (out, poly, limb, coeff) = %s: gpu %d, oracle %d"
                             % (what, len(bad), first, got[first], expect[first]))


SMALL = {
    "tiny": synth.CONFIGS["tiny"],
    "ragged_pool": synth.LayerConfig("ragged_pool", N=1000, L=3, n_in=24, n_out=7, T=48, g=8, ternary=0.5, pool=4),
    "many_outputs": synth.LayerConfig("many_outputs", N=197, L=2, n_in=16, n_out=37, T=16, g=4, ternary=0.4),
    "fold_raw": synth.LayerConfig("fold_raw", N=128, L=2, n_in=8, n_out=3, T=2600, g=8, ternary=0.3),
    "fold_uses": synth.LayerConfig("fold_uses", N=64, L=2, n_in=8, n_out=2, T=4400, g=1, ternary=0.6),
    "big_groups": synth.LayerConfig("big_groups", N=256, L=2, n_in=100, n_out=3, T=400, g=100, ternary=0.5),
    "lds_full": synth.LayerConfig("lds_full", N=128, L=1, n_in=159, n_out=4, T=318, g=53, ternary=0.5, pool=2),
    "all_ternary": synth.LayerConfig("all_ternary", N=320, L=2, n_in=12, n_out=5, T=24, g=6, ternary=1.0, pool=3),
    "all_raw": synth.LayerConfig("all_raw", N=320, L=2, n_in=12, n_out=5, T=24, g=6, ternary=0.0),
    "partial_share": synth.LayerConfig("partial_share", N=256, L=2, n_in=16, n_out=48, T=96, g=12, ternary=0.95),
    # groups wider than the inputs: a group names an input more than once
    "repeated_pool": synth.LayerConfig("repeated_pool", N=256, L=2, n_in=6, n_out=48, T=80, g=10, ternary=0.9,
                                       pool=4),
    "repeated_iid": synth.LayerConfig("repeated_iid", N=256, L=2, n_in=7, n_out=48, T=160, g=20, ternary=0.9),
    # more inputs than one tile's LDS holds: passes over input ranges, groups crossing them
    "wide_320": synth.LayerConfig("wide_320", N=256, L=2, n_in=320, n_out=6, T=640, g=16, ternary=0.6, pool=3),
    "wide_160_bursts": synth.LayerConfig("wide_160_bursts", N=128, L=2, n_in=160, n_out=40, T=320, g=16,
                                         ternary=0.5),
    "wide_partial": synth.LayerConfig("wide_partial", N=128, L=2, n_in=200, n_out=48, T=400, g=40, ternary=0.95),
    "wide_repeat": synth.LayerConfig("wide_repeat", N=96, L=2, n_in=170, n_out=8, T=800, g=200, ternary=0.5),
    # ragged N; 320 inputs, terms on the first 64 only: the other input ranges get no pass
    "wide_sparse": synth.LayerConfig("wide_sparse", N=100, L=2, n_in=320, n_out=5, T=64, g=8, ternary=0.5),
}


def _merge_layers(a, b):
    """The outputs of a followed by those of b (same ring, moduli, seed and inputs)."""
    assert (a.N, a.L, a.n_in, a.seed, list(a.moduli)) == (b.N, b.L, b.n_in, b.seed, list(b.moduli))
    cat = np.concatenate
    return synth.Layer(
        cfg=a.cfg, moduli=a.moduli, seed=a.seed, n_in=a.n_in, n_out=a.n_out + b.n_out,
        out_global=cat([a.out_global, b.out_global + a.n_out]).astype(np.uint32),
        pm_off=cat([a.pm_off, b.pm_off[1:] + a.pm_off[-1]]).astype(np.uint32),
        pm_input=cat([a.pm_input, b.pm_input]).astype(np.uint32),
        pm_pt=cat([a.pm_pt, b.pm_pt + a.n_pt]).astype(np.uint32),
        grp_off=cat([a.grp_off, b.grp_off[1:] + a.grp_off[-1]]).astype(np.uint32),
        grp_mem_off=cat([a.grp_mem_off, b.grp_mem_off[1:] + a.grp_mem_off[-1]]).astype(np.uint32),
        mem_input=cat([a.mem_input, b.mem_input]).astype(np.uint32),
        mem_sign=cat([a.mem_sign, b.mem_sign]).astype(np.int8),
        grp_scale=cat([a.grp_scale, b.grp_scale + len(a.scales)]).astype(np.uint32),
        scales=cat([a.scales, b.scales]).astype(np.uint64),
        pt_global=cat([a.pt_global, b.pt_global]).astype(np.uint64))


def _small_layer(name):
    cfg = SMALL[name]
    if name == "tiny":
        return synth.make_layer(cfg, 1)
    Nq = 1 << max(6, (cfg.N - 1).bit_length())
    return synth.make_layer(cfg, 5, moduli=synth.ntt_primes(Nq, cfg.L))


@pytest.mark.parametrize("name", list(SMALL))
def test_small_layer_elementwise(dev, name):
    layer = _small_layer(name)
    _say("[parity] %s: N=%d L=%d n_in=%d n_out=%d terms/out=%d" % (name, layer.N, layer.L, layer.n_in,
                                                                   layer.n_out, layer.cfg.T))
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    out_t, *_ = _run(layer, dev, x, pt)
    _assert_equal(_host(out_t, layer), expect, name)


@pytest.mark.parametrize("name,flags", [("ragged_pool", fiona.FIONA_PLAN_NO_SHARING),
                                        ("ragged_pool", fiona.FIONA_PLAN_NO_LDS_SUMS),
                                        ("ragged_pool", fiona.FIONA_PLAN_NO_SHARING | fiona.FIONA_PLAN_NO_LDS_SUMS),
                                        ("partial_share", fiona.FIONA_PLAN_NO_PARTIAL_SHARING),
                                        ("partial_share", fiona.FIONA_PLAN_NO_LDS_SUMS),
                                        ("ragged_pool", fiona.FIONA_PLAN_PER_CONTRIBUTION),
                                        ("partial_share", fiona.FIONA_PLAN_PER_CONTRIBUTION),
                                        ("many_outputs", fiona.FIONA_PLAN_NO_OUTPUT_BURSTS),
                                        ("partial_share", fiona.FIONA_PLAN_NO_OUTPUT_BURSTS),
                                        ("fold_raw", fiona.FIONA_PLAN_NO_OUTPUT_BURSTS),
                                        ("repeated_pool", fiona.FIONA_PLAN_NO_LDS_SUMS),
                                        ("repeated_pool", fiona.FIONA_PLAN_NO_PARTIAL_SHARING),
                                        ("wide_partial", fiona.FIONA_PLAN_NO_LDS_SUMS),
                                        ("wide_160_bursts", fiona.FIONA_PLAN_NO_OUTPUT_BURSTS),
                                        ("wide_320", fiona.FIONA_PLAN_PER_CONTRIBUTION)])
def test_plan_variants_agree(dev, name, flags):
    layer = _small_layer(name)
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    out_t, *_ = _run(layer, dev, x, pt, flags=flags)
    _assert_equal(_host(out_t, layer), expect, "flags=%d" % flags)


@pytest.mark.parametrize("name", ["tiny", "ragged_pool", "fold_raw", "partial_share"])
def test_padded_plaintext_pitch(dev, name):
    """Plaintext rows at the library's padded pitch and at an odd pitch (L*N + 1),
    all-ones words in between: the same exact result, so no padding word is read."""
    layer = _small_layer(name)
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    for pitch in ("hint", layer.L * layer.N + 1):
        out_t, *_ = _run(layer, dev, x, pt, pitch=pitch)
        _assert_equal(_host(out_t, layer), expect, "%s pitch %s" % (name, pitch))


@pytest.mark.parametrize("long_first", [True, False])
def test_output_rounds_with_split_outputs(dev, long_first):
    """Three rounds of buffered outputs with two long outputs split over
    wavefronts in the first or the last round (ragged N)."""
    q = synth.ntt_primes(256, 2)
    long_ = synth.make_layer(synth.LayerConfig("long", N=192, L=2, n_in=130, n_out=2, T=1500, g=10,
                                               ternary=0.5), 4, moduli=q)
    short = synth.make_layer(synth.LayerConfig("short", N=192, L=2, n_in=130, n_out=40, T=20, g=10,
                                                ternary=0.5), 4, moduli=q)
    layer = _merge_layers(long_, short) if long_first else _merge_layers(short, long_)
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    st = fiona.Plan.from_layer(ctx, layer, flags=fiona.FIONA_PLAN_HOST_ONLY).stats()
    assert st["output_rounds"] == 3 and st["split_outputs"] == 2 and st["output_buffer_rows"] > 0, st
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    out_t, *_ = _run(layer, dev, x, pt)
    _assert_equal(_host(out_t, layer), expect, "rounds, long outputs %s" % ("first" if long_first else "last"))


def test_seeds_2_and_3_tiny(dev):
    for seed in (2, 3):
        layer = synth.make_layer(synth.CONFIGS["tiny"], seed)
        x, pt = synth.input_values(layer), synth.pt_values(layer)
        out_t, *_ = _run(layer, dev, x, pt)
        _assert_equal(_host(out_t, layer), oracle.weighted_sum_layer(layer, x, pt), "tiny seed %d" % seed)


def test_boundary_values(dev):
    """Largest residues everywhere: inputs and plaintexts q-1, scales 2^20-1."""
    layer = _small_layer("ragged_pool")
    q = np.asarray(layer.moduli, np.uint64)
    x = np.broadcast_to((q - 1)[None, None, :, None], (layer.n_in, 2, layer.L, layer.N)).copy()
    pt = np.broadcast_to((q - 1)[None, :, None], (layer.n_pt, layer.L, layer.N)).copy()
    scales = np.full(len(layer.scales), (1 << 20) - 1, np.uint64)
    lay2 = synth.Layer(**{**layer.__dict__, "scales": scales})
    expect = oracle.weighted_sum_layer(lay2, x, pt)
    out_t, *_ = _run(lay2, dev, x, pt)
    _assert_equal(_host(out_t, lay2), expect, "q-1 everywhere")
    # zeros everywhere
    out_t, *_ = _run(lay2, dev, np.zeros_like(x), np.zeros_like(pt))
    assert (_host(out_t, lay2) == 0).all()


def test_outputs_without_terms(dev):
    q = synth.ntt_primes(128, 1)
    cfg = synth.LayerConfig("empty", N=128, L=1, n_in=3, n_out=3, T=0, g=1, ternary=0.0)
    layer = synth.Layer(cfg=cfg, moduli=q, seed=1, n_in=3, n_out=3, out_global=np.arange(3, dtype=np.uint32),
                        pm_off=np.array([0, 0, 1, 1], np.uint32), pm_input=np.array([2], np.uint32),
                        pm_pt=np.array([0], np.uint32), grp_off=np.array([0, 0, 0, 1], np.uint32),
                        grp_mem_off=np.array([0, 2], np.uint32), mem_input=np.array([0, 1], np.uint32),
                        mem_sign=np.array([0, 0], np.int8), grp_scale=np.array([0], np.uint32),
                        scales=np.array([5], np.uint64), pt_global=np.arange(1, dtype=np.uint64))
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    out_t, *_ = _run(layer, dev, x, pt)
    got = _host(out_t, layer)
    _assert_equal(got, oracle.weighted_sum_layer(layer, x, pt), "empty outputs")
    assert (got[0] == 0).all() and (got[2] == 0).all()


def test_ntt_domain_product_is_ring_product(dev):
    """GPU PMult on NTT(a), NTT(b) at N = 64..256 equals the schoolbook negacyclic product."""
    for N in (64, 256):
        q = synth.ntt_primes(1 << 12, 2)
        psi = [oracle.find_psi(N, qq) for qq in q]
        rng = np.random.default_rng(N)
        a = [rng.integers(0, qq, N, dtype=np.uint64) for qq in q]
        b = [rng.integers(0, qq, N, dtype=np.uint64) for qq in q]
        A = np.stack([oracle.ntt(a[l], q[l], psi[l]) for l in range(2)])
        B = np.stack([oracle.ntt(b[l], q[l], psi[l]) for l in range(2)])
        cfg = synth.LayerConfig("ring", N=N, L=2, n_in=1, n_out=1, T=1, g=1, ternary=0.0)
        layer = synth.Layer(cfg=cfg, moduli=q, seed=1, n_in=1, n_out=1, out_global=np.arange(1, dtype=np.uint32),
                            pm_off=np.array([0, 1], np.uint32), pm_input=np.array([0], np.uint32),
                            pm_pt=np.array([0], np.uint32), grp_off=np.array([0, 0], np.uint32),
                            grp_mem_off=np.array([0], np.uint32), mem_input=np.zeros(0, np.uint32),
                            mem_sign=np.zeros(0, np.int8), grp_scale=np.zeros(0, np.uint32),
                            scales=np.zeros(0, np.uint64), pt_global=np.arange(1, dtype=np.uint64))
        x = np.stack([A, A])[None]
        out_t, *_ = _run(layer, dev, x, B[None])
        got = _host(out_t, layer)
        for l in range(2):
            assert (oracle.intt(got[0, 0, l], q[l], psi[l]) == oracle.negacyclic_mul(a[l], b[l], q[l])).all()


def test_toy_ckks_on_gpu(dev):
    from oracle import ckks_toy
    layer = synth.make_layer(synth.CONFIGS["tiny"], 1)
    toy, x, w, cts, pts, expected = ckks_toy.build_toy(layer)
    out_t, *_ = _run(layer, dev, cts, pts)
    got = _host(out_t, layer)
    _assert_equal(got, oracle.weighted_sum_layer(layer, cts, pts), "toy ckks")
    dec = np.stack([toy.decrypt(got[j]) for j in range(layer.n_out)])
    err = ckks_toy.relative_error(dec, expected)
    _say("[parity] toy CKKS decode relative error %.3g" % err)
    assert err <= 1e-3


def test_device_generator_matches_numpy(dev):
    import torch
    import synth.gpu
    cfg = synth.LayerConfig("gen", N=1000, L=3, n_in=5, n_out=2, T=10, g=5, ternary=0.5)
    layer = synth.make_layer(cfg, 9, moduli=synth.ntt_primes(1024, 3))
    in_t = torch.empty(layer.n_in * 2 * cfg.L * cfg.N, dtype=torch.int64, device=dev)
    synth.gpu.fill_inputs(layer, in_t)
    pt_t = torch.empty(layer.n_pt * cfg.L * cfg.N, dtype=torch.int64, device=dev)
    synth.gpu.fill_pts(layer, pt_t)
    torch.cuda.synchronize()
    assert (in_t.cpu().numpy().view(np.uint64).reshape(layer.n_in, 2, cfg.L, cfg.N) == synth.input_values(layer)).all()
    assert (pt_t.cpu().numpy().view(np.uint64).reshape(layer.n_pt, cfg.L, cfg.N) == synth.pt_values(layer)).all()
    allpm = synth.all_pmult_layer(layer)
    pa_t = torch.empty(allpm.n_pt * cfg.L * cfg.N, dtype=torch.int64, device=dev)
    synth.gpu.fill_pts(allpm, pa_t)
    torch.cuda.synchronize()
    assert (pa_t.cpu().numpy().view(np.uint64).reshape(allpm.n_pt, cfg.L, cfg.N) == synth.pt_values(allpm)).all()


# ---------------------------------------------------------------------------
# Full-size layers, sampled positions
# ---------------------------------------------------------------------------

def _check_sampled(layer, out_t, in_t, n_samples, seed, what):
    limbs, coeffs = synth.sample_positions(layer.N, layer.L, n_samples, seed)
    x_s = synth.input_values(layer, (limbs, coeffs))
    pt_s = synth.pt_values(layer, (limbs, coeffs)) if layer.n_pt else np.zeros((0, len(limbs)), np.uint64)
    # the device-filled inputs at these positions are the generator's values
    xin = in_t.view(layer.n_in, 2, layer.L, layer.N)[:, :, limbs, coeffs].cpu().numpy().view(np.uint64)
    assert (xin == x_s).all(), "device input generator disagrees with NumPy"
    expect = oracle.weighted_sum_sampled(layer, limbs, coeffs, x_s, pt_s, n_threads=16)
    got = out_t[: layer.n_out * 2 * layer.L * layer.N].view(layer.n_out, 2, layer.L, layer.N)[
        :, :, limbs, coeffs].cpu().numpy().view(np.uint64)
    bad = np.argwhere(got != expect)
    if bad.size:
        j, p, s = (int(v) for v in bad[0])
        raise AssertionError("%s: %d mismatches; first at out %d poly %d limb %d coeff %d: gpu %d oracle %d"
                             % (what, len(bad), j, p, limbs[s], coeffs[s], got[j, p, s], expect[j, p, s]))


@pytest.mark.parametrize("name", ["vgg11", "vit768", "bert_ffn"])
def test_full_size_sampled(dev, name):
    import torch
    layer = synth.make_layer(synth.CONFIGS[name], 1)
    _say("[parity] %s full size: %d outputs, %d raw terms, %d groups" % (name, layer.n_out, layer.n_pm,
                                                                        layer.n_group))
    out_t, in_t, pt_t, plan = _run(layer, dev, pitch="hint")   # the benchmark's plaintext layout
    _say("[parity] %s kernel done, plan %s" % (name, plan.stats()))
    del pt_t
    _check_sampled(layer, out_t, in_t, 48, 100, name)
    del out_t, in_t
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,width", [("vgg11", 2048), ("vit768", 2048), ("bert_ffn", 1024)])
def test_full_size_contiguous_tiles(dev, name, width):
    """Full-size layer in the benchmark's launch configuration: every output at
    every coefficient of a run of whole tiles at the start of limb 0 and at the
    end of the last limb (32 resp. 16 tiles each), element by element."""
    import torch
    layer = synth.make_layer(synth.CONFIGS[name], 1)
    out_t, in_t, pt_t, plan = _run(layer, dev, pitch="hint")
    _say("[parity] %s full size, %d contiguous coefficients in the first and last limb" % (name, width))
    del pt_t
    L, N = layer.L, layer.N
    limbs = np.concatenate([np.zeros(width, np.int64), np.full(width, L - 1, np.int64)])
    coeffs = np.concatenate([np.arange(width), np.arange(N - width, N)]).astype(np.int64)
    x_s = synth.input_values(layer, (limbs, coeffs))
    pt_s = synth.pt_values(layer, (limbs, coeffs))
    expect = oracle.weighted_sum_sampled(layer, limbs, coeffs, x_s, pt_s, n_threads=16)
    del pt_s
    got = out_t[: layer.n_out * 2 * L * N].view(layer.n_out, 2, L, N)[:, :, limbs, coeffs].cpu().numpy().view(np.uint64)
    bad = np.argwhere(got != expect)
    if bad.size:
        j, p, i = (int(v) for v in bad[0])
        raise AssertionError("%s: %d mismatches; first at out %d poly %d limb %d coeff %d"
                             % (name, len(bad), j, p, limbs[i], coeffs[i]))
    del out_t, in_t
    torch.cuda.empty_cache()


def test_full_size_large_all_chunks(dev):
    import torch
    import synth.gpu
    layer = synth.make_layer(synth.CONFIGS["large4096"], 1)
    in_t = torch.empty(layer.n_in * 2 * layer.L * layer.N, dtype=torch.int64, device=dev)
    synth.gpu.fill_inputs(layer, in_t)
    limbs, coeffs = synth.sample_positions(layer.N, layer.L, 24, 101)
    x_s = synth.input_values(layer, (limbs, coeffs))
    chunks = synth.output_chunks(layer.n_out, layer.cfg.chunks_hybrid)
    max_pt = max(synth.chunk_layer(layer, a, b).n_pt for a, b in chunks)
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    pitch = ctx.pt_pitch_hint()   # the benchmark's plaintext layout
    pt_t = torch.empty((max_pt - 1) * pitch + layer.L * layer.N, dtype=torch.int64, device=dev)
    out_c = torch.empty((layer.n_out // len(chunks) + 1) * 2 * layer.L * layer.N, dtype=torch.int64, device=dev)
    sign_all = _to_dev(layer.mem_sign, np.int8, dev)
    for ci, (a, b) in enumerate(chunks):
        ch = synth.chunk_layer(layer, a, b)
        synth.gpu.fill_pts(ch, pt_t, pitch)
        plan = fiona.Plan.from_layer(ctx, ch, pt_pitch=pitch)
        sign_t = _to_dev(ch.mem_sign, np.int8, dev)
        scale_t = _to_dev(ch.scales, np.int64, dev)
        fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, out_c)
        torch.cuda.synchronize()
        if ci % 4 == 0 or ci == len(chunks) - 1:
            _say("[parity] large4096 chunk %d/%d (outputs %d..%d) done" % (ci + 1, len(chunks), a, b - 1))
        pt_s = synth.pt_values(ch, (limbs, coeffs))
        expect = oracle.weighted_sum_sampled(ch, limbs, coeffs, x_s, pt_s, n_threads=16)
        got = out_c[: ch.n_out * 2 * layer.L * layer.N].view(ch.n_out, 2, layer.L, layer.N)[
            :, :, limbs, coeffs].cpu().numpy().view(np.uint64)
        assert (got == expect).all(), "large4096 chunk %d mismatch" % ci
    del pt_t, out_c, in_t, sign_all
    torch.cuda.empty_cache()


def test_full_size_all_pmult_route_equivalence(dev):
    """VGG11-like layer: the all-PMult layer gives exactly the hybrid outputs at every position."""
    import torch
    layer = synth.make_layer(synth.CONFIGS["vgg11"], 1)
    out_h, in_t, pt_t, _ = _run(layer, dev, pitch="hint")
    del pt_t
    allpm = synth.all_pmult_layer(layer)
    out_a, in_a, pt_a, _ = _run(allpm, dev, pitch="hint")
    del pt_a, in_a
    assert torch.equal(out_h, out_a)
    _check_sampled(allpm, out_a, in_t, 16, 102, "vgg11 all-PMult")
    del out_h, out_a, in_t
    torch.cuda.empty_cache()


def test_runtime_signs_are_read(dev):
    """The kernel takes the member signs from ternary_groups on every call: with
    a plan built without sharing, flipping or zeroing members' signs after plan
    creation gives the oracle's result for the new signs."""
    layer = _small_layer("ragged_pool")
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    rng = np.random.default_rng(3)
    signs2 = layer.mem_sign.copy()
    nz = np.nonzero(signs2)[0]
    pick = rng.choice(nz, size=len(nz) // 3, replace=False)
    signs2[pick[: len(pick) // 2]] *= -1
    signs2[pick[len(pick) // 2:]] = 0
    lay2 = synth.Layer(**{**layer.__dict__, "mem_sign": signs2})
    expect = oracle.weighted_sum_layer(lay2, x, pt)
    out_t, *_ = _run(layer, dev, x, pt, flags=fiona.FIONA_PLAN_NO_SHARING, signs=signs2)
    _assert_equal(_host(out_t, layer), expect, "run-time signs")


# ---------------------------------------------------------------------------
# Route equivalence at full size (Sec. 3 Obs. 2 / Table 1: the hybrid and the
# all-PMult forms of a layer compute the same outputs), every output chunk
# ---------------------------------------------------------------------------

def _run_all_chunks(layer, dev, in_t, n_chunks, tag):
    """Every output chunk of `layer` in the benchmark's launch configuration
    (padded plaintext rows, one plaintext buffer refilled per chunk); returns
    the full [n_out][2][L][N] output on the device and the chunk ranges."""
    import torch
    import synth.gpu
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    pitch = ctx.pt_pitch_hint()
    chunks = synth.output_chunks(layer.n_out, n_chunks)
    subs = [synth.chunk_layer(layer, a, b) for a, b in chunks]
    LN = layer.L * layer.N
    pt_t = torch.empty((max(max(1, s.n_pt) for s in subs) - 1) * pitch + LN, dtype=torch.int64, device=dev)
    out = torch.full((layer.n_out * 2 * LN,), -1, dtype=torch.int64, device=dev)
    for ci, ((a, b), sub) in enumerate(zip(chunks, subs)):
        synth.gpu.fill_pts(sub, pt_t, pitch)
        plan = fiona.Plan.from_layer(ctx, sub, pt_pitch=pitch)
        sign_t = _to_dev(sub.mem_sign, np.int8, dev) if sub.mem_sign.size else \
            torch.zeros(1, dtype=torch.int8, device=dev)
        scale_t = _to_dev(sub.scales, np.int64, dev) if sub.scales.size else \
            torch.zeros(1, dtype=torch.int64, device=dev)
        fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, out[a * 2 * LN: b * 2 * LN])
        torch.cuda.synchronize()
        if ci % 8 == 0 or ci == len(chunks) - 1:
            _say("[parity] %s chunk %d/%d (outputs %d..%d) done" % (tag, ci + 1, len(chunks), a, b - 1))
        del plan
    del pt_t
    torch.cuda.empty_cache()
    return out, chunks


@pytest.mark.parametrize("name", ["vit768", "bert_ffn", "large4096"])
def test_full_size_all_pmult_every_chunk(dev, name):
    """The all-PMult layer (every signed term a PMult by its constant
    plaintext h*c), run in the benchmark's output chunks, equals the hybrid
    layer at every output, polynomial, limb and coefficient; each all-PMult
    chunk also matches the oracle at sampled positions."""
    import torch
    import synth.gpu
    layer = synth.make_layer(synth.CONFIGS[name], 1)
    in_t = torch.empty(layer.n_in * 2 * layer.L * layer.N, dtype=torch.int64, device=dev)
    synth.gpu.fill_inputs(layer, in_t)
    out_h, _ = _run_all_chunks(layer, dev, in_t, layer.cfg.chunks_hybrid, name + " hybrid")
    allpm = synth.all_pmult_layer(layer)
    out_a, chunks = _run_all_chunks(allpm, dev, in_t, layer.cfg.chunks_allpm, name + " all-PMult")
    LN = layer.L * layer.N
    for ci, (a, b) in enumerate(chunks):
        if not torch.equal(out_h[a * 2 * LN: b * 2 * LN], out_a[a * 2 * LN: b * 2 * LN]):
            diff = (out_h[a * 2 * LN: b * 2 * LN] != out_a[a * 2 * LN: b * 2 * LN]).nonzero()
            w = int(diff[0]) + a * 2 * LN
            raise AssertionError("%s all-PMult chunk %d differs from hybrid at %d words; first at out %d poly %d "
                                 "limb %d coeff %d" % (name, ci, diff.numel(), w // (2 * LN), (w // LN) % 2,
                                                       (w // layer.N) % layer.L, w % layer.N))
    _say("[parity] %s: all-PMult == hybrid at all %d outputs x 2 x %d x %d" % (name, layer.n_out, layer.L, layer.N))
    limbs, coeffs = synth.sample_positions(layer.N, layer.L, 10, 103)
    x_s = synth.input_values(layer, (limbs, coeffs))
    for ci, (a, b) in enumerate(chunks):
        sub = synth.chunk_layer(allpm, a, b)
        expect = oracle.weighted_sum_sampled(sub, limbs, coeffs, x_s, synth.pt_values(sub, (limbs, coeffs)),
                                             n_threads=16)
        got = out_a[a * 2 * LN: b * 2 * LN].view(b - a, 2, layer.L, layer.N)[:, :, limbs, coeffs]
        got = got.cpu().numpy().view(np.uint64)
        bad = np.argwhere(got != expect)
        if bad.size:
            j, p, s = (int(v) for v in bad[0])
            raise AssertionError("%s all-PMult chunk %d: %d mismatches with the oracle; first at out %d poly %d "
                                 "limb %d coeff %d" % (name, ci, len(bad), a + j, p, limbs[s], coeffs[s]))
    del out_h, out_a, in_t
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["tiny", "ragged_pool", "partial_share", "repeated_pool"])
def test_small_all_pmult_elementwise(dev, name):
    """The all-PMult form of a small layer on the GPU, element by element
    against the oracle, and equal to the hybrid form's oracle result."""
    layer = _small_layer(name)
    allpm = synth.all_pmult_layer(layer)
    x = synth.input_values(layer)
    expect = oracle.weighted_sum_layer(allpm, x, synth.pt_values(allpm), n_threads=8)
    _assert_equal(expect, oracle.weighted_sum_layer(layer, x, synth.pt_values(layer), n_threads=8),
                  name + " oracle: all-PMult vs hybrid")
    out_t, *_ = _run(allpm, dev, x, synth.pt_values(allpm))
    _assert_equal(_host(out_t, allpm), expect, name + " all-PMult")


@pytest.mark.parametrize("chunk", [0, 15])
def test_full_size_large_contiguous_tiles(dev, chunk):
    """Large 4096x4096 layer, one output chunk in the benchmark's launch
    configuration: every output of the chunk at every coefficient of 16 whole
    tiles at the start of limb 0 and 16 at the end of the last limb."""
    import torch
    import synth.gpu
    layer = synth.make_layer(synth.CONFIGS["large4096"], 1)
    a, b = synth.output_chunks(layer.n_out, layer.cfg.chunks_hybrid)[chunk]
    sub = synth.chunk_layer(layer, a, b)
    _say("[parity] large4096 chunk %d (outputs %d..%d): contiguous tiles" % (chunk, a, b - 1))
    out_t, in_t, pt_t, plan = _run(sub, dev, pitch="hint")
    del pt_t
    L, N, width = layer.L, layer.N, 1024
    limbs = np.concatenate([np.zeros(width, np.int64), np.full(width, L - 1, np.int64)])
    coeffs = np.concatenate([np.arange(width), np.arange(N - width, N)]).astype(np.int64)
    x_s = synth.input_values(sub, (limbs, coeffs))
    expect = oracle.weighted_sum_sampled(sub, limbs, coeffs, x_s, synth.pt_values(sub, (limbs, coeffs)),
                                         n_threads=16)
    got = out_t[: sub.n_out * 2 * L * N].view(sub.n_out, 2, L, N)[:, :, limbs, coeffs].cpu().numpy().view(np.uint64)
    bad = np.argwhere(got != expect)
    if bad.size:
        j, p, i = (int(v) for v in bad[0])
        raise AssertionError("large4096 chunk %d: %d mismatches; first at out %d poly %d limb %d coeff %d"
                             % (chunk, len(bad), a + j, p, limbs[i], coeffs[i]))
    del out_t, in_t
    torch.cuda.empty_cache()


def test_checking_plan(dev):
    """A checking plan (FIONA_PLAN_CHECK_INPUTS) computes the same outputs; a
    call whose signs differ from the plan's, or whose input breaks the 2^50
    bound, is refused before anything is launched (the output keeps its fill)."""
    import torch
    layer = _small_layer("ragged_pool")
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    out_t, in_t, pt_t, plan = _run(layer, dev, x, pt, flags=fiona.FIONA_PLAN_CHECK_INPUTS)
    _assert_equal(_host(out_t, layer), expect, "checking plan")
    signs2 = layer.mem_sign.copy()
    nz = int(np.nonzero(signs2)[0][0])
    signs2[nz] = -signs2[nz]
    scale_t = _to_dev(layer.scales, np.int64, dev)
    out2 = torch.full_like(out_t, -1)
    with pytest.raises(fiona.FionaError) as e:
        fiona.hybrid_linear(plan, in_t, pt_t, _to_dev(signs2, np.int8, dev), scale_t, out2)
    assert e.value.status == fiona.FIONA_ERR_PRECONDITION
    x2 = x.copy()
    x2[-1, 1, -1, -1] = np.uint64(1 << 50)
    with pytest.raises(fiona.FionaError) as e:
        fiona.hybrid_linear(plan, _to_dev(x2, np.int64, dev), pt_t, _to_dev(layer.mem_sign, np.int8, dev), scale_t,
                            out2)
    assert e.value.status == fiona.FIONA_ERR_PRECONDITION
    torch.cuda.synchronize()
    assert bool((out2 == -1).all())


def test_checking_plan_input_passes(dev):
    """A checking plan over several input passes: the same outputs, and a
    changed sign of a member in the second pass's range is refused."""
    import torch
    layer = _small_layer("wide_320")
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    out_t, in_t, pt_t, plan = _run(layer, dev, x, pt, flags=fiona.FIONA_PLAN_CHECK_INPUTS)
    assert plan.stats()["input_passes"] == 3
    _assert_equal(_host(out_t, layer), oracle.weighted_sum_layer(layer, x, pt, n_threads=8), "checking plan, passes")
    signs2 = layer.mem_sign.copy()
    k = int(np.nonzero((layer.mem_input >= 150) & (signs2 != 0))[0][0])
    signs2[k] = -signs2[k]
    with pytest.raises(fiona.FionaError) as e:
        fiona.hybrid_linear(plan, in_t, pt_t, _to_dev(signs2, np.int8, dev), _to_dev(layer.scales, np.int64, dev),
                            torch.empty_like(out_t))
    assert e.value.status == fiona.FIONA_ERR_PRECONDITION


def test_input_pass_gap(dev):
    """320 inputs, terms on inputs 0..59 and 260..319 only: the middle input
    range gets no pass, and the last pass adds to the first one's outputs."""
    base = synth.make_layer(synth.LayerConfig("gap", N=192, L=2, n_in=120, n_out=6, T=240, g=12, ternary=0.6, pool=3),
                            7, moduli=synth.ntt_primes(256, 2))
    remap = lambda a: np.where(a < 60, a, a + 200).astype(np.uint32)
    layer = synth.Layer(**{**base.__dict__, "n_in": 320, "pm_input": remap(base.pm_input),
                           "mem_input": remap(base.mem_input)})
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    st = fiona.Plan.from_layer(ctx, layer, flags=fiona.FIONA_PLAN_HOST_ONLY).stats()
    assert st["input_passes"] == 2
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    out_t, *_ = _run(layer, dev, x, pt)
    _assert_equal(_host(out_t, layer), expect, "input pass gap")


@pytest.mark.parametrize("seed", range(64))
def test_random_layer(dev, seed):
    """Random layer descriptions (random terms and members, repeated inputs,
    empty outputs and groups, shared and reversed sums, hot pairs, input
    passes, ragged N, moduli near 2^20 and 2^50) under random plan flags and
    plaintext pitches, element by element against the oracle."""
    layer = random_layers.random_layer(seed)
    flags, pitch = random_layers.random_flags(seed)
    _say("random layer %d: N=%d L=%d n_in=%d n_out=%d raw=%d groups=%d members=%d flags=%d pitch=%s"
         % (seed, layer.N, layer.L, layer.n_in, layer.n_out, layer.n_pm, layer.n_group, layer.n_member, flags, pitch))
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    out_t, *_ = _run(layer, dev, x, pt, flags=flags, pitch=pitch)
    _assert_equal(_host(out_t, layer), expect, "random layer %d" % seed)
