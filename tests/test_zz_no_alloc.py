"""fiona_hybrid_linear_static (word blocks in the library's static device
array, no allocation) against fiona_hybrid_linear, through the C ABI: two
calls in a row, the second on a smaller layer with fewer word blocks, each
bit-identical to the existing entry point's result (and to the oracle); the
size limit and the checking-plan refusal."""
import numpy as np
import pytest

import oracle
import synth
import paper_2609_35352_amd as fiona

pytestmark = pytest.mark.gpu

FIRST = synth.LayerConfig("static_first", N=512, L=3, n_in=20, n_out=40, T=80, g=8, ternary=0.7, pool=4)
SECOND = synth.LayerConfig("static_second", N=200, L=2, n_in=10, n_out=9, T=40, g=5, ternary=0.6)


def _dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fiona.lib()
    return torch.device("cuda:0")


def _t(a, dt, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(dt)).to(dev)


def _both(layer, dev):
    """Outputs of the existing entry point and of the static one on the same inputs."""
    import torch
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    plan = fiona.Plan.from_layer(ctx, layer)
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    in_t, pt_t = _t(x, np.int64, dev), _t(pt, np.int64, dev)
    sign_t, scale_t = _t(layer.mem_sign, np.int8, dev), _t(layer.scales, np.int64, dev)
    n = layer.n_out * 2 * layer.L * layer.N
    ref = torch.full((n,), -1, dtype=torch.int64, device=dev)
    got = torch.full((n,), -2, dtype=torch.int64, device=dev)
    print("[no-alloc] %s: N=%d L=%d outputs=%d stats=%s" % (layer.cfg.name, layer.N, layer.L, layer.n_out,
                                                            plan.stats()), flush=True)
    fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, ref)
    fiona.hybrid_linear_static(plan, in_t, pt_t, sign_t, scale_t, got)
    torch.cuda.synchronize()
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    r = ref.cpu().numpy().view(np.uint64).reshape(expect.shape)
    g = got.cpu().numpy().view(np.uint64).reshape(expect.shape)
    return r, g, expect, plan


def test_static_entry_point_two_calls():
    dev = _dev()
    a = synth.make_layer(FIRST, 3, moduli=synth.ntt_primes(512, 3))
    b = synth.make_layer(SECOND, 4, moduli=synth.ntt_primes(256, 2))
    ra, ga, ea, pa = _both(a, dev)
    rb, gb, eb, pb = _both(b, dev)
    # the second call reads fewer word blocks than the first left in the array
    assert pb.stats()["n_use"] < pa.stats()["n_use"]
    for name, r, g, e in (("first", ra, ga, ea), ("second", rb, gb, eb)):
        assert np.array_equal(r, e), name + ": fiona_hybrid_linear differs from the oracle"
        bad = np.argwhere(g != r)
        assert not bad.size, "%s call: %d words differ, first at %s" % (name, len(bad), tuple(bad[0]))


def test_static_entry_point_limits():
    import torch
    dev = _dev()
    # 20000 uses: more word blocks than the 4 MiB array holds
    big = synth.make_layer(synth.LayerConfig("static_big", N=64, L=1, n_in=8, n_out=20, T=8000, g=8, ternary=1.0),
                           5, moduli=synth.ntt_primes(64, 1))
    ctx = fiona.Ctx(big.N, big.L, big.moduli)
    plan = fiona.Plan.from_layer(ctx, big)
    assert plan.stats()["n_use"] > 16384
    in_t = torch.zeros(big.n_in * 2 * big.N, dtype=torch.int64, device=dev)
    out_t = torch.zeros(big.n_out * 2 * big.N, dtype=torch.int64, device=dev)
    sign_t, scale_t = _t(big.mem_sign, np.int8, dev), _t(big.scales, np.int64, dev)
    with pytest.raises(fiona.FionaError) as e:
        fiona.hybrid_linear_static(plan, in_t, None, sign_t, scale_t, out_t)
    assert e.value.status == -3
    small = synth.make_layer(SECOND, 4, moduli=synth.ntt_primes(256, 2))
    ctx2 = fiona.Ctx(small.N, small.L, small.moduli)
    chk = fiona.Plan.from_layer(ctx2, small, flags=fiona.FIONA_PLAN_CHECK_INPUTS)
    x, pt = synth.input_values(small), synth.pt_values(small)
    out2 = torch.zeros(small.n_out * 2 * small.L * small.N, dtype=torch.int64, device=dev)
    with pytest.raises(fiona.FionaError) as e:
        fiona.hybrid_linear_static(chk, _t(x, np.int64, dev), _t(pt, np.int64, dev),
                                   _t(small.mem_sign, np.int8, dev), _t(small.scales, np.int64, dev), out2)
    assert e.value.status == fiona.FIONA_ERR_ARG


def test_static_entry_point_input_passes():
    """A layer over several input passes: every pass's word blocks go to the
    same static array in turn on the stream."""
    dev = _dev()
    wide = synth.make_layer(synth.LayerConfig("static_wide", N=128, L=2, n_in=200, n_out=12, T=400, g=16,
                                              ternary=0.6), 6, moduli=synth.ntt_primes(128, 2))
    r, g, e, plan = _both(wide, dev)
    assert plan.stats()["input_passes"] == 2
    assert np.array_equal(r, e) and np.array_equal(g, r)


@pytest.mark.parametrize("seed", range(0, 64, 4))
def test_static_entry_point_random_layers(seed):
    """The random layer descriptions (random_layers.py) under their plan flags
    (checking plans aside, which the static entry point refuses): both entry
    points bit-identical, and equal to the oracle."""
    import torch
    import random_layers
    dev = _dev()
    layer = random_layers.random_layer(seed)
    flags, _ = random_layers.random_flags(seed)
    flags &= ~fiona.FIONA_PLAN_CHECK_INPUTS
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    plan = fiona.Plan.from_layer(ctx, layer, flags=flags)
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    one = lambda a, dt, t: _t(a, dt, dev) if a.size else torch.zeros(1, dtype=t, device=dev)
    in_t, pt_t = one(x, np.int64, torch.int64), one(pt, np.int64, torch.int64)
    sign_t, scale_t = one(layer.mem_sign, np.int8, torch.int8), one(layer.scales, np.int64, torch.int64)
    n = layer.n_out * 2 * layer.L * layer.N
    ref = torch.full((n,), -1, dtype=torch.int64, device=dev)
    got = torch.full((n,), -2, dtype=torch.int64, device=dev)
    print("[no-alloc] random layer %d: N=%d L=%d n_in=%d outputs=%d flags=%d" % (seed, layer.N, layer.L, layer.n_in,
                                                                                   layer.n_out, flags), flush=True)
    fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, ref)
    fiona.hybrid_linear_static(plan, in_t, pt_t, sign_t, scale_t, got)
    torch.cuda.synchronize()
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    r = ref.cpu().numpy().view(np.uint64).reshape(expect.shape)
    g = got.cpu().numpy().view(np.uint64).reshape(expect.shape)
    assert np.array_equal(r, expect), "fiona_hybrid_linear differs from the oracle"
    bad = np.argwhere(g != r)
    assert not bad.size, "%d words differ, first at %s" % (len(bad), tuple(bad[0]))


def test_entry_points_in_a_hip_graph():
    """Both entry points captured in a HIP graph (the callers the static entry
    point is for) and replayed three times, with eager work on the outputs
    and a synchronisation between the replays; every replay equals the eager
    result, which equals the oracle."""
    import torch
    dev = _dev()
    layer = synth.make_layer(FIRST, 6, moduli=synth.ntt_primes(512, 3))
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    plan = fiona.Plan.from_layer(ctx, layer)
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    in_t, pt_t = _t(x, np.int64, dev), _t(pt, np.int64, dev)
    sign_t, scale_t = _t(layer.mem_sign, np.int8, dev), _t(layer.scales, np.int64, dev)
    n = layer.n_out * 2 * layer.L * layer.N
    ref = torch.full((n,), -1, dtype=torch.int64, device=dev)
    fiona.hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, ref)
    torch.cuda.synchronize()
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    assert np.array_equal(ref.cpu().numpy().view(np.uint64).reshape(expect.shape), expect)
    s = torch.cuda.Stream(device=dev)
    for name, entry in (("fiona_hybrid_linear", fiona.hybrid_linear), ("fiona_hybrid_linear_static",
                                                                        fiona.hybrid_linear_static)):
        out = torch.full((n,), -2, dtype=torch.int64, device=dev)
        entry(plan, in_t, pt_t, sign_t, scale_t, out, stream=s)   # outside the graph first
        torch.cuda.synchronize()
        print("[no-alloc] graph capture of %s" % name, flush=True)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            entry(plan, in_t, pt_t, sign_t, scale_t, out, stream=s)
        for r in range(3):
            out.fill_(-3)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(out, ref), "%s: replay %d differs from the eager result" % (name, r)
        del g
