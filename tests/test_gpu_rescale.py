"""GPU parity of the rescale epilogue (fiona_rescale) against the oracle's
exact CRT rounding division (oracle/rescale.py), bit-exact on every limb and
coefficient of every ciphertext checked."""
import sys

import numpy as np
import pytest

import oracle
import synth
import paper_2609_35352_amd as fiona
from oracle import rescale as rs

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fiona.lib()
    return torch.device("cuda:0")


def _random_cts(n_ct, moduli, N, seed):
    rng = np.random.default_rng(seed)
    L = len(moduli)
    cts = np.zeros((n_ct, 2, L, N), dtype=np.uint64)
    for l, q in enumerate(moduli):
        cts[:, :, l, :] = rng.integers(0, q, (n_ct, 2, N), dtype=np.uint64)
    return cts


def _gpu_rescale(cts, moduli, dev, max_ct=None):
    import torch
    n_ct, _, L, N = cts.shape
    ctx = fiona.Ctx(N, L, moduli)
    r = fiona.Rescaler(ctx, max_ct or n_ct)
    in_t = torch.from_numpy(cts.reshape(-1).view(np.int64)).to(dev)
    out_t = torch.full((n_ct * 2 * (L - 1) * N,), -1, dtype=torch.int64, device=dev)
    fiona.rescale(r, in_t, n_ct, out_t)
    torch.cuda.synchronize()
    return out_t.cpu().numpy().view(np.uint64).reshape(n_ct, 2, L - 1, N)


@pytest.mark.parametrize("N,L,n_ct,seed", [(256, 2, 2, 1), (1 << 12, 3, 3, 2), (1 << 13, 5, 2, 3),
                                           (1 << 11, 4, 1, 4), (1 << 17, 2, 1, 5)])
def test_rescale_matches_oracle(dev, N, L, n_ct, seed):
    _say("[rescale] N=%d L=%d n_ct=%d seed=%d" % (N, L, n_ct, seed))
    moduli = synth.ntt_primes(N, L)
    cts = _random_cts(n_ct, moduli, N, seed)
    got = _gpu_rescale(cts, moduli, dev, max_ct=n_ct + 1)
    for c in range(n_ct):
        want = rs.rescale(cts[c], moduli)
        assert np.array_equal(got[c], want), "ciphertext %d differs" % c


@pytest.mark.parametrize("max_ct,launches", [(16384, 4), (10000, 2)])
def test_rescale_limbs_over_several_launches(dev, max_ct, launches):
    """A workspace for many ciphertexts limits the limbs per launch pair
    (65535 vectors per launch): 4 limbs in 4 launch pairs of 1, or in 2 of
    3 and 1; results as with one launch."""
    N, L, n_ct = 256, 5, 3
    assert -(-(L - 1) // min(L - 1, 65535 // (2 * max_ct))) == launches
    _say("[rescale] N=%d L=%d n_ct=%d max_ct=%d" % (N, L, n_ct, max_ct))
    moduli = synth.ntt_primes(N, L)
    cts = _random_cts(n_ct, moduli, N, 17)
    got = _gpu_rescale(cts, moduli, dev, max_ct=max_ct)
    for c in range(n_ct):
        assert np.array_equal(got[c], rs.rescale(cts[c], moduli)), "ciphertext %d differs" % c


def test_rescale_boundary_values(dev):
    """Coefficients at the rounding boundary and residues q-1 and 0."""
    N, L = 1 << 10, 3
    moduli = synth.ntt_primes(N, L)
    psis = [oracle.find_psi(N, q) for q in moduli]
    ql = moduli[-1]
    coeffs = [(ql - 1) // 2, (ql + 1) // 2, 0, ql - 1, ql, 2 * ql - 1] * (N // 6) + [1] * (N % 6)
    poly = np.stack([oracle.ntt(np.array([c % q for c in coeffs], dtype=np.uint64), q, psi)
                     for q, psi in zip(moduli, psis)])
    cts = np.stack([np.stack([poly, np.stack([np.full(N, q - 1, dtype=np.uint64) for q in moduli])])])
    got = _gpu_rescale(cts, moduli, dev)
    assert np.array_equal(got[0], rs.rescale(cts[0], moduli))


@pytest.mark.parametrize("name", ["vgg11", "large4096"])
def test_rescale_full_size(dev, name):
    """N = 2^16 with the VGG11-like layer's 8 limbs and the Large layer's 16
    (the four-step split 256 x 256; 7 and 15 forward limbs in one launch pair)."""
    cfg = synth.CONFIGS[name]
    moduli = synth.ntt_primes(cfg.N, cfg.L)
    _say("[rescale] full size N=%d L=%d" % (cfg.N, cfg.L))
    cts = _random_cts(1, moduli, cfg.N, 9)
    got = _gpu_rescale(cts, moduli, dev, max_ct=4)
    assert np.array_equal(got[0], rs.rescale(cts[0], moduli))


def test_hybrid_then_rescale(dev):
    """The epilogue after the hot path: hybrid weighted sum, then one rescale
    of each output (Sec. 4.2 "Combining"), against oracle sum then oracle rescale."""
    import torch
    layer = synth.make_layer(synth.CONFIGS["tiny"], 1)
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    expect = oracle.weighted_sum_layer(layer, x, pt, n_threads=8)
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    plan = fiona.Plan.from_layer(ctx, layer)
    to = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a).reshape(-1).view(dt)).to(dev)
    out_t = torch.empty(layer.n_out * 2 * layer.L * layer.N, dtype=torch.int64, device=dev)
    fiona.hybrid_linear(plan, to(x, np.int64), to(pt, np.int64), to(layer.mem_sign, np.int8),
                        to(layer.scales, np.int64), out_t)
    r = fiona.Rescaler(ctx, layer.n_out)
    res_t = torch.empty(layer.n_out * 2 * (layer.L - 1) * layer.N, dtype=torch.int64, device=dev)
    fiona.rescale(r, out_t, layer.n_out, res_t)
    torch.cuda.synchronize()
    got = res_t.cpu().numpy().view(np.uint64).reshape(layer.n_out, 2, layer.L - 1, layer.N)
    for j in range(layer.n_out):
        assert np.array_equal(got[j], rs.rescale(expect[j], layer.moduli))


def test_rescale_errors(dev):
    import torch
    N, L = 1 << 10, 3
    moduli = synth.ntt_primes(N, L)
    ctx = fiona.Ctx(N, L, moduli)
    r = fiona.Rescaler(ctx, 2)
    a = torch.zeros(3 * 2 * L * N, dtype=torch.int64, device=dev)
    b = torch.zeros(3 * 2 * (L - 1) * N, dtype=torch.int64, device=dev)
    with pytest.raises(fiona.FionaError) as e:
        fiona.rescale(r, a, 3, b)          # beyond max_ct
    assert e.value.status == -1
    with pytest.raises(fiona.FionaError) as e:
        fiona.rescale(r, a, 1, a[8:])      # output overlaps the input
    assert e.value.status == -5


def test_rescale_in_a_hip_graph(dev):
    """fiona_rescale captured in a HIP graph (one call = four NTT pass
    launches, no memset or copy) and replayed three times, with eager work on
    the output between the replays: every replay equals the eager call, which
    equals the oracle."""
    import torch
    N, L, n_ct = 1 << 12, 3, 3
    _say("[rescale] graph capture N=%d L=%d n_ct=%d" % (N, L, n_ct))
    moduli = synth.ntt_primes(N, L)
    cts = _random_cts(n_ct, moduli, N, 9)
    ctx = fiona.Ctx(N, L, moduli)
    r = fiona.Rescaler(ctx, n_ct)
    in_t = torch.from_numpy(cts.reshape(-1).view(np.int64)).to(dev)
    n = n_ct * 2 * (L - 1) * N
    ref = torch.full((n,), -1, dtype=torch.int64, device=dev)
    fiona.rescale(r, in_t, n_ct, ref)
    torch.cuda.synchronize()
    got = ref.cpu().numpy().view(np.uint64).reshape(n_ct, 2, L - 1, N)
    for c in range(n_ct):
        assert np.array_equal(got[c], rs.rescale(cts[c], moduli))
    s = torch.cuda.Stream(device=dev)
    out = torch.full((n,), -2, dtype=torch.int64, device=dev)
    fiona.rescale(r, in_t, n_ct, out, stream=s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        fiona.rescale(r, in_t, n_ct, out, stream=s)
    for rep in range(3):
        out.fill_(-3)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), "replay %d differs from the eager call" % rep
    del g
