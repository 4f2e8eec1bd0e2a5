"""GPU parity of the hoisted rotations (fiona_hoisted_rotate) against the
rotation oracle, bit for bit: random ciphertexts and random keys (in natural
NTT order, converted by fiona_rotation_key_layout), several rotations per
call, small and full-size rings; plus the toy CKKS round trip with real keys
and the argument checks."""
import numpy as np
import pytest

import synth
from oracle import ckks_toy
from oracle import rotate as orot
import paper_2609_35352_amd as fiona

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def _u64(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint64).view(np.int64)).to(dev)


def _host(t, shape):
    return t.cpu().numpy().view(np.uint64).reshape(shape)


def _random_case(N, L, n_rot, seed):
    ps = synth.ntt_primes(N, L + 1)
    moduli, P = ps[:L], ps[L]
    mods = moduli + [P]
    rng = np.random.default_rng(seed)
    ct = np.stack([np.stack([rng.integers(0, q, N, dtype=np.uint64) for q in moduli]) for _ in range(2)])
    keys = np.zeros((n_rot, L, 2, L + 1, N), dtype=np.uint64)
    for i, m in enumerate(mods):
        keys[:, :, :, i, :] = rng.integers(0, m, (n_rot, L, 2, N), dtype=np.uint64)
    return moduli, P, ct, keys


def _run_gpu(moduli, P, ct, keys, galois, dev, psi=None):
    L, N = ct.shape[1], ct.shape[2]
    n_rot = len(galois)
    ctx = fiona.Ctx(N, L, moduli)
    rot = fiona.Rotator(ctx, P, max(n_rot, 1), psi=psi)
    kw = rot.key_words()
    nat = _u64(keys.reshape(n_rot, kw), dev)
    lib_keys = torch.empty(n_rot * kw, dtype=torch.int64, device=dev)
    for r, g in enumerate(galois):
        fiona.rotation_key_layout(rot, g, nat[r], lib_keys[r * kw:(r + 1) * kw])
    out = torch.empty(n_rot * 2 * L * N, dtype=torch.int64, device=dev)
    print("[rotate] N=%d L=%d rotations=%s" % (N, L, list(galois)), flush=True)
    fiona.hoisted_rotate(rot, _u64(ct, dev), galois, lib_keys, out)
    torch.cuda.synchronize()
    return _host(out, (n_rot, 2, L, N)), rot, ctx


@pytest.mark.parametrize("N,L,steps,seed", [
    (256, 1, [1, 3], 1),
    (1024, 3, [1, 5, -1], 2),
    (4096, 4, [1, 2, 17, 1000], 3),
    (2048, 10, [7], 4),
    (1 << 17, 2, [1, 30000], 5),   # the largest ring: DFT sides 512 x 256
])
def test_rotate_matches_oracle(N, L, steps, seed):
    dev = _dev()
    galois = [orot.galois_element(r, N) for r in steps]
    moduli, P, ct, keys = _random_case(N, L, len(galois), seed)
    got, _, _ = _run_gpu(moduli, P, ct, keys, galois, dev)
    for r, g in enumerate(galois):
        want = orot.rotate(ct, g, keys[r], moduli, P)
        bad = np.argwhere(got[r] != want)
        assert bad.size == 0, "rotation %d (g=%d): %d mismatches, first %s" % (r, g, len(bad), bad[:3].tolist())


def test_rotate_conjugation_and_identity():
    dev = _dev()
    N, L = 512, 2
    galois = [2 * N - 1, 1]
    moduli, P, ct, keys = _random_case(N, L, len(galois), 8)
    got, _, _ = _run_gpu(moduli, P, ct, keys, galois, dev)
    for r, g in enumerate(galois):
        np.testing.assert_array_equal(got[r], orot.rotate(ct, g, keys[r], moduli, P))


def test_rotate_toy_ckks_decrypts_to_rotated_slots():
    """Real keys: the GPU result is the oracle's bit for bit and decrypts to the rotated slots."""
    dev = _dev()
    N, L = 2048, 3
    ps = synth.ntt_primes(N, L + 1)
    moduli, P = ps[:L], ps[L]
    tk = ckks_toy.ToyCKKS(N, moduli, seed=21)
    rng = np.random.default_rng(22)
    z = rng.uniform(-1, 1, N // 2)
    ct = tk.encrypt(z)
    steps = [1, 4, 100]
    galois = [orot.galois_element(r, N) for r in steps]
    keys = np.stack([orot.rotation_key(tk.s, g, moduli, P, rng, psis=tk.psi) for g in galois])
    psi = list(tk.psi) + [orot.find_psi(N, P)]
    got, _, _ = _run_gpu(moduli, P, ct, keys, galois, dev, psi=psi)
    for r, (g, st) in enumerate(zip(galois, steps)):
        np.testing.assert_array_equal(got[r], orot.rotate(ct, g, keys[r], moduli, P, psis=tk.psi))
        dec = tk.decrypt(got[r], scale_bits=ckks_toy.DELTA_BITS)
        assert np.max(np.abs(dec - np.roll(z, -st))) < 1e-6


def test_rotate_full_size_vgg11_baby_steps():
    """N = 2^16, L = 8 (the VGG11-like layer's ring): its 63 baby-step rotations
    in one call; the first and the last are checked against the oracle in full."""
    dev = _dev()
    cfg = synth.CONFIGS["vgg11"]
    N, L = cfg.N, cfg.L
    ps = synth.ntt_primes(N, L + 1)
    moduli, P = ps[:L], ps[L]
    steps = list(range(1, cfg.n_in))
    galois = [orot.galois_element(r, N) for r in steps]
    ctx = fiona.Ctx(N, L, moduli)
    rot = fiona.Rotator(ctx, P, len(galois))
    kw = rot.key_words()
    rng = np.random.default_rng(31)
    ct = np.stack([np.stack([rng.integers(0, q, N, dtype=np.uint64) for q in moduli]) for _ in range(2)])
    checked = {0: None, len(galois) - 1: None}
    lib_keys = torch.empty(len(galois) * kw, dtype=torch.int64, device=dev)
    for r, g in enumerate(galois):
        kr = np.zeros((L, 2, L + 1, N), dtype=np.uint64)
        for i, m in enumerate(moduli + [P]):
            kr[:, :, i, :] = rng.integers(0, m, (L, 2, N), dtype=np.uint64)
        if r in checked:
            checked[r] = kr
        fiona.rotation_key_layout(rot, g, _u64(kr, dev), lib_keys[r * kw:(r + 1) * kw])
    out = torch.empty(len(galois) * 2 * L * N, dtype=torch.int64, device=dev)
    print("[rotate] full size N=%d L=%d, %d rotations" % (N, L, len(galois)), flush=True)
    fiona.hoisted_rotate(rot, _u64(ct, dev), galois, lib_keys, out)
    torch.cuda.synchronize()
    got = _host(out, (len(galois), 2, L, N))
    for r, kr in checked.items():
        want = orot.rotate(ct, galois[r], kr, moduli, P)
        assert np.array_equal(got[r], want), "rotation %d differs" % r
    # every rotation: canonical residues
    for i, q in enumerate(moduli):
        assert (got[:, :, i] < q).all()


def test_rotate_argument_errors():
    dev = _dev()
    N, L = 256, 2
    moduli, P, ct, keys = _random_case(N, L, 2, 5)
    ctx = fiona.Ctx(N, L, moduli)
    rot = fiona.Rotator(ctx, P, 2)
    kw = rot.key_words()
    assert kw == L * 2 * (L + 1) * N
    ct_t = _u64(ct, dev)
    k_t = torch.zeros(2 * kw, dtype=torch.int64, device=dev)
    out = torch.empty(2 * 2 * L * N, dtype=torch.int64, device=dev)
    for galois in ([2, 5], [5, 2 * N + 1]):
        with pytest.raises(fiona.FionaError) as e:
            fiona.hoisted_rotate(rot, ct_t, galois, k_t, out)
        assert e.value.status == -1
    with pytest.raises(fiona.FionaError):
        fiona.hoisted_rotate(rot, ct_t, [5, 5, 5], torch.zeros(3 * kw, dtype=torch.int64, device=dev),
                             torch.empty(3 * 2 * L * N, dtype=torch.int64, device=dev))
    with pytest.raises(fiona.FionaError) as e:   # output overlapping the input
        fiona.hoisted_rotate(rot, out[: 2 * L * N], [5], k_t, out)
    assert e.value.status == -5
    with pytest.raises(fiona.FionaError) as e:   # keys 8 but not 16 bytes aligned
        fiona.hoisted_rotate(rot, ct_t, [5], k_t[1:], out)
    assert e.value.status == -4
    fiona.hoisted_rotate(rot, ct_t, [], k_t, out)   # nothing to do
    torch.cuda.synchronize()


@pytest.mark.parametrize("name,steps,check", [
    ("vit768", [1, 5, 23], [0, 2]),
    ("large4096", [1, 2, 64, 127], [0, 3]),
])
def test_rotate_full_size_batched_digits(name, steps, check):
    """The full rings with L > 8 (digit batches of 16, padded for L = 10):
    keys drawn on the device in natural order, rotations checked in full."""
    import synth.gpu
    dev = _dev()
    cfg = synth.CONFIGS[name]
    N, L = cfg.N, cfg.L
    ps = synth.ntt_primes(N, L + 1)
    moduli, P = ps[:L], ps[L]
    galois = [orot.galois_element(r, N) for r in steps]
    ctx = fiona.Ctx(N, L, moduli)
    rot = fiona.Rotator(ctx, P, len(galois))
    kw = rot.key_words()
    nat_words = L * 2 * (L + 1) * N
    nat = torch.empty(len(galois) * nat_words, dtype=torch.int64, device=dev)
    synth.gpu.fill_rows(nat, len(galois) * L * 2 * (L + 1), moduli + [P], N, 41, synth.TAG_KEY)
    lib_keys = torch.empty(len(galois) * kw, dtype=torch.int64, device=dev)
    for r, g in enumerate(galois):
        fiona.rotation_key_layout(rot, g, nat[r * nat_words:(r + 1) * nat_words], lib_keys[r * kw:(r + 1) * kw])
    rng = np.random.default_rng(43)
    ct = np.stack([np.stack([rng.integers(0, q, N, dtype=np.uint64) for q in moduli]) for _ in range(2)])
    out = torch.empty(len(galois) * 2 * L * N, dtype=torch.int64, device=dev)
    print("[rotate] full size %s N=%d L=%d steps=%s" % (name, N, L, steps), flush=True)
    fiona.hoisted_rotate(rot, _u64(ct, dev), galois, lib_keys, out)
    torch.cuda.synchronize()
    got = _host(out, (len(galois), 2, L, N))
    for r in check:
        key = _host(nat[r * nat_words:(r + 1) * nat_words], (L, 2, L + 1, N))
        want = orot.rotate(ct, galois[r], key, moduli, P)
        assert np.array_equal(got[r], want), "%s rotation %d differs" % (name, r)


def test_rotate_two_output_rounds():
    """More rotations than one round of buffered outputs (64): 70 rotations,
    the round edges checked against the oracle."""
    dev = _dev()
    N, L = 256, 2
    steps = list(range(1, 71))
    galois = [orot.galois_element(r, N) for r in steps]
    moduli, P, ct, keys = _random_case(N, L, len(galois), 12)
    got, _, _ = _run_gpu(moduli, P, ct, keys, galois, dev)
    for r in (0, 1, 62, 63, 64, 65, 69):
        np.testing.assert_array_equal(got[r], orot.rotate(ct, galois[r], keys[r], moduli, P))


def test_rotate_max_rotations():
    """The most rotations one call takes (256: four rounds of buffered
    outputs), steps repeating; the round edges checked against the oracle."""
    dev = _dev()
    N, L = 256, 2
    steps = [1 + (i % 127) for i in range(256)]
    galois = [orot.galois_element(r, N) for r in steps]
    moduli, P, ct, keys = _random_case(N, L, len(galois), 13)
    got, _, _ = _run_gpu(moduli, P, ct, keys, galois, dev)
    for r in (0, 63, 64, 127, 128, 191, 192, 255):
        np.testing.assert_array_equal(got[r], orot.rotate(ct, galois[r], keys[r], moduli, P))


@pytest.mark.parametrize("N,g", [(256, 5), (2048, 2 * 2048 - 1)])
def test_rotation_key_layout_format(N, g):
    """The library's key layout word for word, as include/fiona.h documents
    it: every row of N residues permuted by the rotation's slot map and
    stored transposed, K'[row][k2 N1 + k1] = K[row][pi^-1(k2 + N2 k1)],
    pi^-1(i) = (i - (g - 1) / 2) g^-1 mod N."""
    dev = _dev()
    L = 2
    moduli, P, _, keys = _random_case(N, L, 1, 14)
    ctx = fiona.Ctx(N, L, moduli)
    rot = fiona.Rotator(ctx, P, 1)
    kw = rot.key_words()
    out = torch.empty(kw, dtype=torch.int64, device=dev)
    fiona.rotation_key_layout(rot, g, _u64(keys[0].reshape(-1), dev), out)
    torch.cuda.synchronize()
    got = _host(out, (-1, N))
    logn = N.bit_length() - 1
    log_n1, log_n2 = (logn + 1) // 2, logn // 2
    a = np.arange(N)
    i = (a >> log_n1) + ((a & ((1 << log_n1) - 1)) << log_n2)   # a = k2 N1 + k1 holds i = k2 + N2 k1
    src = ((i - (g - 1) // 2) * pow(g, -1, N)) % N
    np.testing.assert_array_equal(got, keys[0].reshape(-1, N)[:, src])



def test_rotate_in_a_hip_graph():
    """fiona_hoisted_rotate captured in a HIP graph (one call = its launches,
    the Galois elements passed by value, no memset or copy) and replayed three
    times, with eager work on the output between the replays: every replay
    equals the eager call, which equals the oracle."""
    dev = _dev()
    N, L = 4096, 3
    galois = [orot.galois_element(r, N) for r in (1, 2, 5)]
    moduli, P, ct, keys = _random_case(N, L, len(galois), 7)
    ref_host, rot, ctx = _run_gpu(moduli, P, ct, keys, galois, dev)
    for r, g in enumerate(galois):
        assert np.array_equal(ref_host[r], orot.rotate(ct, g, keys[r], moduli, P))
    kw = rot.key_words()
    nat = _u64(keys.reshape(len(galois), kw), dev)
    lib_keys = torch.empty(len(galois) * kw, dtype=torch.int64, device=dev)
    for r, g in enumerate(galois):
        fiona.rotation_key_layout(rot, g, nat[r], lib_keys[r * kw:(r + 1) * kw])
    ct_t = _u64(ct, dev)
    ref = _u64(ref_host.reshape(-1), dev)
    s = torch.cuda.Stream(device=dev)
    out = torch.full((len(galois) * 2 * L * N,), -2, dtype=torch.int64, device=dev)
    fiona.hoisted_rotate(rot, ct_t, galois, lib_keys, out, stream=s)
    torch.cuda.synchronize()
    print("[rotate] graph capture N=%d L=%d rotations=%s" % (N, L, galois), flush=True)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        fiona.hoisted_rotate(rot, ct_t, galois, lib_keys, out, stream=s)
    for rep in range(3):
        out.fill_(-3)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), "replay %d differs from the eager call" % rep
    del graph
