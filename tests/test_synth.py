"""Checks of the seeded input generators (synth) -- no GPU needed."""
import numpy as np
import pytest

import oracle
import synth


def _primes_below(n):
    sieve = np.ones(n, dtype=bool)
    sieve[:2] = False
    for p in range(2, int(n ** 0.5) + 1):
        if sieve[p]:
            sieve[p * p::p] = False
    return np.nonzero(sieve)[0].astype(np.uint64)


_SMALL_PRIMES = None


def _trial_division_prime(n: int) -> bool:
    """Independent of Miller-Rabin: divide by every prime below 2^25 (> sqrt(2^50))."""
    global _SMALL_PRIMES
    if _SMALL_PRIMES is None:
        _SMALL_PRIMES = _primes_below(1 << 25)
    ps = _SMALL_PRIMES[_SMALL_PRIMES * _SMALL_PRIMES <= np.uint64(n)]
    return not np.any(np.uint64(n) % ps == 0)


@pytest.mark.parametrize("N,L", [(1 << 12, 3), (1 << 16, 16)])
def test_prime_rule(N, L):
    qs = synth.ntt_primes(N, L)
    assert len(qs) == L and qs == sorted(qs, reverse=True)
    for q in qs:
        assert q < (1 << 50) and q % (2 * N) == 1
        assert _trial_division_prime(q)
    # completeness: no q' = 1 (mod 2N) between 2^50 and the first prime, or
    # between consecutive primes, is prime
    top = ((1 << 50) - 2) // (2 * N) * (2 * N) + 1
    cands = list(range(top, qs[-1], -2 * N))
    for c in cands:
        assert (c in qs) == _trial_division_prime(c)
    # a shorter list is a prefix
    assert synth.ntt_primes(N, 2) == qs[:2]


def test_generator_vector_matches_scalar_definition():
    idx = np.array([0, 1, 2, 12345, (1 << 40) + 7, (1 << 63) - 1], dtype=np.uint64)
    for seed, tag in [(1, synth.TAG_IN), (2, synth.TAG_PT), (3, synth.TAG_SIGN)]:
        v = synth.u64_np(seed, tag, idx)
        for k, i in enumerate(idx):
            assert int(v[k]) == synth.u64_int(seed, tag, int(i))
    # residues
    q = synth.ntt_primes(1 << 16, 1)[0]
    r = synth.uniform_mod_np(1, synth.TAG_IN, idx, q)
    for k, i in enumerate(idx):
        assert int(r[k]) == synth.uniform_mod_int(1, synth.TAG_IN, int(i), q) < q


def test_splitmix64_reference_values():
    # SplitMix64 seeded with 0: its first outputs are the published test values
    # of the generator (e.g. the reference implementation by Vigna).
    state = 0
    outs = []
    for _ in range(3):
        state = (state + synth.GOLDEN) & synth.MASK64
        outs.append(synth.mix64_int(state))
    assert outs == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_sign_distribution():
    u = synth.u64_np(1, synth.TAG_SIGN, np.arange(200000, dtype=np.uint64))
    s = synth.signs_from_u64(u)
    frac = [(s == v).mean() for v in (1, -1, 0)]
    assert abs(frac[0] - 0.35) < 0.005 and abs(frac[1] - 0.35) < 0.005 and abs(frac[2] - 0.30) < 0.005


EXPECTED_COUNTS = {
    # K = round(f * O * T / g); ternary terms = K * g; raw terms = O*T - K*g
    "tiny": (4, 32, 32),
    "vgg11": (543, 4344, 3848),       # round(0.53*128*64/8)   = round(542.72)
    "vit768": (749, 11984, 6448),     # round(0.65*24*768/16)  = round(748.8)
    "bert_ffn": (3663, 58608, 15120), # round(0.795*96*768/16) = round(3663.36)
    "large4096": (11469, 367008, 157280),  # round(0.70*128*4096/32) = round(11468.8)
}


@pytest.mark.parametrize("name", list(EXPECTED_COUNTS))
def test_layer_structure_counts(name):
    cfg = synth.CONFIGS[name]
    lay = synth.make_layer(cfg, 1)
    K, tern, raw = EXPECTED_COUNTS[name]
    assert lay.n_group == K and lay.n_member == tern and lay.n_pm == raw
    assert lay.ct_terms == cfg.n_out * cfg.T
    per_out = np.diff(lay.grp_off)
    assert per_out.max() - per_out.min() <= 1 and per_out.sum() == K
    # every member of a group is a distinct input; term t reads input t mod n_in
    for gi in range(0, K, max(1, K // 50)):
        mi = lay.mem_input[lay.grp_mem_off[gi]:lay.grp_mem_off[gi + 1]]
        assert len(set(mi.tolist())) == cfg.g
    assert (lay.scales >= 1).all() and (lay.scales < (1 << 20)).all()
    assert set(np.unique(lay.mem_sign).tolist()) <= {-1, 0, 1}


def test_pool_sharing_has_repeats():
    lay = synth.make_layer(synth.CONFIGS["vit768"], 1)
    sums = set()
    for gi in range(lay.n_group):
        a, b = lay.grp_mem_off[gi], lay.grp_mem_off[gi + 1]
        mi, ms = lay.mem_input[a:b], lay.mem_sign[a:b]
        nz = ms != 0
        key = tuple(sorted(zip(mi[nz].tolist(), ms[nz].tolist())))
        neg = tuple(sorted(zip(mi[nz].tolist(), (-ms[nz]).tolist())))
        sums.add(min(key, neg))
    assert len(sums) <= 48 < lay.n_group


def test_chunks_cover_the_layer():
    lay = synth.make_layer(synth.CONFIGS["vgg11"], 1)
    total_pm = total_grp = 0
    for j0, j1 in synth.output_chunks(lay.n_out, 5):
        ch = synth.chunk_layer(lay, j0, j1)
        total_pm += ch.n_pm
        total_grp += ch.n_group
        assert ch.n_pt == ch.n_pm
        assert (ch.pt_global == lay.pt_global[lay.pm_pt[lay.pm_off[j0]:lay.pm_off[j1]]]).all()
    assert total_pm == lay.n_pm and total_grp == lay.n_group


def test_sampled_values_match_full_arrays():
    cfg = synth.LayerConfig("s", N=256, L=3, n_in=6, n_out=3, T=12, g=4, ternary=0.5)
    lay = synth.make_layer(cfg, 4, moduli=synth.ntt_primes(256, 3))
    xf = synth.input_values(lay)
    pf = synth.pt_values(lay)
    limbs, coeffs = synth.sample_positions(cfg.N, cfg.L, 20, 2)
    xs = synth.input_values(lay, (limbs, coeffs))
    ps = synth.pt_values(lay, (limbs, coeffs))
    assert (xs == xf[:, :, limbs, coeffs]).all()
    assert (ps == pf[:, limbs, coeffs]).all()
    for l in range(cfg.L):
        assert (xf[:, :, l] < lay.moduli[l]).all() and (pf[:, l] < lay.moduli[l]).all()


def test_all_pmult_layer_is_the_same_function():
    """Route equivalence through the oracle: turning every signed term into a
    PMult by the constant plaintext h*c gives the same outputs."""
    cfg = synth.LayerConfig("r", N=128, L=2, n_in=8, n_out=4, T=16, g=4, ternary=0.5)
    lay = synth.make_layer(cfg, 6, moduli=synth.ntt_primes(128, 2))
    allpm = synth.all_pmult_layer(lay)
    assert allpm.n_group == 0 and allpm.n_pm == lay.ct_terms
    x = synth.input_values(lay)
    out_h = oracle.weighted_sum_layer(lay, x, synth.pt_values(lay))
    out_a = oracle.weighted_sum_layer(allpm, x, synth.pt_values(allpm))
    assert (out_h == out_a).all()
    # chunked all-PMult layers also agree
    for j0, j1 in synth.output_chunks(allpm.n_out, 3):
        ch = synth.chunk_layer(allpm, j0, j1)
        assert (oracle.weighted_sum_layer(ch, x, synth.pt_values(ch)) == out_h[j0:j1]).all()


def test_algorithmic_bytes():
    lay = synth.make_layer(synth.CONFIGS["vgg11"], 1)
    # 8 * L * N * (2*n_in + P + 2*O) = 8*8*65536*(128 + 3848 + 256)
    assert synth.algorithmic_bytes(lay) == 8 * 8 * 65536 * (128 + 3848 + 256)
