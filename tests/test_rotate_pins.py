"""Pins of the rotation oracle (oracle/rotate.py) against what the mathematics
fixes, independently of the GPU path.

* The automorphism X -> X^g: monomials by repeated reduction with X^N = -1,
  the ring-homomorphism and group laws against the schoolbook negacyclic
  product, and its meaning on the slots (rotation by r for g = 5^r, complex
  conjugation for g = 2N - 1) through the canonical-embedding decoder.
* The division by the special prime: exact on multiples of P, and rounding
  away any error below P/2 (closed forms).
* End to end with real keys in the toy CKKS scheme: a rotated ciphertext
  decrypts to the rotated slots within the noise, and a key for another
  rotation does not.
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import ckks_toy
from oracle import rotate as orot
from oracle.rescale import crt_coefficients


def _primes(N, L):
    ps = synth.ntt_primes(N, L + 1)
    return ps[:L], ps[L]


@pytest.mark.parametrize("g", [1, 3, 5, 25, 31, 33, 63])
def test_automorphism_monomials(g):
    N = 32
    for n in range(N):
        a = np.zeros(N, dtype=np.int64)
        a[n] = 7
        e, sign = n * g, 1
        while e >= N:            # X^N = -1, one reduction at a time
            e -= N
            sign = -sign
        want = np.zeros(N, dtype=np.int64)
        want[e] = 7 * sign
        np.testing.assert_array_equal(orot.automorphism_int(a, g), want)


def test_automorphism_ring_and_group_laws():
    N = 64
    q = synth.ntt_primes(N, 1)[0]
    rng = np.random.default_rng(3)
    a = rng.integers(0, q, N, dtype=np.uint64)
    b = rng.integers(0, q, N, dtype=np.uint64)
    sig = lambda x, g: np.mod(orot.automorphism_int(x.astype(np.int64), g), q).astype(np.uint64)
    for g in (3, 5, 77, 2 * N - 1):
        np.testing.assert_array_equal(sig(oracle.negacyclic_mul(a, b, q), g),
                                      oracle.negacyclic_mul(sig(a, g), sig(b, g), q))
        for h in (5, 9, 2 * N - 1):
            np.testing.assert_array_equal(sig(sig(a, h), g), sig(a, (g * h) % (2 * N)))
    np.testing.assert_array_equal(sig(a, 1), a)


@pytest.mark.parametrize("r", [1, 2, 7, 100, 255])
def test_automorphism_rotates_slots(r):
    N = 1024
    rng = np.random.default_rng(r)
    z = rng.uniform(-1, 1, N // 2) + 1j * rng.uniform(-1, 1, N // 2)
    scale = float(1 << 30)
    m = ckks_toy.encode(z, N, scale)
    g = orot.galois_element(r, N)
    got = ckks_toy.decode(orot.automorphism_int(m, g), N, scale)
    np.testing.assert_allclose(got, np.roll(z, -r), atol=1e-6)
    conj = ckks_toy.decode(orot.automorphism_int(m, 2 * N - 1), N, scale)
    np.testing.assert_allclose(conj, np.conj(z), atol=1e-6)


def test_galois_element_of_negative_and_wrapped_steps():
    N = 256
    assert orot.galois_element(0, N) == 1
    assert orot.galois_element(N // 2, N) == 1
    g1, gm1 = orot.galois_element(1, N), orot.galois_element(-1, N)
    assert (g1 * gm1) % (2 * N) == 1


def test_mod_down_divides_multiples_of_p_exactly():
    N, L = 256, 4
    moduli, P = _primes(N, L)
    psis = [oracle.find_psi(N, q) for q in moduli]
    psi_p = oracle.find_psi(N, P)
    rng = np.random.default_rng(5)
    x = [rng.integers(0, q, N, dtype=np.uint64) for q in moduli]   # coefficients mod q_i
    # an integer polynomial X with these residues; P X + e with |e| < P / 2
    X, Q = crt_coefficients(x, moduli)
    for e_bound in (0, P // 2 - 1):
        e = [int(v) for v in rng.integers(-e_bound, e_bound + 1, N)] if e_bound else [0] * N
        U = [P * int(c) + ei for c, ei in zip(X, e)]   # in (-P/2, Q P)
        U = [u % (Q * P) for u in U]   # X = 0, e < 0: Q P - |e| rounds to Q = 0 mod q_i
        mods = moduli + [P]
        roots = psis + [psi_p]
        u = np.stack([oracle.ntt(np.array([v % m for v in U], dtype=np.uint64), m, psi) for m, psi in zip(mods, roots)])
        got = orot.mod_down(u, moduli, P, psis, psi_p)
        want = np.stack([oracle.ntt(np.array([int(c) % q for c in X], dtype=np.uint64), q, psi)
                         for q, psi in zip(moduli, psis)])
        np.testing.assert_array_equal(got, want)


@pytest.fixture(scope="module")
def toy():
    N, L = 2048, 3
    moduli, P = _primes(N, L)
    return ckks_toy.ToyCKKS(N, moduli, seed=11), P


@pytest.mark.parametrize("r", [1, 6, 511])
def test_rotation_decrypts_to_rotated_slots(toy, r):
    tk, P = toy
    N = tk.N
    rng = np.random.default_rng(100 + r)
    z = rng.uniform(-1, 1, N // 2)
    ct = tk.encrypt(z)
    g = orot.galois_element(r, N)
    key = orot.rotation_key(tk.s, g, tk.moduli, P, rng, psis=tk.psi)
    rot = orot.rotate(ct, g, key, tk.moduli, P, psis=tk.psi)
    assert rot.shape == ct.shape and all((rot[:, i] < q).all() for i, q in enumerate(tk.moduli))
    dec = tk.decrypt(rot, scale_bits=ckks_toy.DELTA_BITS)
    err = np.max(np.abs(dec - np.roll(z, -r)))
    assert err < 1e-6, err


def test_identity_key_switch_keeps_the_message(toy):
    tk, P = toy
    rng = np.random.default_rng(9)
    z = rng.uniform(-1, 1, tk.N // 2)
    ct = tk.encrypt(z)
    key = orot.rotation_key(tk.s, 1, tk.moduli, P, rng, psis=tk.psi)
    dec = tk.decrypt(orot.rotate(ct, 1, key, tk.moduli, P, psis=tk.psi), scale_bits=ckks_toy.DELTA_BITS)
    assert np.max(np.abs(dec - z)) < 1e-6


def test_key_of_another_rotation_fails(toy):
    """Negative control: the end-to-end pin has teeth."""
    tk, P = toy
    N = tk.N
    rng = np.random.default_rng(12)
    z = rng.uniform(-1, 1, N // 2)
    ct = tk.encrypt(z)
    g = orot.galois_element(1, N)
    wrong = orot.rotation_key(tk.s, orot.galois_element(2, N), tk.moduli, P, rng, psis=tk.psi)
    dec = tk.decrypt(orot.rotate(ct, g, wrong, tk.moduli, P, psis=tk.psi), scale_bits=ckks_toy.DELTA_BITS)
    assert np.max(np.abs(dec - np.roll(z, -1))) > 1.0
