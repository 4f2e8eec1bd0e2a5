"""Pins of the rescale oracle (oracle/rescale.py), CPU only.

The oracle divides each coefficient's CRT integer by the last modulus with
rounding (CKKS rescaling, paper Sec. 2 "Levels and Bootstrapping").  These
tests pin it to facts that do not go through its own formula:
  * inputs built as C = q_last * m + r with known m and |r| < q_last / 2 must
    give exactly m (remainders at +-(q_last - 1)/2 separate rounding from a
    floor or a ceiling; a wrong limb or CRT weight changes m);
  * the textbook RNS algorithm (only the last limb leaves the NTT domain;
    subtract its centred remainder and multiply by q_last^-1) must agree;
  * on toy CKKS ciphertexts the decrypted message is divided by q_last within
    the rescale error bound (1 + ||s||_1) / 2 per coefficient.
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import rescale as rs
from oracle.ckks_toy import ToyCKKS


def _ntt_limbs(coeffs_int, moduli, psis):
    return np.stack([oracle.ntt(np.array([int(c) % q for c in coeffs_int], dtype=np.uint64), q, psi)
                     for q, psi in zip(moduli, psis)])


@pytest.mark.parametrize("N,L,seed", [(16, 2, 1), (64, 3, 2), (256, 4, 3)])
def test_known_quotient_and_remainder(N, L, seed):
    moduli = synth.ntt_primes(N, L)
    psis = [oracle.find_psi(N, q) for q in moduli]
    ql = moduli[-1]
    rng = np.random.default_rng(seed)
    Qp = 1
    for q in moduli[:-1]:
        Qp *= q
    m = [int(v) for v in rng.integers(-(1 << 40), 1 << 40, N)]   # small, both signs
    r = [int(v) for v in rng.integers(-(ql // 2), ql // 2 + 1, N)]
    r[0], r[1], r[2] = (ql - 1) // 2, -((ql - 1) // 2), 0            # the rounding boundaries
    C = [ql * mi + ri for mi, ri in zip(m, r)]
    ct_poly = _ntt_limbs(C, moduli, psis)
    got = rs.rescale_poly(ct_poly, moduli, psis)
    want = _ntt_limbs([mi % Qp for mi in m], moduli[:-1], psis[:-1])
    assert np.array_equal(got, want)


def _rns_rescale(poly, moduli, psis):
    """Textbook RNS rescale, written independently of the oracle: only the last
    limb is inverse-transformed; its centred remainder is moved to each other
    limb, subtracted there, and the difference multiplied by q_last^-1."""
    L, N = poly.shape
    ql = moduli[-1]
    last = oracle.intt(poly[L - 1], ql, psis[L - 1])
    cent = [int(v) - ql if int(v) > ql // 2 else int(v) for v in last]
    out = np.zeros((L - 1, N), dtype=np.uint64)
    for l in range(L - 1):
        q = moduli[l]
        rem_hat = oracle.ntt(np.array([c % q for c in cent], dtype=np.uint64), q, psis[l])
        inv = pow(ql, -1, q)
        out[l] = np.array([((int(a) - int(b)) * inv) % q for a, b in zip(poly[l], rem_hat)], dtype=np.uint64)
    return out


@pytest.mark.parametrize("N,L,seed", [(32, 3, 4), (128, 5, 5)])
def test_rns_algorithm_agrees(N, L, seed):
    moduli = synth.ntt_primes(N, L)
    psis = [oracle.find_psi(N, q) for q in moduli]
    rng = np.random.default_rng(seed)
    poly = np.stack([np.array([int(v) for v in rng.integers(0, q, N, dtype=np.uint64)], dtype=np.uint64)
                     for q in moduli])
    assert np.array_equal(rs.rescale_poly(poly, moduli, psis), _rns_rescale(poly, moduli, psis))


def _message_ints(toy, ct):
    """Centred integer coefficients of the message of ct (CRT of c0 + c1*s)."""
    res = []
    for l, (q, psi) in enumerate(zip(toy.moduli, toy.psi)):
        m_hat = [(int(a) + int(b) * int(s)) % q for a, b, s in zip(ct[0, l], ct[1, l], toy.s_hat[l])]
        res.append(oracle.intt(np.array(m_hat, dtype=np.uint64), q, psi))
    C, Q = rs.crt_coefficients(res, toy.moduli)
    return [int(c) - Q if int(c) > Q // 2 else int(c) for c in C]


def test_toy_ckks_message_divided_by_last_modulus():
    N = 64
    moduli = synth.ntt_primes(N, 3)
    toy = ToyCKKS(N, moduli, seed=11)
    z = np.random.default_rng(12).uniform(-1, 1, N // 2)
    ct = toy.encrypt(z)
    # multiply by the integer constant 2^24 (a constant PMult): the message then
    # sits at scale 2^64, as after a weighted sum, far above q_last ~ 2^50
    K = 1 << 24
    ct = np.stack([np.stack([np.array([(int(v) * K) % q for v in ct[p, l]], dtype=np.uint64)
                             for l, q in enumerate(moduli)]) for p in range(2)])
    m = _message_ints(toy, ct)
    ct2 = rs.rescale(ct, moduli, toy.psi)
    small = ToyCKKS.__new__(ToyCKKS)
    small.N, small.moduli, small.psi, small.s, small.s_hat = N, moduli[:-1], toy.psi[:-1], toy.s, toy.s_hat[:-1]
    m2 = _message_ints(small, ct2)
    bound = (1 + int(np.sum(np.abs(toy.s)))) / 2 + 1
    ql = moduli[-1]
    err = max(abs(a - b / ql) for a, b in zip(m2, m))
    assert err <= bound
    # the message is large enough that dividing it (or not) is visible
    assert max(abs(b) for b in m) > 10 * ql and max(abs(a) for a in m2) > 10 * bound
