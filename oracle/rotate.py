"""Oracle for hoisted baby-step rotations -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module; the GPU library never does.

What is computed.  The input ciphertexts A_i of a linear layer are the
packed input rotated by the layout's baby steps (paper Sec. 2, "Homomorphic
Operations": Rot cyclically shifts the slots; Sec. 2.2: a layer combines
PMult, Rot and Add; Sec. 4.2: the A_i are prepared according to the packing
layout).  The paper runs its layers in SEAL (Sec. 5) and does not spell out
how a rotation is computed, so this oracle takes the standard CKKS
construction, written out from its definition:

* Rot by r slots is the automorphism sigma_g: a(X) -> a(X^g), g = 5^r mod 2N,
  applied to both polynomials, then a key switch of the second one from
  sigma_g(s) back to the secret s.  Slot j of a message is its value at
  zeta^(5^j), zeta = exp(i pi / N) (the encoding of ``ckks_toy``), so sigma_g
  moves slot j + r to slot j.
* Key switching as SEAL does it: the second polynomial c1 is decomposed by
  RNS limb (digit j = the coefficients of c1 mod q_j, as integers in
  [0, q_j)), every digit is multiplied by its key polynomial over the data
  moduli and one special prime P, the products are summed, and the sum is
  divided by P with rounding.
* Hoisting: the digits are formed once per ciphertext and shared by all its
  rotations; the automorphism then acts on the integer digits.

For a ciphertext (c0, c1) over q_0 .. q_{L-1} (NTT domain) and a key
ksk[j][p] (j < L, p = 0, 1; NTT domain over q_0 .. q_{L-1}, P):

    D_j        = INTT_{q_j}(c1 limb j), integers in [0, q_j)
    sigma(D_j) = D_j(X^g) mod (X^N + 1), integer coefficients in (-q_j, q_j)
    u_p        = sum_j sigma(D_j) ksk[j][p]   in Z_m[X]/(X^N + 1), every modulus m
    v_p        = round(U_p / P) mod q_i, U_p in [0, Q P) the integer whose
                 residues are u_p (Chinese remainder theorem), per coefficient
    Rot(ct)    = (sigma(c0) + v_0, v_1)

The products use the oracle's NTT (pinned against the schoolbook negacyclic
product); the automorphism and the rounding division are done on the
coefficients, in exact integers.  Slow; meant for single ciphertexts.
"""
from __future__ import annotations

import numpy as np

from . import find_psi, intt, mul_acc, ntt
from .rescale import crt_coefficients


def galois_element(r: int, N: int) -> int:
    """g = 5^r mod 2N: the automorphism that rotates the slots by r."""
    return pow(5, r % (N // 2), 2 * N)


def automorphism_int(a: np.ndarray, g: int) -> np.ndarray:
    """a(X^g) mod (X^N + 1) for integer coefficients a (int64), g odd.

    X^n -> X^(n g); with e = n g mod 2N, X^e = -X^(e - N) when e >= N."""
    a = np.asarray(a, dtype=np.int64)
    N = len(a)
    if g % 2 == 0:
        raise ValueError("g must be odd")
    e = (np.arange(N, dtype=np.int64) * (g % (2 * N))) % (2 * N)
    neg = e >= N
    out = np.zeros(N, dtype=np.int64)
    out[np.where(neg, e - N, e)] = np.where(neg, -a, a)
    return out


def _limb(x: np.ndarray, m: int) -> np.ndarray:
    """Integer coefficients (int64, |x| < 2^63) -> residues in [0, m) as uint64."""
    return np.mod(np.asarray(x, dtype=np.int64), m).astype(np.uint64)


def automorphism_ntt(a_hat: np.ndarray, g: int, q: int, psi: int) -> np.ndarray:
    """sigma_g of one NTT-domain limb: to coefficients, X -> X^g, back."""
    a = intt(a_hat, q, psi).astype(np.int64)
    return ntt(_limb(automorphism_int(a, g), q), q, psi)


def _roots(N, moduli, P, psis, psi_p):
    moduli = [int(q) for q in moduli]
    if psis is None:
        psis = [find_psi(N, q) for q in moduli]
    if psi_p is None:
        psi_p = find_psi(N, int(P))
    return moduli, [int(p) for p in psis], int(P), int(psi_p)


def digits(c1: np.ndarray, moduli, psis) -> np.ndarray:
    """D_j = coefficients of c1 limb j, integers in [0, q_j): [L][N] int64."""
    return np.stack([intt(c1[j], int(q), int(psi)).astype(np.int64)
                     for j, (q, psi) in enumerate(zip(moduli, psis))])


def key_switch_sum(D: np.ndarray, key: np.ndarray, g: int, moduli, P, psis, psi_p) -> np.ndarray:
    """u [2][L+1][N] (NTT domain over q_0 .. q_{L-1}, P): sum_j sigma_g(D_j) ksk[j][p].

    key: [L][2][L+1][N], digit j, polynomial p, modulus (P last), NTT domain."""
    L, N = D.shape
    mods = list(moduli) + [P]
    roots = list(psis) + [psi_p]
    u = np.zeros((2, L + 1, N), dtype=np.uint64)
    for j in range(L):
        sd = automorphism_int(D[j], g)
        for i, (m, psi) in enumerate(zip(mods, roots)):
            d_hat = ntt(_limb(sd, m), m, psi)
            for p in range(2):
                mul_acc(u[p, i], d_hat, key[j, p, i], m)
    return u


def mod_down(u_poly: np.ndarray, moduli, P, psis, psi_p) -> np.ndarray:
    """[L+1][N] over q_0 .. q_{L-1}, P (NTT domain) -> [L][N]: each coefficient's
    integer U in [0, Q P) divided by P and rounded, round(U / P) =
    floor((2 U + P) / (2 P)) (P odd: no ties), reduced mod q_i."""
    mods = list(moduli) + [P]
    roots = list(psis) + [psi_p]
    coeffs = [intt(u_poly[i], m, psi) for i, (m, psi) in enumerate(zip(mods, roots))]
    U, _ = crt_coefficients(coeffs, mods)
    V = [(2 * int(x) + P) // (2 * P) for x in U]
    out = np.zeros((len(moduli), len(V)), dtype=np.uint64)
    for i, (q, psi) in enumerate(zip(moduli, psis)):
        out[i] = ntt(np.array([v % q for v in V], dtype=np.uint64), q, psi)
    return out


def rotate(ct: np.ndarray, g: int, key: np.ndarray, moduli, P, psis=None, psi_p=None) -> np.ndarray:
    """Rot(ct) for a ciphertext [2][L][N] (NTT domain), Galois element g and
    its key [L][2][L+1][N] (NTT domain, natural order): [2][L][N]."""
    N = ct.shape[2]
    moduli, psis, P, psi_p = _roots(N, moduli, P, psis, psi_p)
    D = digits(ct[1], moduli, psis)
    return rotate_hoisted(ct[0], D, g, key, moduli, P, psis, psi_p)


def rotate_hoisted(c0: np.ndarray, D: np.ndarray, g: int, key: np.ndarray, moduli, P, psis, psi_p) -> np.ndarray:
    """Rot with the digits D of c1 already formed (hoisting)."""
    u = key_switch_sum(D, key, g, moduli, P, psis, psi_p)
    v = [mod_down(u[p], moduli, P, psis, psi_p) for p in range(2)]
    out = np.zeros((2, len(moduli), c0.shape[1]), dtype=np.uint64)
    for i, (q, psi) in enumerate(zip(moduli, psis)):
        out[0, i] = (automorphism_ntt(c0[i], g, q, psi) + v[0][i]) % np.uint64(q)
        out[1, i] = v[1][i]
    return out


def rotation_key(s: np.ndarray, g: int, moduli, P, rng, sigma: float = 3.2, psis=None, psi_p=None) -> np.ndarray:
    """A key that switches sigma_g(s) to s, for the toy CKKS checks: [L][2][L+1][N],
    ksk[j][1] = a_j uniform, ksk[j][0] = -a_j s + e_j + P sigma_g(s) [m = q_j]
    (e_j rounded Gaussian), so that sum_j d_j ksk[j] = P d sigma_g(s) - (...) s
    + small for any digits d_j = d mod q_j."""
    N = len(s)
    moduli, psis, P, psi_p = _roots(N, moduli, P, psis, psi_p)
    L = len(moduli)
    mods = moduli + [P]
    roots = psis + [psi_p]
    sg = automorphism_int(np.asarray(s, dtype=np.int64), g)
    key = np.zeros((L, 2, L + 1, N), dtype=np.uint64)
    for j in range(L):
        e = np.rint(rng.normal(0.0, sigma, N)).astype(np.int64)
        for i, (m, psi) in enumerate(zip(mods, roots)):
            a = rng.integers(0, m, N, dtype=np.uint64)
            s_hat = ntt(_limb(s, m), m, psi)
            k0 = ntt(_limb(e, m), m, psi)
            mul_acc(k0, (np.uint64(m) - a) % np.uint64(m), s_hat, m)
            if i == j:
                mul_acc(k0, ntt(_limb(sg, m), m, psi), np.full(N, P % m, dtype=np.uint64), m)
            key[j, 0, i] = k0
            key[j, 1, i] = a
    return key
