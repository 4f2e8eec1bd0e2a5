"""Oracle for the rescale that follows the hybrid weighted sum -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module; the GPU library never does.

What is computed (paper Sec. 2, "Levels and Bootstrapping": a rescale
restores the scale after a multiplication and consumes one level; Sec. 4.2,
"Combining the Signed and Raw Routes": an output is rescaled once, after its
routes are summed).  CKKS rescaling divides the ciphertext's integer
coefficients by the last modulus of the chain and rounds.  Written out here
from that definition, coefficient by coefficient, in exact integers:

  1. every limb l of every polynomial goes back from the NTT domain to its
     coefficients mod q_l (the oracle's inverse NTT, whose convention is
     a_hat_k = sum_n a_n psi_l^((2k+1) n));
  2. the L residues of a coefficient give its integer C in [0, Q),
     Q = q_0 ... q_{L-1}, by the Chinese remainder theorem;
  3. C' = round(C / q_{L-1}), computed exactly as floor((2C + q_{L-1}) / (2 q_{L-1}))
     (q_{L-1} is odd, so there are no ties);
  4. C' mod q_l for l < L-1, forward NTT per limb.

The result has L-1 limbs.  Python integers carry the CRT; this is slow and
meant for single ciphertexts.
"""
from __future__ import annotations

import numpy as np

from . import find_psi, intt, ntt


def crt_coefficients(residues, moduli):
    """Integers C in [0, Q) from their residues: residues[l][k] = C_k mod moduli[l]."""
    Q = 1
    for q in moduli:
        Q *= int(q)
    acc = np.zeros(len(residues[0]), dtype=object)
    for l, q in enumerate(moduli):
        q = int(q)
        Ql = Q // q
        coef = Ql * pow(Ql, -1, q)
        acc = acc + np.array([int(v) for v in residues[l]], dtype=object) * coef
    return np.array([int(v) % Q for v in acc], dtype=object), Q


def rescale_poly(poly, moduli, psis=None):
    """One polynomial [L][N] in the NTT domain -> [L-1][N] after dividing by q_{L-1} with rounding."""
    L, N = poly.shape
    moduli = [int(q) for q in moduli]
    if psis is None:
        psis = [find_psi(N, q) for q in moduli]
    coeffs = [intt(poly[l], moduli[l], psis[l]) for l in range(L)]
    C, _ = crt_coefficients(coeffs, moduli)
    ql = moduli[-1]
    Cp = [(2 * int(c) + ql) // (2 * ql) for c in C]
    out = np.zeros((L - 1, N), dtype=np.uint64)
    for l in range(L - 1):
        q = moduli[l]
        out[l] = ntt(np.array([c % q for c in Cp], dtype=np.uint64), q, psis[l])
    return out


def rescale(ct, moduli, psis=None):
    """A ciphertext [2][L][N] (NTT domain) -> [2][L-1][N]."""
    return np.stack([rescale_poly(ct[p], moduli, psis) for p in range(ct.shape[0])])
