"""Toy CKKS round trip -- TEST INFRASTRUCTURE ONLY.

Gives the hybrid weighted sum its meaning end to end: real slot vectors are
encoded and encrypted into RNS/NTT-domain ciphertexts, the weighted sum is
evaluated on the ciphertexts, and decrypting and decoding the result must give
the plaintext weighted sum

    y_j = sum_raw w_pi (*) x_i + sum_groups gamma_g * sum_members h * x_i

(paper Sec. 4.2, Eq. (routed-example) and Eq. (shared-example); slot-wise
products, gamma_g the group's reconstruction factor).  This plays the role of
the paper's check of decrypted compiled layers against an independent FP64
evaluation (Sec. 6.2).

Parameters of this toy (not the paper's, which uses SEAL with N = 2^16 and
scale 2^46 in Sec. 5): ciphertext scale Delta = 2^40, weight scale
Delta_w = 2^20, a uniform ternary secret, rounded Gaussian errors with
sigma = 3.2, symmetric encryption c1 = a, c0 = -a*s + m + e.  A raw weight
vector is encoded at Delta_w; a ternary group's integer scale c stands for the
reconstruction factor gamma = c / Delta_w (a constant vector, whose encoding is
the constant polynomial c).  Outputs stay at scale Delta * Delta_w (no rescale).

Encoding is the CKKS canonical embedding: slot j of m(X) is m(zeta^(5^j)) with
zeta = exp(i pi / N), j < N/2 (Cheon, Kim, Kim, Song, ASIACRYPT 2017).
"""
from __future__ import annotations

import numpy as np

from . import find_psi, intt, ntt, weighted_sum_layer

DELTA_BITS = 40
DELTA_W_BITS = 20


def _slot_roots(N: int):
    e = np.array([pow(5, j, 2 * N) for j in range(N // 2)], dtype=np.int64)
    t = (e - 1) // 2
    t_conj = ((2 * N - e) - 1) // 2
    return t, t_conj


def encode(z: np.ndarray, N: int, scale: float) -> np.ndarray:
    """Integer coefficients m with m(zeta^(5^j)) ~= scale * z_j (int64)."""
    t, tc = _slot_roots(N)
    F = np.zeros(N, dtype=np.complex128)
    F[t] = scale * z
    F[tc] = np.conj(scale * z)
    v = np.fft.fft(F) / N                      # inverse of F_t = sum_n v_n e^(2 pi i t n / N)
    zeta_neg = np.exp(-1j * np.pi * np.arange(N) / N)
    return np.rint((v * zeta_neg).real).astype(np.int64)


def decode(m: np.ndarray, N: int, scale: float) -> np.ndarray:
    """Slots m(zeta^(5^j)) / scale for real coefficients m."""
    t, _ = _slot_roots(N)
    v = np.asarray(m, dtype=np.float64) * np.exp(1j * np.pi * np.arange(N) / N)
    F = N * np.fft.ifft(v)                     # F_t = m(zeta^(2t+1))
    return F[t] / scale


def _mod_vec(m: np.ndarray, q: int) -> np.ndarray:
    return np.array([int(v) % q for v in m], dtype=np.uint64)


def _mul_mod(a: np.ndarray, b: np.ndarray, q: int) -> np.ndarray:
    return np.array([(int(x) * int(y)) % q for x, y in zip(a, b)], dtype=np.uint64)


def _add_mod(a: np.ndarray, b: np.ndarray, q: int) -> np.ndarray:
    return np.array([(int(x) + int(y)) % q for x, y in zip(a, b)], dtype=np.uint64)


class ToyCKKS:
    def __init__(self, N: int, moduli, seed: int = 7):
        self.N = N
        self.moduli = [int(q) for q in moduli]
        self.psi = [find_psi(N, q) for q in self.moduli]
        if not all(self.psi):
            raise ValueError("moduli must be 1 mod 2N")
        self.rng = np.random.default_rng(seed)
        self.s = self.rng.integers(-1, 2, N)                      # ternary secret
        self.s_hat = [ntt(_mod_vec(self.s, q), q, psi) for q, psi in zip(self.moduli, self.psi)]

    def encrypt(self, z: np.ndarray) -> np.ndarray:
        """[2][L][N] ciphertext (NTT domain) of slot vector z at scale 2^40."""
        N, L = self.N, len(self.moduli)
        m = encode(z, N, float(1 << DELTA_BITS))
        e = np.rint(self.rng.normal(0.0, 3.2, N)).astype(np.int64)
        ct = np.zeros((2, L, N), dtype=np.uint64)
        for l, (q, psi) in enumerate(zip(self.moduli, self.psi)):
            a_hat = np.array([int(v) for v in self.rng.integers(0, q, N, dtype=np.uint64)], dtype=np.uint64)
            me_hat = ntt(_mod_vec(m + e, q), q, psi)
            as_hat = _mul_mod(a_hat, self.s_hat[l], q)
            ct[0, l] = _add_mod(me_hat, np.array([(q - int(v)) % q for v in as_hat], dtype=np.uint64), q)
            ct[1, l] = a_hat
        return ct

    def encode_weight(self, w: np.ndarray) -> np.ndarray:
        """[L][N] NTT-domain plaintext of weight vector w at scale 2^20."""
        m = encode(w, self.N, float(1 << DELTA_W_BITS))
        return np.stack([ntt(_mod_vec(m, q), q, psi) for q, psi in zip(self.moduli, self.psi)])

    def decrypt(self, ct: np.ndarray, scale_bits: int = DELTA_BITS + DELTA_W_BITS) -> np.ndarray:
        """Slots of a [2][L][N] ciphertext whose message has scale 2^scale_bits."""
        N = self.N
        res = []
        for l, (q, psi) in enumerate(zip(self.moduli, self.psi)):
            m_hat = _add_mod(ct[0, l], _mul_mod(ct[1, l], self.s_hat[l], q), q)
            res.append(intt(m_hat, q, psi))
        Q = 1
        for q in self.moduli:
            Q *= q
        coeffs = np.zeros(N, dtype=np.float64)
        for k in range(N):
            acc = 0
            for l, q in enumerate(self.moduli):
                Ql = Q // q
                acc += int(res[l][k]) * Ql * pow(Ql, -1, q)
            acc %= Q
            if acc > Q // 2:
                acc -= Q
            coeffs[k] = acc / float(1 << scale_bits)
        return decode(coeffs, N, 1.0)


def build_toy(layer, seed: int = 7):
    """Encrypt random inputs and encode random raw weights for a synth Layer.

    Returns (toy, x_slots [n_in][N/2], w_slots [n_pt][N/2], in_cts [n_in][2][L][N],
    pts [n_pt][L][N], expected [n_out][N/2]) with the expected plaintext
    weighted sum in float64.
    """
    N = layer.N
    toy = ToyCKKS(N, layer.moduli, seed)
    rng = np.random.default_rng(seed + 1)
    x = rng.uniform(-1.0, 1.0, (layer.n_in, N // 2))
    w = rng.uniform(-1.0, 1.0, (layer.n_pt, N // 2))
    cts = np.stack([toy.encrypt(x[i]) for i in range(layer.n_in)])
    pts = np.stack([toy.encode_weight(w[p]) for p in range(layer.n_pt)]) if layer.n_pt else \
        np.zeros((0, len(layer.moduli), N), np.uint64)
    expected = np.zeros((layer.n_out, N // 2))
    for j in range(layer.n_out):
        for t in range(int(layer.pm_off[j]), int(layer.pm_off[j + 1])):
            expected[j] += w[layer.pm_pt[t]] * x[layer.pm_input[t]]
        for g in range(int(layer.grp_off[j]), int(layer.grp_off[j + 1])):
            gamma = float(layer.scales[layer.grp_scale[g]]) / float(1 << DELTA_W_BITS)
            u = np.zeros(N // 2)
            for m in range(int(layer.grp_mem_off[g]), int(layer.grp_mem_off[g + 1])):
                u += float(layer.mem_sign[m]) * x[layer.mem_input[m]]
            expected[j] += gamma * u
    return toy, x, w, cts, pts, expected


def relative_error(dec: np.ndarray, expected: np.ndarray) -> float:
    """Normwise relative error max|dec - y| / max|y| (real parts of the slots)."""
    return float(np.max(np.abs(dec.real - expected)) / np.max(np.abs(expected)))


def run_oracle(layer, seed: int = 7):
    toy, x, w, cts, pts, expected = build_toy(layer, seed)
    out = weighted_sum_layer(layer, cts, pts)
    dec = np.stack([toy.decrypt(out[j]) for j in range(layer.n_out)])
    return relative_error(dec, expected), out, (toy, cts, pts, expected)
