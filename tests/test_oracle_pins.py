"""Pins of the oracle to facts it does not compute itself.

Each test checks the oracle against something fixed by the paper or by the
mathematics: ring multiplication by schoolbook negacyclic convolution,
brute-force evaluation with multiplication done as repeated addition, the exact
grouping and sharing identities of Sec. 4.2, linearity, degenerate layers with
known results, and the toy CKKS decode against the float64 weighted sum.
"""
import json
import os

import numpy as np
import pytest

import oracle
import synth
from oracle import ckks_toy

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

Q12 = synth.ntt_primes(1 << 12, 3)
Q16 = synth.ntt_primes(1 << 16, 4)


def _single_output_layer(raw, groups):
    """raw: [(input, pt)], groups: [(scale, [(input, sign)])] for one output."""
    pm_off = np.array([0, len(raw)], np.uint32)
    pm_input = np.array([r[0] for r in raw], np.uint32)
    pm_pt = np.array([r[1] for r in raw], np.uint32)
    grp_off = np.array([0, len(groups)], np.uint32)
    mem_off = [0]
    mem_in, mem_sg, scales = [], [], []
    for c, mems in groups:
        for i, h in mems:
            mem_in.append(i)
            mem_sg.append(h)
        mem_off.append(len(mem_in))
        scales.append(c)
    return dict(pm_off=pm_off, pm_input=pm_input, pm_pt=pm_pt, grp_off=grp_off,
                grp_mem_off=np.array(mem_off, np.uint32), mem_input=np.array(mem_in, np.uint32),
                mem_sign=np.array(mem_sg, np.int8), grp_scale=np.arange(len(groups), dtype=np.uint32),
                scales=np.array(scales, np.uint64))


def _ws(q_pos, x, pt, d):
    return oracle.weighted_sum(q_pos, x, pt, d["pm_off"], d["pm_input"], d["pm_pt"], d["grp_off"],
                               d["grp_mem_off"], d["mem_input"], d["mem_sign"], d["grp_scale"], d["scales"])


# ---------------------------------------------------------------------------
# PMult meaning: element-wise NTT-domain product == multiplication in Z_q[X]/(X^N+1)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("N", [8, 16, 64, 256])
@pytest.mark.parametrize("q", [Q12[0], Q12[2], Q16[3]])
def test_pmult_is_negacyclic_ring_product(N, q):
    rng = np.random.default_rng(N + q % 1000)
    psi = oracle.find_psi(N, q)
    assert psi and pow(psi, N, q) == q - 1
    a = rng.integers(0, q, N, dtype=np.uint64)
    b = rng.integers(0, q, N, dtype=np.uint64)
    A, B = oracle.ntt_naive(a, q, psi), oracle.ntt_naive(b, q, psi)
    # one output, one raw term: plaintext B applied to ciphertext (A, A)
    d = _single_output_layer([(0, 0)], [])
    x = np.stack([A, A])[None]
    out = _ws(np.full(N, q, np.uint64), x, B[None], d)
    assert (out[0, 0] == out[0, 1]).all()
    prod = oracle.intt_naive(out[0, 0], q, psi)
    assert (prod == oracle.negacyclic_mul(a, b, q)).all()


def test_schoolbook_special_cases():
    q = Q12[0]
    N = 8
    # X * X^(N-1) = X^N = -1
    a = np.zeros(N, np.uint64); a[1] = 1
    b = np.zeros(N, np.uint64); b[N - 1] = 1
    c = oracle.negacyclic_mul(a, b, q)
    assert c[0] == q - 1 and (c[1:] == 0).all()


@pytest.mark.parametrize("N", [16, 128, 1024])
def test_fast_ntt_matches_definition_and_inverts(N):
    q = Q16[1]
    psi = oracle.find_psi(N, q)
    rng = np.random.default_rng(N)
    a = rng.integers(0, q, N, dtype=np.uint64)
    A = oracle.ntt(a, q, psi)
    if N <= 128:
        assert (A == oracle.ntt_naive(a, q, psi)).all()
    assert (oracle.intt(A, q, psi) == a).all()


def test_ntt_of_constant_is_constant():
    # A constant reconstruction factor encodes to a constant polynomial; its
    # NTT is the same constant in every slot, so its PMult is a scalar product.
    N, q = 64, Q12[1]
    psi = oracle.find_psi(N, q)
    c = np.zeros(N, np.uint64); c[0] = 777777
    assert (oracle.ntt(c, q, psi) == 777777).all()


# ---------------------------------------------------------------------------
# Brute force: tiny moduli, multiplication as repeated addition
# ---------------------------------------------------------------------------

def _brute_force(q_pos, x, pt, d):
    n_out = len(d["pm_off"]) - 1
    S = len(q_pos)
    out = np.zeros((n_out, 2, S), np.uint64)
    for s in range(S):
        q = int(q_pos[s])
        for j in range(n_out):
            for p in range(2):
                acc = 0
                for t in range(int(d["pm_off"][j]), int(d["pm_off"][j + 1])):
                    w = int(pt[d["pm_pt"][t], s])
                    xv = int(x[d["pm_input"][t], p, s])
                    for _ in range(w):          # w * xv as w additions
                        acc = (acc + xv) % q
                for g in range(int(d["grp_off"][j]), int(d["grp_off"][j + 1])):
                    c = int(d["scales"][d["grp_scale"][g]])
                    for m in range(int(d["grp_mem_off"][g]), int(d["grp_mem_off"][g + 1])):
                        xv = int(x[d["mem_input"][m], p, s])
                        h = int(d["mem_sign"][m])
                        for _ in range(c):      # c additions (or subtractions) of xv
                            if h > 0:
                                acc = (acc + xv) % q
                            elif h < 0:
                                acc = (acc - xv) % q
                out[j, p, s] = acc
    return out


def test_brute_force_tiny_moduli():
    rng = np.random.default_rng(5)
    qs = np.array([97, 193, 257, 12289, 2, 3], np.uint64)
    S = len(qs)
    n_in, n_out, n_pt = 5, 3, 6
    x = np.stack([rng.integers(0, qs) for _ in range(n_in * 2)]).reshape(n_in, 2, S).astype(np.uint64)
    pt = np.stack([rng.integers(0, qs) for _ in range(n_pt)]).astype(np.uint64)
    d = dict(pm_off=np.array([0, 2, 2, 5], np.uint32), pm_input=np.array([0, 4, 1, 1, 3], np.uint32),
             pm_pt=np.array([0, 5, 1, 2, 3], np.uint32), grp_off=np.array([0, 1, 3, 3], np.uint32),
             grp_mem_off=np.array([0, 3, 5, 6], np.uint32), mem_input=np.array([1, 2, 3, 0, 4, 2], np.uint32),
             mem_sign=np.array([1, -1, 0, -1, -1, 1], np.int8), grp_scale=np.array([2, 0, 1], np.uint32),
             scales=np.array([5, 11, 3], np.uint64))
    assert (_ws(qs, x, pt, d) == _brute_force(qs, x, pt, d)).all()


# ---------------------------------------------------------------------------
# Sec. 4.2 identities: grouping and sharing are exact
# ---------------------------------------------------------------------------

def test_grouping_identity_exact():
    """(sum_t h_t x_t) * c == sum_t (h_t c) x_t  (mod q), U formed in exact integers."""
    rng = np.random.default_rng(11)
    S = 64
    q_pos = np.array([Q16[s % 4] for s in range(S)], np.uint64)
    n_in = 16
    x = np.stack([rng.integers(0, q_pos) for _ in range(n_in * 2)]).reshape(n_in, 2, S).astype(np.uint64)
    signs = rng.choice([-1, 0, 1], size=n_in)
    c = int(rng.integers(1, 1 << 20))
    d = _single_output_layer([], [(c, [(i, int(signs[i])) for i in range(n_in)])])
    out = _ws(q_pos, x, np.zeros((0, S), np.uint64), d)
    for s in range(S):
        q = int(q_pos[s])
        for p in range(2):
            U = sum(int(signs[i]) * int(x[i, p, s]) for i in range(n_in))   # exact, unreduced
            assert int(out[0, p, s]) == (c * U) % q


def test_sharing_identity_exact():
    """Two outputs that share U (one with -U) == each output evaluated on its own."""
    rng = np.random.default_rng(12)
    S = 32
    q_pos = np.array([Q12[s % 3] for s in range(S)], np.uint64)
    x = np.stack([rng.integers(0, q_pos) for _ in range(8)]).reshape(4, 2, S).astype(np.uint64)
    c1, c2 = 12345, 999
    d = dict(pm_off=np.zeros(3, np.uint32), pm_input=np.zeros(0, np.uint32), pm_pt=np.zeros(0, np.uint32),
             grp_off=np.array([0, 1, 2], np.uint32), grp_mem_off=np.array([0, 3, 6], np.uint32),
             mem_input=np.array([0, 2, 3, 0, 2, 3], np.uint32), mem_sign=np.array([1, -1, 1, -1, 1, -1], np.int8),
             grp_scale=np.array([0, 1], np.uint32), scales=np.array([c1, c2], np.uint64))
    out = _ws(q_pos, x, np.zeros((0, S), np.uint64), d)
    for s in range(S):
        q = int(q_pos[s])
        for p in range(2):
            U = int(x[0, p, s]) - int(x[2, p, s]) + int(x[3, p, s])
            assert int(out[0, p, s]) == (c1 * U) % q
            assert int(out[1, p, s]) == (c2 * (-U)) % q


def test_linearity():
    rng = np.random.default_rng(13)
    lay = synth.make_layer(synth.LayerConfig("lin", N=64, L=2, n_in=12, n_out=5, T=24, g=6, ternary=0.5), 3,
                           moduli=Q16[:2])
    q_pos = np.repeat(np.asarray(lay.moduli, np.uint64), lay.N)
    S = q_pos.size
    X = np.stack([rng.integers(0, q_pos) for _ in range(lay.n_in * 2)]).reshape(lay.n_in, 2, S).astype(np.uint64)
    Y = np.stack([rng.integers(0, q_pos) for _ in range(lay.n_in * 2)]).reshape(lay.n_in, 2, S).astype(np.uint64)
    pt = np.stack([rng.integers(0, q_pos) for _ in range(lay.n_pt)]).astype(np.uint64)
    a = 987654321
    Z = np.array([[[(a * int(X[i, p, s]) + int(Y[i, p, s])) % int(q_pos[s]) for s in range(S)]
                   for p in range(2)] for i in range(lay.n_in)], dtype=np.uint64)
    f = lambda inp: oracle.weighted_sum(q_pos, inp, pt, lay.pm_off, lay.pm_input, lay.pm_pt, lay.grp_off,
                                        lay.grp_mem_off, lay.mem_input, lay.mem_sign, lay.grp_scale, lay.scales)
    oX, oY, oZ = f(X), f(Y), f(Z)
    for j in range(lay.n_out):
        for p in range(2):
            for s in range(S):
                assert int(oZ[j, p, s]) == (a * int(oX[j, p, s]) + int(oY[j, p, s])) % int(q_pos[s])


# ---------------------------------------------------------------------------
# Degenerate layers with known outputs
# ---------------------------------------------------------------------------

def test_special_cases():
    rng = np.random.default_rng(14)
    S = 40
    q_pos = np.array([Q16[s % 4] for s in range(S)], np.uint64)
    x = np.stack([rng.integers(0, q_pos) for _ in range(6)]).reshape(3, 2, S).astype(np.uint64)
    one = np.ones((1, S), np.uint64)
    # pt == 1, one term: copy of the input
    out = _ws(q_pos, x, one, _single_output_layer([(2, 0)], []))
    assert (out[0] == x[2]).all()
    # c = 1, h = +1, single member: copy; h = -1: negation
    out = _ws(q_pos, x, one, _single_output_layer([], [(1, [(1, 1)])]))
    assert (out[0] == x[1]).all()
    out = _ws(q_pos, x, one, _single_output_layer([], [(1, [(1, -1)])]))
    assert (out[0] == (q_pos - x[1]) % q_pos).all()
    # all signs zero: only the raw part remains
    out_raw = _ws(q_pos, x, one, _single_output_layer([(0, 0)], []))
    out_z = _ws(q_pos, x, one, _single_output_layer([(0, 0)], [(77, [(1, 0), (2, 0)])]))
    assert (out_raw == out_z).all()
    # an output with no terms is zero
    out = _ws(q_pos, x, one, _single_output_layer([], []))
    assert (out == 0).all()
    # boundary values: q-1 everywhere, pt q-1: (q-1)^2 = 1 mod q per term
    xm = np.broadcast_to(q_pos - 1, (3, 2, S)).copy()
    ptm = (q_pos - 1)[None].copy()
    out = _ws(q_pos, xm, ptm, _single_output_layer([(0, 0), (1, 0), (2, 0)], []))
    assert (out == 3).all()


# ---------------------------------------------------------------------------
# Paper's worked example (Sec. 4.2)
# ---------------------------------------------------------------------------

def test_worked_example_routed_equals_shared_form():
    ex = json.load(open(os.path.join(GOLDEN, "routed_example.json")))
    rng = np.random.default_rng(15)
    S = 16
    q_pos = np.array([Q12[s % 3] for s in range(S)], np.uint64)
    n_in = ex["n_in"]
    x = np.stack([rng.integers(0, q_pos) for _ in range(n_in * 2)]).reshape(n_in, 2, S).astype(np.uint64)
    names = sorted({r[1] for o in ex["outputs"] for r in o["raw"]})
    pt = np.stack([rng.integers(0, q_pos) for _ in names]).astype(np.uint64)
    gam = {"gamma1": 4321, "gamma2": 8765}
    pm_off, pm_in, pm_pt, grp_mem_off, mem_in, mem_sg, sc = [0], [], [], [0], [], [], []
    for o in ex["outputs"]:
        for i, nm in o["raw"]:
            pm_in.append(i)
            pm_pt.append(names.index(nm))
        pm_off.append(len(pm_in))
        for i, h in o["signed"]["members"]:
            mem_in.append(i)
            mem_sg.append(h)
        grp_mem_off.append(len(mem_in))
        sc.append(gam[o["signed"]["factor"]])
    d = dict(pm_off=np.array(pm_off, np.uint32), pm_input=np.array(pm_in, np.uint32),
             pm_pt=np.array(pm_pt, np.uint32), grp_off=np.array([0, 1, 2], np.uint32),
             grp_mem_off=np.array(grp_mem_off, np.uint32), mem_input=np.array(mem_in, np.uint32),
             mem_sign=np.array(mem_sg, np.int8), grp_scale=np.array([0, 1], np.uint32),
             scales=np.array(sc, np.uint64))
    out = _ws(q_pos, x, pt, d)
    # Eq. (shared-example): y1 = g1 U + g12 A2 + g14 A4, y2 = g2 U + g22 A2, U = A1 - A3
    for s in range(S):
        q = int(q_pos[s])
        for p in range(2):
            A = [int(x[i, p, s]) for i in range(4)]
            U = A[0] - A[2]
            P = {nm: int(pt[k, s]) for k, nm in enumerate(names)}
            y1 = gam["gamma1"] * U + P["g12"] * A[1] + P["g14"] * A[3]
            y2 = gam["gamma2"] * U + P["g22"] * A[1]
            assert int(out[0, p, s]) == y1 % q
            assert int(out[1, p, s]) == y2 % q


# ---------------------------------------------------------------------------
# CKKS meaning: decrypted output matches the float64 weighted sum
# ---------------------------------------------------------------------------

def test_toy_ckks_decode_matches_float64():
    lay = synth.make_layer(synth.CONFIGS["tiny"], 1)
    err, _, _ = ckks_toy.run_oracle(lay)
    assert err <= 1e-3, err
    assert err < 2e-4   # expected ~ sqrt(N) * 0.5 / 2^20 per raw term


def test_toy_ckks_detects_a_planted_sign_error():
    """The decode check has power: flip one member's sign in what the oracle
    evaluates (not in the float64 reference) and the error is far above 1e-3."""
    lay = synth.make_layer(synth.CONFIGS["tiny"], 1)
    toy, x, w, cts, pts, expected = ckks_toy.build_toy(lay)
    bad = synth.make_layer(synth.CONFIGS["tiny"], 1)
    m = int(np.nonzero(bad.mem_sign)[0][0])
    bad.mem_sign[m] = -bad.mem_sign[m]
    out = oracle.weighted_sum_layer(bad, cts, pts)
    dec = np.stack([toy.decrypt(out[j]) for j in range(bad.n_out)])
    assert ckks_toy.relative_error(dec, expected) > 1e-2


def test_toy_ckks_detects_a_transposed_plaintext():
    lay = synth.make_layer(synth.CONFIGS["tiny"], 1)
    toy, x, w, cts, pts, expected = ckks_toy.build_toy(lay)
    bad = synth.make_layer(synth.CONFIGS["tiny"], 1)
    bad.pm_pt[[0, 1]] = bad.pm_pt[[1, 0]]
    out = oracle.weighted_sum_layer(bad, cts, pts)
    dec = np.stack([toy.decrypt(out[j]) for j in range(bad.n_out)])
    assert ckks_toy.relative_error(dec, expected) > 1e-2
