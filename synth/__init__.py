"""Seeded synthetic inputs for the hybrid weighted sum.

This module is shared by the tests, the benchmark and the oracle's callers.  It
holds only input generation: the counter-based random generator, the choice of
RNS moduli, the synthetic layer structure (which terms are raw, which are
ternary, their signs and integer scales) and the uniform ciphertext/plaintext
residues.  It does none of the method's arithmetic: no products, no sums of
ciphertexts, no reductions of results.

Random generator (both this NumPy version and the HIP fill kernels in
``synth/csrc/synth_fill.hip`` implement exactly this definition):

* ``mix64`` is the SplitMix64 output function (Steele, Lea and Flood, "Fast
  splittable pseudorandom number generators", OOPSLA 2014, with the
  "Mix13"-style constants that SplitMix64 uses).
* ``key(seed, tag) = mix64(mix64(seed) + tag * GOLDEN)`` names one stream.
* ``u64(seed, tag, idx) = mix64(key(seed, tag) + (idx + 1) * GOLDEN)`` is the
  ``idx``-th output of SplitMix64 started at state ``key`` (all mod 2^64), so
  any element can be generated on its own (counter-based).
* A residue uniform in ``[0, q)`` is ``floor(u * q / 2^64)`` (bias < q/2^64).

Layer structure (a stand-in for the paper's packed linear layers, Sec. 4.2 and
Sec. 6.2, whose trained weights are not available):

* output ``j`` has ``T`` terms; term ``t`` reads input ciphertext ``t mod n_in``;
* the terms of an output form ``T / g`` blocks of ``g`` consecutive terms; a
  block is either raw (every term is one PMult by its own plaintext) or a
  ternary group: ``g`` signed terms that share one integer scale (the
  "grouping reconstruction operations" of Sec. 4.2);
* ``K = round(f * O * T / g)`` ternary groups in the whole layer, spread over
  outputs as evenly as possible; which blocks of an output are ternary is a
  seeded choice;
* signs are iid with P(+1) = P(-1) = 0.35, P(0) = 0.3, or, for the layers with
  cross-output sharing, drawn from a per-input-class pool of 16 sign vectors
  with an independent global flip (so equal and opposite signed sums recur,
  Sec. 4.2 "Sharing Signed Sums");
* scales are integers uniform in ``[1, 2^20)``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB

# Stream tags.  Each kind of random quantity has its own stream.
TAG_IN = 1        # input ciphertext coefficients
TAG_PT = 2        # raw-route plaintext coefficients
TAG_SIGN = 3      # iid member signs
TAG_SCALE = 4     # per-group integer scales
TAG_BLOCKSEL = 5  # which blocks of an output are ternary
TAG_POOL = 6      # sign vectors of a sharing pool
TAG_PICK = 7      # pool entry picked by a group
TAG_FLIP = 8      # global sign flip of a pooled group
TAG_SAMPLE = 9    # sampled positions for checks at full size
TAG_CT = 10        # stand-alone ciphertexts (e.g. the outputs a rescale receives)
TAG_KEY = 11       # rotation keys

SIGN_T1 = (35 << 64) // 100  # u < T1 -> +1
SIGN_T2 = (70 << 64) // 100  # T1 <= u < T2 -> -1, else 0
SCALE_BITS = 20


# ----------------------------------------------------------------------------
# Counter-based generator: scalar (Python int) and vector (NumPy uint64) forms
# ----------------------------------------------------------------------------

def mix64_int(z: int) -> int:
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX1) & MASK64
    z = ((z ^ (z >> 27)) * MIX2) & MASK64
    return z ^ (z >> 31)


def key_int(seed: int, tag: int) -> int:
    return mix64_int((mix64_int(seed) + tag * GOLDEN) & MASK64)


def u64_int(seed: int, tag: int, idx: int) -> int:
    return mix64_int((key_int(seed, tag) + (idx + 1) * GOLDEN) & MASK64)


def _mix64_np(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> np.uint64(30))
    z = z * np.uint64(MIX1)
    z = z ^ (z >> np.uint64(27))
    z = z * np.uint64(MIX2)
    return z ^ (z >> np.uint64(31))


def u64_np(seed: int, tag: int, idx) -> np.ndarray:
    """Vector form of ``u64_int`` over an array of indices."""
    idx = np.asarray(idx, dtype=np.uint64)
    with np.errstate(over="ignore"):
        state = np.uint64(key_int(seed, tag)) + (idx + np.uint64(1)) * np.uint64(GOLDEN)
        return _mix64_np(state)


def mulhi64_np(a: np.ndarray, b) -> np.ndarray:
    """floor(a * b / 2^64) for uint64 arrays (b may be a scalar or an array)."""
    a = np.asarray(a, dtype=np.uint64)
    b = np.asarray(b, dtype=np.uint64)
    m32 = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    a0, a1 = a & m32, a >> s32
    b0, b1 = b & m32, b >> s32
    with np.errstate(over="ignore"):
        p00 = a0 * b0
        p01 = a0 * b1
        p10 = a1 * b0
        p11 = a1 * b1
        mid = (p00 >> s32) + (p01 & m32) + (p10 & m32)
        return p11 + (p01 >> s32) + (p10 >> s32) + (mid >> s32)


def uniform_mod_np(seed: int, tag: int, idx, q) -> np.ndarray:
    """Residues uniform in [0, q) for the given flat indices (q per index or scalar)."""
    return mulhi64_np(u64_np(seed, tag, idx), q)


def uniform_mod_int(seed: int, tag: int, idx: int, q: int) -> int:
    return (u64_int(seed, tag, idx) * q) >> 64


def signs_from_u64(u: np.ndarray) -> np.ndarray:
    u = np.asarray(u, dtype=np.uint64)
    out = np.zeros(u.shape, dtype=np.int8)
    out[u < np.uint64(SIGN_T1)] = 1
    out[(u >= np.uint64(SIGN_T1)) & (u < np.uint64(SIGN_T2))] = -1
    return out


# ----------------------------------------------------------------------------
# RNS moduli
# ----------------------------------------------------------------------------

_MR_BASES = (2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37)


def is_probable_prime(n: int) -> bool:
    """Deterministic Miller-Rabin, exact for n < 3.3e24 with these bases."""
    if n < 2:
        return False
    for p in _MR_BASES:
        if n % p == 0:
            return n == p
    d, s = n - 1, 0
    while d % 2 == 0:
        d //= 2
        s += 1
    for a in _MR_BASES:
        x = pow(a, d, n)
        if x in (1, n - 1):
            continue
        for _ in range(s - 1):
            x = x * x % n
            if x == n - 1:
                break
        else:
            return False
    return True


def ntt_primes(N: int, L: int, bits: int = 50) -> list:
    """The first L primes q < 2^bits with q = 1 (mod 2N), searched downwards.

    q = m * 2N + 1 with m descending from floor((2^bits - 2) / 2N), so the list
    for a given N is the same for every L (a shorter list is a prefix).
    """
    step = 2 * N
    m = ((1 << bits) - 2) // step
    out = []
    while len(out) < L:
        if m <= 0:
            raise ValueError("not enough primes below 2^%d for N=%d" % (bits, N))
        q = m * step + 1
        if is_probable_prime(q):
            out.append(q)
        m -= 1
    return out


# ----------------------------------------------------------------------------
# Layer configurations
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    N: int
    L: int
    n_in: int
    n_out: int
    T: int                 # terms per output
    g: int                 # members per ternary group
    ternary: float         # fraction of all (output, term) pairs that are ternary
    n_groups: Optional[int] = None   # explicit K, overrides the fraction
    pool: int = 0          # 0 = iid signs; S > 0 = sharing pool of S sign vectors per input class
    chunks_hybrid: int = 1
    chunks_allpm: int = 1
    description: str = ""

    @property
    def K(self) -> int:
        if self.n_groups is not None:
            return self.n_groups
        return int(round(self.ternary * self.n_out * self.T / self.g))

    @property
    def ct_terms(self) -> int:
        return self.n_out * self.T


CONFIGS = {
    "tiny": LayerConfig(
        "tiny", N=1 << 12, L=3, n_in=64, n_out=1, T=64, g=8, ternary=0.5, n_groups=4,
        description="N=2^12, L=3, 64 inputs, 1 output; 32 PMult terms, 32 ternary terms in 4 groups of 8"),
    "vgg11": LayerConfig(
        "vgg11", N=1 << 16, L=8, n_in=64, n_out=128, T=64, g=8, ternary=0.53,
        description="VGG11-like conv layer: N=2^16, L=8, 64 inputs, 128 outputs x 64 terms, 53% ternary in groups of 8"),
    "vit768": LayerConfig(
        "vit768", N=1 << 16, L=10, n_in=24, n_out=24, T=768, g=16, ternary=0.65, pool=16,
        description="ViT-Base 768x768 diagonal-packed projection: N=2^16, L=10, 24 baby-step inputs, "
                    "24 outputs x 768 terms, 65% ternary in groups of 16, shared signed sums"),
    "bert_ffn": LayerConfig(
        "bert_ffn", N=1 << 16, L=12, n_in=32, n_out=96, T=768, g=16, ternary=0.795, chunks_allpm=4,
        description="BERT-Base FFN up-projection 768x3072: N=2^16, L=12, 32 inputs, 96 outputs x 768 terms, "
                    "79.5% ternary in groups of 16"),
    "large4096": LayerConfig(
        "large4096", N=1 << 16, L=16, n_in=128, n_out=128, T=4096, g=32, ternary=0.70, pool=16,
        chunks_hybrid=16, chunks_allpm=32,
        description="4096x4096 diagonal-packed matmul: N=2^16, L=16, 128 inputs, 128 outputs x 4096 terms, "
                    "70% ternary in groups of 32, heavy cross-output sharing"),
}


# ----------------------------------------------------------------------------
# Layer structure
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Layer:
    """Raw per-(output, term) description of one layer (or one chunk of outputs).

    Raw route (one PMult per term), per output CSR:
      pm_off[n_out+1], pm_input[P], pm_pt[P]  (pm_pt indexes this layer's pt table)
    Signed route, per output CSR over groups and per group CSR over members:
      grp_off[n_out+1], grp_mem_off[K+1], mem_input[M], mem_sign[M] (int8 in {-1,0,1}),
      grp_scale[K] (index into ``scales``), scales[n_scale] (uint64 integers)
    ``pt_global[n_pt]`` is the global plaintext id of each local plaintext (it
    selects the generator stream positions, so chunks see the same values).
    ``pt_const`` (all-PMult layers only): per local plaintext either -1 (uniform
    random plaintext, id pt_global) or a constant plaintext (sign, scale) packed
    as sign_code * 2^32 + scale with sign_code 1 for +1 and 2 for -1, 0 for 0.
    """
    cfg: LayerConfig
    moduli: list
    seed: int
    n_in: int
    n_out: int
    out_global: np.ndarray
    pm_off: np.ndarray
    pm_input: np.ndarray
    pm_pt: np.ndarray
    grp_off: np.ndarray
    grp_mem_off: np.ndarray
    mem_input: np.ndarray
    mem_sign: np.ndarray
    grp_scale: np.ndarray
    scales: np.ndarray
    pt_global: np.ndarray
    pt_const: Optional[np.ndarray] = None

    @property
    def N(self):
        return self.cfg.N

    @property
    def L(self):
        return self.cfg.L

    @property
    def n_pt(self):
        return int(self.pt_global.shape[0])

    @property
    def n_pm(self):
        return int(self.pm_off[-1])

    @property
    def n_group(self):
        return int(self.grp_off[-1])

    @property
    def n_member(self):
        return int(self.grp_mem_off[-1])

    @property
    def ct_terms(self):
        return self.n_pm + self.n_member


def _ternary_blocks(cfg: LayerConfig, seed: int):
    """Per output, the sorted list of block indices that are ternary."""
    B = cfg.T // cfg.g
    K = cfg.K
    O = cfg.n_out
    if cfg.T % cfg.g != 0:
        raise ValueError("T must be a multiple of g")
    if K > O * B:
        raise ValueError("more ternary groups than blocks")
    base, extra = divmod(K, O)
    keys = u64_np(seed, TAG_BLOCKSEL, np.arange(O * B, dtype=np.uint64)).reshape(O, B)
    out = []
    for j in range(O):
        kj = base + (1 if j < extra else 0)
        if kj > B:
            raise ValueError("output %d would need %d ternary blocks of %d" % (j, kj, B))
        order = np.argsort(keys[j], kind="stable")
        out.append(np.sort(order[:kj]))
    return out


def make_layer(cfg: LayerConfig, seed: int = 1, moduli: Optional[list] = None) -> Layer:
    """Build the raw description of the whole layer (all outputs)."""
    if moduli is None:
        moduli = ntt_primes(cfg.N, cfg.L)
    O, T, g, n_in = cfg.n_out, cfg.T, cfg.g, cfg.n_in
    B = T // g
    tern = _ternary_blocks(cfg, seed)

    # pool classes: block b starts at input (b*g) mod n_in
    starts = sorted({(b * g) % n_in for b in range(B)})
    class_of_start = {s: c for c, s in enumerate(starts)}
    S = cfg.pool
    if S:
        pool_idx = np.arange(len(starts) * S * g, dtype=np.uint64)
        pool = signs_from_u64(u64_np(seed, TAG_POOL, pool_idx)).reshape(len(starts), S, g)

    pm_off = np.zeros(O + 1, dtype=np.uint32)
    grp_off = np.zeros(O + 1, dtype=np.uint32)
    pm_input, pm_pt = [], []
    grp_mem_off = [0]
    mem_input, mem_sign = [], []
    n_pt = 0
    k_group = 0
    m_global = 0
    for j in range(O):
        tset = set(int(b) for b in tern[j])
        for b in range(B):
            terms = np.arange(b * g, (b + 1) * g)
            inputs = terms % n_in
            if b in tset:
                if S:
                    c = class_of_start[(b * g) % n_in]
                    pick = int(mulhi64_np(u64_np(seed, TAG_PICK, [k_group]), S)[0])
                    flip = int(u64_np(seed, TAG_FLIP, [k_group])[0] >> np.uint64(63))
                    sg = pool[c, pick].copy()
                    if flip:
                        sg = -sg
                else:
                    sg = signs_from_u64(u64_np(seed, TAG_SIGN, np.arange(m_global, m_global + g, dtype=np.uint64)))
                mem_input.append(inputs.astype(np.uint32))
                mem_sign.append(sg.astype(np.int8))
                m_global += g
                grp_mem_off.append(m_global)
                k_group += 1
            else:
                pm_input.append(inputs.astype(np.uint32))
                pm_pt.append(np.arange(n_pt, n_pt + g, dtype=np.uint32))
                n_pt += g
        pm_off[j + 1] = n_pt
        grp_off[j + 1] = k_group
    assert k_group == cfg.K
    scales = (np.uint64(1) + mulhi64_np(u64_np(seed, TAG_SCALE, np.arange(k_group, dtype=np.uint64)),
                                        np.uint64((1 << SCALE_BITS) - 1))).astype(np.uint64)
    cat32 = lambda xs: np.concatenate(xs).astype(np.uint32) if xs else np.zeros(0, np.uint32)
    return Layer(
        cfg=cfg, moduli=list(moduli), seed=seed, n_in=n_in, n_out=O,
        out_global=np.arange(O, dtype=np.uint32),
        pm_off=pm_off, pm_input=cat32(pm_input), pm_pt=cat32(pm_pt),
        grp_off=grp_off, grp_mem_off=np.asarray(grp_mem_off, dtype=np.uint32),
        mem_input=cat32(mem_input),
        mem_sign=np.concatenate(mem_sign).astype(np.int8) if mem_sign else np.zeros(0, np.int8),
        grp_scale=np.arange(k_group, dtype=np.uint32), scales=scales,
        pt_global=np.arange(n_pt, dtype=np.uint64))


def chunk_layer(layer: Layer, j0: int, j1: int) -> Layer:
    """The sub-layer of outputs [j0, j1): same inputs, its own pt table, scales and members."""
    p0, p1 = int(layer.pm_off[j0]), int(layer.pm_off[j1])
    g0, g1 = int(layer.grp_off[j0]), int(layer.grp_off[j1])
    m0, m1 = int(layer.grp_mem_off[g0]), int(layer.grp_mem_off[g1])
    pts = layer.pm_pt[p0:p1]
    pt_lo = int(pts.min()) if pts.size else 0
    if pts.size and int(pts.max()) - pt_lo + 1 != pts.size:
        raise ValueError("chunk plaintexts are not contiguous")
    pt_const = None
    if layer.pt_const is not None:
        pt_const = layer.pt_const[pt_lo:pt_lo + pts.size].copy()
    return Layer(
        cfg=layer.cfg, moduli=layer.moduli, seed=layer.seed, n_in=layer.n_in, n_out=j1 - j0,
        out_global=layer.out_global[j0:j1].copy(),
        pm_off=(layer.pm_off[j0:j1 + 1] - p0).astype(np.uint32),
        pm_input=layer.pm_input[p0:p1].copy(),
        pm_pt=(pts - pt_lo).astype(np.uint32),
        grp_off=(layer.grp_off[j0:j1 + 1] - g0).astype(np.uint32),
        grp_mem_off=(layer.grp_mem_off[g0:g1 + 1] - m0).astype(np.uint32),
        mem_input=layer.mem_input[m0:m1].copy(), mem_sign=layer.mem_sign[m0:m1].copy(),
        grp_scale=(layer.grp_scale[g0:g1] - g0).astype(np.uint32) if g1 > g0 else np.zeros(0, np.uint32),
        scales=layer.scales[g0:g1].copy(),
        pt_global=layer.pt_global[pt_lo:pt_lo + pts.size].copy(), pt_const=pt_const)


def all_pmult_layer(layer: Layer) -> Layer:
    """The same layer with every signed term turned into a PMult.

    A signed term with sign h and group scale c becomes a PMult by the constant
    plaintext whose every NTT-domain coefficient is h*c mod q (the constant
    polynomial h*c has a constant negacyclic NTT).  Raw terms keep their
    plaintexts.  Every term gets its own plaintext, in (output, term) order.
    """
    O = layer.n_out
    pm_off = np.zeros(O + 1, dtype=np.uint32)
    ins, consts, glob = [], [], []
    for j in range(O):
        count = 0
        a, b = int(layer.pm_off[j]), int(layer.pm_off[j + 1])
        ins.append(layer.pm_input[a:b])
        consts.append(np.full(b - a, -1, dtype=np.int64))
        glob.append(layer.pt_global[layer.pm_pt[a:b]].astype(np.uint64))
        count += b - a
        for gi in range(int(layer.grp_off[j]), int(layer.grp_off[j + 1])):
            m0, m1 = int(layer.grp_mem_off[gi]), int(layer.grp_mem_off[gi + 1])
            c = int(layer.scales[layer.grp_scale[gi]])
            sg = layer.mem_sign[m0:m1].astype(np.int64)
            code = np.where(sg > 0, 1, np.where(sg < 0, 2, 0)).astype(np.int64)
            ins.append(layer.mem_input[m0:m1])
            consts.append(code * (1 << 32) + c)
            glob.append(np.zeros(m1 - m0, dtype=np.uint64))
            count += m1 - m0
        pm_off[j + 1] = pm_off[j] + count
    pm_input = np.concatenate(ins).astype(np.uint32)
    n = pm_input.size
    assert int(pm_off[-1]) == n
    return Layer(
        cfg=layer.cfg, moduli=layer.moduli, seed=layer.seed, n_in=layer.n_in, n_out=O,
        out_global=layer.out_global.copy(), pm_off=pm_off, pm_input=pm_input,
        pm_pt=np.arange(n, dtype=np.uint32),
        grp_off=np.zeros(O + 1, dtype=np.uint32), grp_mem_off=np.zeros(1, dtype=np.uint32),
        mem_input=np.zeros(0, np.uint32), mem_sign=np.zeros(0, np.int8),
        grp_scale=np.zeros(0, np.uint32), scales=np.zeros(0, np.uint64),
        pt_global=np.concatenate(glob).astype(np.uint64), pt_const=np.concatenate(consts).astype(np.int64))


def output_chunks(n_out: int, n_chunks: int):
    """Split [0, n_out) into n_chunks contiguous ranges of near-equal size."""
    base, extra = divmod(n_out, n_chunks)
    out, j = [], 0
    for c in range(n_chunks):
        k = base + (1 if c < extra else 0)
        out.append((j, j + k))
        j += k
    return out


# ----------------------------------------------------------------------------
# Residues: inputs and plaintexts
# ----------------------------------------------------------------------------

def input_values(layer: Layer, positions=None) -> np.ndarray:
    """Input ciphertext coefficients.

    positions=None: the full limb-major array [n_in][2][L][N].
    positions = (limbs, coeffs) arrays of equal length S: array [n_in][2][S].
    """
    N, L, seed = layer.N, layer.L, layer.seed
    q = np.asarray(layer.moduli, dtype=np.uint64)
    if positions is None:
        i = np.arange(layer.n_in * 2 * L * N, dtype=np.uint64)
        limb = (i // np.uint64(N)) % np.uint64(L)
        return uniform_mod_np(seed, TAG_IN, i, q[limb]).reshape(layer.n_in, 2, L, N)
    limbs, coeffs = (np.asarray(a, dtype=np.uint64) for a in positions)
    ip = np.arange(layer.n_in * 2, dtype=np.uint64)[:, None]
    idx = (ip * np.uint64(L) + limbs[None, :]) * np.uint64(N) + coeffs[None, :]
    return uniform_mod_np(seed, TAG_IN, idx, q[limbs][None, :]).reshape(layer.n_in, 2, -1)


def pt_values(layer: Layer, positions=None, pt_ids=None) -> np.ndarray:
    """Plaintext coefficients of this layer's pt table.

    positions=None: [n_pt][L][N]; else positions = (limbs, coeffs) -> [n_pt][S].
    pt_ids restricts to those local plaintext ids.
    """
    N, L, seed = layer.N, layer.L, layer.seed
    q = np.asarray(layer.moduli, dtype=np.uint64)
    ids = np.arange(layer.n_pt) if pt_ids is None else np.asarray(pt_ids)
    glob = layer.pt_global[ids].astype(np.uint64)
    if positions is None:
        limbs = np.repeat(np.arange(L, dtype=np.uint64), N)
        coeffs = np.tile(np.arange(N, dtype=np.uint64), L)
    else:
        limbs, coeffs = (np.asarray(a, dtype=np.uint64) for a in positions)
    idx = (glob[:, None] * np.uint64(L) + limbs[None, :]) * np.uint64(N) + coeffs[None, :]
    vals = uniform_mod_np(seed, TAG_PT, idx, q[limbs][None, :])
    if layer.pt_const is not None:
        pc = layer.pt_const[ids]
        const = pc >= 0
        if const.any():
            code = (pc[const] >> 32)
            c = (pc[const] & 0xFFFFFFFF).astype(np.uint64)
            qq = q[limbs][None, :]
            cm = c[:, None] % qq
            v = np.where(code[:, None] == 1, cm, np.where(code[:, None] == 2, (qq - cm) % qq, np.uint64(0)))
            vals[const] = v.astype(np.uint64)
    if positions is None:
        return vals.reshape(len(ids), L, N)
    return vals


def sample_positions(N: int, L: int, count: int, seed: int):
    """Seeded sample of (limb, coeff) positions, always including tile edges."""
    limbs = [0, L - 1, 0, L - 1, L // 2, L // 2]
    coeffs = [0, N - 1, min(63, N - 1), max(0, N - 64), min(64, N - 1), N // 2]
    r = u64_np(seed, TAG_SAMPLE, np.arange(2 * count, dtype=np.uint64))
    limbs += list((mulhi64_np(r[:count], L)).astype(np.int64))
    coeffs += list((mulhi64_np(r[count:], N)).astype(np.int64))
    return np.asarray(limbs, dtype=np.int64), np.asarray(coeffs, dtype=np.int64)


def algorithmic_bytes(layer: Layer) -> int:
    """Bytes the path must move once: inputs, plaintexts and outputs (8 B words)."""
    return 8 * layer.L * layer.N * (2 * layer.n_in + layer.n_pm + 2 * layer.n_out)
