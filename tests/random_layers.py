"""Seeded random layer descriptions for the plan compiler and GPU parity tests.

Unlike synth.make_layer (the configurations' block structure: term t reads
input t mod n_in), these layers draw every term and group member at random:
repeated inputs, empty outputs, empty groups, groups of one, all-zero signs,
groups that repeat an earlier one (equal or with every sign reversed, so that
whole-sum sharing applies), a few hot input pairs that many groups contain
(so that common partial sums are found), plaintexts used by several terms,
more inputs than one tile's LDS holds (input passes), and moduli near both
ends of the accepted range.
"""
import numpy as np

import synth
import paper_2609_35352_amd as fiona

FLAG_CHOICES = [0, 0, 0, fiona.FIONA_PLAN_NO_SHARING, fiona.FIONA_PLAN_NO_LDS_SUMS,
                fiona.FIONA_PLAN_NO_PARTIAL_SHARING, fiona.FIONA_PLAN_PER_CONTRIBUTION,
                fiona.FIONA_PLAN_NO_OUTPUT_BURSTS, fiona.FIONA_PLAN_CHECK_INPUTS]


def _moduli(rng, L):
    """L distinct moduli in (2^20, 2^50): some NTT primes, one just above 2^20,
    one just below 2^50 (the weighted sum needs neither primality nor q = 1 mod 2N)."""
    pool = list(synth.ntt_primes(1 << 8, 3)) + [(1 << 20) + 7, (1 << 50) - 27, (1 << 35) + 53]
    pick = rng.choice(len(pool), size=L, replace=False)
    return [int(pool[i]) for i in pick]


def random_layer(seed: int) -> synth.Layer:
    rng = np.random.default_rng(seed)
    N = int(rng.choice([1, 7, 64, 65, 130, 200]))
    L = int(rng.integers(1, 4))
    n_in = int(rng.choice([1, 3, 17, 64, 159, 160, 230, 300]))
    shape = rng.choice(["mixed", "mixed", "long", "wide"])
    # long: few outputs with many terms (split over wavefronts); wide: many
    # short outputs (output bursts in several rounds)
    n_out = int(rng.choice({"mixed": [1, 2, 9, 33], "long": [1, 2, 3], "wide": [70, 150]}[shape]))
    max_raw, max_grp = {"mixed": (40, 7), "long": (3000, 60), "wide": (6, 3)}[shape]
    n_scale = int(rng.integers(1, 9))
    scales = rng.integers(1, 1 << synth.SCALE_BITS, size=n_scale, dtype=np.uint64)
    scales[0] = 1
    if n_scale > 1:
        scales[-1] = (1 << synth.SCALE_BITS) - 1
    n_pt_pool = int(rng.integers(1, 120 if shape != "long" else 4000))
    hot = [tuple(rng.choice(n_in, size=2, replace=n_in < 2)) for _ in range(2)]
    pm_off, grp_off, grp_mem_off = [0], [0], [0]
    pm_input, pm_pt, mem_input, mem_sign, grp_scale = [], [], [], [], []
    groups = []   # (inputs, signs) of every group so far
    for _ in range(n_out):
        kind = rng.random()
        n_raw = 0 if kind < 0.1 else int(rng.integers(0, max_raw))
        n_grp = 0 if kind < 0.15 else int(rng.integers(0, max_grp))
        for _ in range(n_raw):
            pm_input.append(int(rng.integers(0, n_in)))
            pm_pt.append(int(rng.integers(0, n_pt_pool)))
        for _ in range(n_grp):
            r = rng.random()
            if groups and r < 0.25:   # repeat an earlier group, maybe reversed
                ins, sg = groups[int(rng.integers(0, len(groups)))]
                sg = sg if rng.random() < 0.5 else -sg
            else:
                size = int(rng.choice([0, 1, 2, 5, 16, 33, 60]))
                ins = rng.integers(0, n_in, size=size)
                sg = rng.integers(-1, 2, size=size)
                if r < 0.35:
                    sg = np.zeros(size, dtype=np.int64)
                if size >= 2 and r > 0.45:   # a hot pair, same relative sign each time
                    a, b = hot[int(rng.integers(0, 2))]
                    ins = ins.copy()
                    ins[0], ins[1] = a, b
                    sg = sg.copy()
                    sg[0], sg[1] = 1, -1
            groups.append((np.asarray(ins), np.asarray(sg)))
            mem_input.extend(int(v) for v in ins)
            mem_sign.extend(int(v) for v in sg)
            grp_mem_off.append(len(mem_input))
            grp_scale.append(int(rng.integers(0, n_scale)))
        pm_off.append(len(pm_input))
        grp_off.append(len(grp_scale))
    used_pt = sorted(set(pm_pt))
    remap = {p: i for i, p in enumerate(used_pt)}
    u32 = lambda a: np.asarray(a, dtype=np.uint32)
    cfg = synth.LayerConfig("random%d" % seed, N=N, L=L, n_in=n_in, n_out=n_out, T=1, g=1, ternary=0.0)
    return synth.Layer(
        cfg=cfg, moduli=_moduli(rng, L), seed=1000 + seed, n_in=n_in, n_out=n_out,
        out_global=np.arange(n_out, dtype=np.uint32),
        pm_off=u32(pm_off), pm_input=u32(pm_input), pm_pt=u32([remap[p] for p in pm_pt]),
        grp_off=u32(grp_off), grp_mem_off=u32(grp_mem_off), mem_input=u32(mem_input),
        mem_sign=np.asarray(mem_sign, dtype=np.int8), grp_scale=u32(grp_scale), scales=scales,
        pt_global=np.asarray(used_pt, dtype=np.uint64))


def random_flags(seed: int):
    """Plan flags and plaintext pitch (0 packed, "hint" padded) for a seed."""
    rng = np.random.default_rng(10_000 + seed)
    return int(rng.choice(FLAG_CHOICES)), ("hint" if rng.random() < 0.5 else 0)
