"""C-ABI checks that need no GPU: exported symbols, argument and plan
validation, and the plan compiler's grouping/sharing counts (host-only plans)."""
import ctypes
import json
import os
import re

import numpy as np
import pytest

import random_layers
import synth
import paper_2609_35352_amd as fiona

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")
HOST = fiona.FIONA_PLAN_HOST_ONLY

pytestmark = pytest.mark.skipif(not os.path.exists(fiona.LIB_PATH), reason="libfiona.so not built")


def _declared_functions(path):
    src = open(path).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(fiona_\w+)\s*\(", src, flags=re.M)))


def test_every_declared_symbol_is_exported():
    names = _declared_functions(os.path.join(ROOT, "include", "fiona.h"))
    assert set(names) >= {"fiona_ctx_create", "fiona_ctx_destroy", "fiona_plan_create", "fiona_plan_destroy",
                          "fiona_plan_stats", "fiona_hybrid_linear", "fiona_status_string"}
    lib = ctypes.CDLL(fiona.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_synth_library_exports():
    import synth.gpu
    if not os.path.exists(synth.gpu.LIB_PATH):
        pytest.skip("synth library not built")
    lib = ctypes.CDLL(synth.gpu.LIB_PATH)
    assert hasattr(lib, "synth_fill_uniform") and hasattr(lib, "synth_fill_pts")


def test_status_strings():
    L = fiona.lib()
    for code in range(-10, 1):
        assert L.fiona_status_string(code)
    assert L.fiona_status_string(0) == b"ok"


def test_ctx_validation():
    q = synth.ntt_primes(1 << 12, 2)
    fiona.Ctx(1 << 12, 2, q).close()
    for N, L, mods, status in [(0, 2, q, -3), (1 << 21, 2, q, -3), (4096, 0, q, -3), (4096, 65, q * 40, -3),
                               (4096, 2, [q[0], 1 << 50], -3), (4096, 2, [q[0], 1], -3)]:
        with pytest.raises(fiona.FionaError) as e:
            fiona.Ctx(N, L, mods)
        assert e.value.status == status
    h = ctypes.c_void_p()
    assert fiona.lib().fiona_ctx_create(16, 1, None, ctypes.byref(h)) == -1


def _small_layer(**kw):
    cfg = synth.LayerConfig("t", N=256, L=2, n_in=16, n_out=6, T=32, g=8, ternary=0.5, **kw)
    return synth.make_layer(cfg, 3, moduli=synth.ntt_primes(256, 2))


def _plan_args(layer):
    return dict(n_in=layer.n_in, n_out=layer.n_out, n_pt=layer.n_pt, n_scale=len(layer.scales),
                pm_off=layer.pm_off, pm_input=layer.pm_input, pm_pt=layer.pm_pt, grp_off=layer.grp_off,
                grp_mem_off=layer.grp_mem_off, mem_input=layer.mem_input, mem_sign=layer.mem_sign,
                grp_scale=layer.grp_scale)


def test_plan_validation_errors():
    lay = _small_layer()
    ctx = fiona.Ctx(lay.N, lay.L, lay.moduli)
    ok = _plan_args(lay)
    fiona.Plan(ctx, flags=HOST, **ok).close()
    bad_cases = []
    a = dict(ok); a["pm_input"] = ok["pm_input"].copy(); a["pm_input"][3] = lay.n_in; bad_cases.append(a)
    a = dict(ok); a["pm_pt"] = ok["pm_pt"].copy(); a["pm_pt"][0] = lay.n_pt; bad_cases.append(a)
    a = dict(ok); a["mem_input"] = ok["mem_input"].copy(); a["mem_input"][1] = 999; bad_cases.append(a)
    a = dict(ok); a["mem_sign"] = ok["mem_sign"].copy(); a["mem_sign"][2] = 2; bad_cases.append(a)
    a = dict(ok); a["grp_scale"] = ok["grp_scale"].copy(); a["grp_scale"][0] = len(lay.scales); bad_cases.append(a)
    a = dict(ok); a["pm_off"] = ok["pm_off"].copy(); a["pm_off"][2], a["pm_off"][3] = a["pm_off"][3], a["pm_off"][2]
    bad_cases.append(a)
    a = dict(ok); a["grp_mem_off"] = ok["grp_mem_off"].copy(); a["grp_mem_off"][0] = 1; bad_cases.append(a)
    for a in bad_cases:
        with pytest.raises(fiona.FionaError) as e:
            fiona.Plan(ctx, flags=HOST, **a)
        assert e.value.status == -2
    a = dict(ok); a["n_in"] = 0
    with pytest.raises(fiona.FionaError) as e:
        fiona.Plan(ctx, flags=HOST, **a)
    assert e.value.status == -1
    a = dict(ok); a["n_in"] = 65537   # beyond FIONA_MAX_LAYER_INPUTS
    with pytest.raises(fiona.FionaError) as e:
        fiona.Plan(ctx, flags=HOST, **a)
    assert e.value.status == -3


def test_plaintext_pitch_checks():
    """pt_pitch: 0 (packed) and anything >= L*N are accepted, a pitch below L*N is
    FIONA_ERR_ARG; the hint is L*N rounded up to 64 words plus 128."""
    lay = _small_layer()
    ctx = fiona.Ctx(lay.N, lay.L, lay.moduli)
    ln = lay.L * lay.N
    assert ctx.pt_pitch_hint() == (ln + 63) // 64 * 64 + 128
    assert fiona.lib().fiona_pt_pitch_hint(None) == 0
    for pitch in (0, ln, ln + 1, ctx.pt_pitch_hint()):
        fiona.Plan(ctx, flags=HOST, pt_pitch=pitch, **_plan_args(lay)).close()
    for pitch in (1, ln - 1):
        with pytest.raises(fiona.FionaError) as e:
            fiona.Plan(ctx, flags=HOST, pt_pitch=pitch, **_plan_args(lay))
        assert e.value.status == -1
    ctx2 = fiona.Ctx(1000, 3, synth.ntt_primes(1024, 3))
    assert ctx2.pt_pitch_hint() == 3008 + 128


def test_hybrid_linear_error_paths_without_device():
    lay = _small_layer()
    ctx = fiona.Ctx(lay.N, lay.L, lay.moduli)
    plan = fiona.Plan(ctx, flags=HOST, **_plan_args(lay))
    L = fiona.lib()
    assert L.fiona_hybrid_linear(None, None, None, None, None, None, None) == -1
    # host-only plan: refused before any pointer is used
    assert L.fiona_hybrid_linear(plan.handle, 8, 8, 8, 8, 16, None) == -8


def test_worked_example_counts():
    """Sec. 4.2: 7 PMults term by term, 5 after grouping, one Sub saved by sharing U = A1 - A3."""
    ex = json.load(open(os.path.join(GOLDEN, "routed_example.json")))
    pm_off, pm_in, pm_pt, gm_off, m_in, m_sg = [0], [], [], [0], [], []
    for o in ex["outputs"]:
        for i, _ in o["raw"]:
            pm_in.append(i)
            pm_pt.append(len(pm_pt))
        pm_off.append(len(pm_in))
        for i, h in o["signed"]["members"]:
            m_in.append(i)
            m_sg.append(h)
        gm_off.append(len(m_in))
    q = synth.ntt_primes(16, 1)
    ctx = fiona.Ctx(16, 1, q)
    args = dict(n_in=ex["n_in"], n_out=2, n_pt=len(pm_pt), n_scale=2, pm_off=pm_off, pm_input=pm_in, pm_pt=pm_pt,
                grp_off=[0, 1, 2], grp_mem_off=gm_off, mem_input=m_in, mem_sign=m_sg, grp_scale=[0, 1])
    st = fiona.Plan(ctx, flags=HOST, **args).stats()
    assert st["pmult_per_contribution"] == ex["pmult_per_contribution"] == 7
    assert st["pmult_grouped"] == ex["pmult_grouped"] == 5
    assert st["addsub_unshared"] - st["addsub_shared"] == ex["addsub_saved_by_sharing"] == 1
    assert st["n_sum_distinct"] == 1 and st["n_use"] == 2 and st["n_sum_resident"] == 1
    assert st["ct_terms"] == 8 and st["n_member_nonzero"] == 4
    st2 = fiona.Plan(ctx, flags=HOST | fiona.FIONA_PLAN_NO_SHARING, **args).stats()
    assert st2["n_sum_distinct"] == 2 and st2["addsub_shared"] == st2["addsub_unshared"] == 2
    assert st2["pmult_grouped"] == 5


def test_sharing_finds_opposite_sums():
    # output 0: A0 - A1 + A2 ; output 1: -A0 + A1 - A2 (all reversed) ; output 2: A2 + A1 - A0 (other order)
    q = synth.ntt_primes(16, 1)
    ctx = fiona.Ctx(16, 1, q)
    args = dict(n_in=3, n_out=3, n_pt=0, n_scale=3, pm_off=[0, 0, 0, 0], pm_input=[], pm_pt=[],
                grp_off=[0, 1, 2, 3], grp_mem_off=[0, 3, 6, 9], mem_input=[0, 1, 2, 0, 1, 2, 2, 1, 0],
                mem_sign=[1, -1, 1, -1, 1, -1, 1, -1, 1], grp_scale=[0, 1, 2])
    st = fiona.Plan(ctx, flags=HOST, **args).stats()
    # the third sum is A2 - A1 + A0 = the first one
    assert st["n_sum_distinct"] == 1 and st["n_use"] == 3
    assert st["addsub_unshared"] == 6 and st["addsub_shared"] == 2


def test_long_groups_are_split_and_zero_groups_dropped():
    q = synth.ntt_primes(16, 1)
    ctx = fiona.Ctx(16, 1, q)
    n = 150
    args = dict(n_in=150, n_out=2, n_pt=0, n_scale=2, pm_off=[0, 0, 0], pm_input=[], pm_pt=[],
                grp_off=[0, 1, 2], grp_mem_off=[0, n, n + 4], mem_input=list(range(n)) + [0, 1, 2, 3],
                mem_sign=[1] * n + [0, 0, 0, 0], grp_scale=[0, 1])
    st = fiona.Plan(ctx, flags=HOST, **args).stats()
    assert st["n_use"] == 4            # ceil(150 / 48) sub-sums; the all-zero group contributes nothing
    assert st["n_member_nonzero"] == 150 and st["n_member"] == 154
    assert st["pmult_grouped"] == 4 and st["pmult_per_contribution"] == 150


@pytest.mark.parametrize("name", ["vgg11", "vit768", "bert_ffn"])
def test_config_plans(name):
    lay = synth.make_layer(synth.CONFIGS[name], 1)
    ctx = fiona.Ctx(lay.N, lay.L, lay.moduli)
    st = fiona.Plan.from_layer(ctx, lay, flags=HOST).stats()
    assert st["ct_terms"] == lay.ct_terms and st["n_pmult"] == lay.n_pm
    assert st["pmult_grouped"] == lay.n_pm + st["n_use"]
    if name == "vit768":
        assert st["n_sum_distinct"] <= 48 and st["n_sum_resident"] == st["n_sum_distinct"]
    assert st["grid"] == lay.L * lay.N // 64
    assert st["lds_bytes"] == (lay.n_in + st["n_partial"] + st["n_sum_resident"] + st["segment_slots"] + 1
                               + st["output_buffer_rows"]) * 1024 <= 160 * 1024
    assert st["waves"] in (8, 16)
    # outputs in rounds that each fit the output buffer (bursts where outputs are at least
    # 2.5% of the bytes: VGG11's 6%, not ViT's or BERT's); without bursts, one round stored directly
    if name == "vgg11":
        assert st["output_rounds"] == 2 and st["output_buffer_rows"] == 64 and st["waves"] == 16
        assert st["output_rounds"] * st["output_buffer_rows"] >= lay.n_out - st["split_outputs"]
    else:
        assert st["output_rounds"] == 1 and st["output_buffer_rows"] == 0
    nb = fiona.Plan.from_layer(ctx, lay, flags=HOST | fiona.FIONA_PLAN_NO_OUTPUT_BURSTS).stats()
    assert nb["output_rounds"] == 1 and nb["output_buffer_rows"] == 0
    assert nb["lds_bytes"] == st["lds_bytes"] - st["output_buffer_rows"] * 1024


def test_output_rounds_split_evenly():
    """Consecutive outputs go to rounds of at most the free LDS rows; 150 outputs
    over 64 inputs (95 free rows) make two rounds of 75; 9 free rows force 17."""
    for n_in, n_out, rounds, rows in ((64, 150, 2, 75), (150, 150, 17, 9)):
        cfg = synth.LayerConfig("r", N=128, L=1, n_in=n_in, n_out=n_out, T=4, g=1, ternary=0.0)
        lay = synth.make_layer(cfg, 2, moduli=synth.ntt_primes(128, 1))
        ctx = fiona.Ctx(lay.N, lay.L, lay.moduli)
        st = fiona.Plan.from_layer(ctx, lay, flags=HOST).stats()
        assert (st["output_rounds"], st["output_buffer_rows"], st["waves"]) == (rounds, rows, 16)


def test_partial_sharing_finds_common_terms():
    """Sec. 4.2 candidate search: groups of one layer that only partly overlap
    share common signed pairs; the estimate k*m - m - k decides."""
    cfg = synth.LayerConfig("partial_share", N=256, L=2, n_in=16, n_out=48, T=96, g=12, ternary=0.95)
    lay = synth.make_layer(cfg, 5, moduli=synth.ntt_primes(256, 2))
    ctx = fiona.Ctx(lay.N, lay.L, lay.moduli)
    st = fiona.Plan.from_layer(ctx, lay, flags=HOST).stats()
    assert st["n_partial"] > 0 and st["partial_levels"] >= 2
    # one Add/Sub forms each common pair; every sum that holds it saves one
    assert st["addsub_partial"] < st["addsub_shared"] <= st["addsub_unshared"]
    assert st["lds_bytes"] == (lay.n_in + st["n_partial"] + st["n_sum_resident"] + st["segment_slots"] + 1
                               + st["output_buffer_rows"]) * 1024
    off = fiona.Plan.from_layer(ctx, lay, flags=HOST | fiona.FIONA_PLAN_NO_PARTIAL_SHARING).stats()
    assert off["n_partial"] == 0 and off["addsub_partial"] == off["addsub_shared"] == st["addsub_shared"]
    none = fiona.Plan.from_layer(ctx, lay, flags=HOST | fiona.FIONA_PLAN_NO_SHARING).stats()
    assert none["n_partial"] == 0 and none["n_sum_distinct"] == none["n_use"]


def test_partial_sharing_worked_pair():
    """Three sums over inputs 0..3 that all contain A0 - A1 (20 uses each, so
    k = 60): the pair is formed once, and each sum holds it as one member."""
    q = synth.ntt_primes(16, 1)
    ctx = fiona.Ctx(16, 1, q)
    groups = [([0, 1, 2], [1, -1, 1]), ([0, 1, 3], [-1, 1, 1]), ([0, 1, 2, 3], [1, -1, -1, 1])] * 20
    mem_in, mem_sg, gm = [], [], [0]
    for ins, sg in groups:
        mem_in += ins
        mem_sg += sg
        gm.append(len(mem_in))
    n_out = len(groups)
    args = dict(n_in=4, n_out=n_out, n_pt=0, n_scale=n_out, pm_off=[0] * (n_out + 1), pm_input=[], pm_pt=[],
                grp_off=list(range(n_out + 1)), grp_mem_off=gm, mem_input=mem_in, mem_sign=mem_sg,
                grp_scale=list(range(n_out)))
    st = fiona.Plan(ctx, flags=HOST | fiona.FIONA_PLAN_NO_LDS_SUMS, **args).stats()
    assert st["n_sum_distinct"] == 3 and st["n_partial"] >= 1
    # the three distinct sums need 2 + 2 + 3 Add/Sub; with A0 - A1 shared: 1 + 1 + 1 + 2 (+ 1 to form it)
    assert st["addsub_shared"] == 7 and st["addsub_partial"] <= 5


@pytest.mark.parametrize("name", ["vgg11", "bert_ffn"])
def test_ablation_plans(name):
    """Sec. 6.2 compilations on one layer: per-contribution applies a scalar
    product per nonzero signed term; grouping applies one per group (sub-sum);
    sharing and partial sharing only lower the Add/Sub count."""
    lay = synth.make_layer(synth.CONFIGS[name], 1)
    ctx = fiona.Ctx(lay.N, lay.L, lay.moduli)
    pc = fiona.Plan.from_layer(ctx, lay, flags=HOST | fiona.FIONA_PLAN_PER_CONTRIBUTION).stats()
    gr = fiona.Plan.from_layer(ctx, lay, flags=HOST | fiona.FIONA_PLAN_NO_SHARING).stats()
    sh = fiona.Plan.from_layer(ctx, lay, flags=HOST | fiona.FIONA_PLAN_NO_PARTIAL_SHARING).stats()
    pa = fiona.Plan.from_layer(ctx, lay, flags=HOST).stats()
    assert pc["n_use"] == pc["n_member_nonzero"] == pc["n_sum_distinct"]
    assert pc["pmult_grouped"] == pc["pmult_per_contribution"] and pc["addsub_partial"] == 0 and pc["n_partial"] == 0
    assert gr["n_use"] == sh["n_use"] == pa["n_use"] == lay.n_group   # no group here exceeds 48 members
    assert gr["pmult_grouped"] == lay.n_pm + lay.n_group < pc["pmult_grouped"]
    assert gr["addsub_partial"] == gr["addsub_unshared"] >= sh["addsub_partial"] >= pa["addsub_partial"]


def test_rescaler_validation_without_device():
    L = fiona.lib()
    L.fiona_rescaler_create.restype = ctypes.c_int
    L.fiona_rescaler_create.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32,
                                        ctypes.POINTER(ctypes.c_void_p)]
    h = ctypes.c_void_p()
    assert L.fiona_rescaler_create(None, None, 4, ctypes.byref(h)) == -1
    q3 = synth.ntt_primes(1 << 12, 3)
    ctx = fiona.Ctx(1 << 12, 3, q3)
    assert L.fiona_rescaler_create(ctx.handle, None, 0, ctypes.byref(h)) == -1          # no ciphertexts
    one = fiona.Ctx(1 << 12, 1, q3[:1])
    assert L.fiona_rescaler_create(one.handle, None, 4, ctypes.byref(h)) == -3          # nothing to drop
    small = fiona.Ctx(128, 2, synth.ntt_primes(128, 2))
    assert L.fiona_rescaler_create(small.handle, None, 4, ctypes.byref(h)) == -3        # N below 2^8
    odd = fiona.Ctx(1 << 12, 2, [q3[0], (1 << 40) + 15])                                 # not 1 mod 2N
    assert L.fiona_rescaler_create(odd.handle, None, 4, ctypes.byref(h)) == -3
    bad_psi = (ctypes.c_uint64 * 3)(2, 2, 2)                                             # not 2N-th roots
    assert L.fiona_rescaler_create(ctx.handle, ctypes.cast(bad_psi, ctypes.c_void_p), 4, ctypes.byref(h)) == -3
    L.fiona_rescale.restype = ctypes.c_int
    L.fiona_rescale.argtypes = [ctypes.c_void_p] * 2 + [ctypes.c_uint32] + [ctypes.c_void_p] * 2
    assert L.fiona_rescale(None, None, 1, None, None) == -1


def test_rotator_validation():
    """fiona_rotator_create checks its arguments before touching the device."""
    N, L = 256, 2
    ps = synth.ntt_primes(N, L + 1)
    ctx = fiona.Ctx(N, L, ps[:L])
    for P, max_rot, status in [(ps[L] + 2, 1, -3), (ps[0], 1, -3), (ps[L], 0, -1), (1 << 50, 1, -3),
                               (3, 1, -3), (ps[L], 257, -3)]:
        with pytest.raises(fiona.FionaError) as e:
            fiona.Rotator(ctx, P, max_rot)
        assert e.value.status == status
    small = fiona.Ctx(128, L, synth.ntt_primes(128, L))
    with pytest.raises(fiona.FionaError) as e:
        fiona.Rotator(small, synth.ntt_primes(128, L + 1)[L], 1)
    assert e.value.status == -3
    assert fiona.lib().fiona_rotation_key_words(None) == 0


def test_rescaler_size_limit():
    """fiona_rescaler_create rejects more ciphertexts than one launch can hold (before touching the device)."""
    N, L = 256, 2
    ctx = fiona.Ctx(N, L, synth.ntt_primes(N, L))
    with pytest.raises(fiona.FionaError) as e:
        fiona.Rescaler(ctx, 40000)
    assert e.value.status == -3


def test_partial_sharing_with_repeated_inputs():
    """A group may name the same input twice (a diagonal group wider than the
    baby steps).  Pairs of one input with itself are no sharing candidates,
    and taking a pair out of a sum removes exactly its two members: 32 groups
    {A0, A0, Ak, Ak+1} keep their 4 members each (3 Add/Sub per sum)."""
    q = synth.ntt_primes(16, 1)
    ctx = fiona.Ctx(16, 1, q)
    n_out = 32
    mem_in, gm = [], [0]
    for k in range(1, n_out + 1):
        mem_in += [0, 0, k, k + 1]
        gm.append(len(mem_in))
    args = dict(n_in=n_out + 2, n_out=n_out, n_pt=0, n_scale=n_out, pm_off=[0] * (n_out + 1), pm_input=[],
                pm_pt=[], grp_off=list(range(n_out + 1)), grp_mem_off=gm, mem_input=mem_in,
                mem_sign=[1] * len(mem_in), grp_scale=list(range(n_out)))
    st = fiona.Plan(ctx, flags=HOST | fiona.FIONA_PLAN_NO_LDS_SUMS, **args).stats()
    assert st["n_member_nonzero"] == 4 * n_out
    assert st["addsub_shared"] == 3 * n_out
    assert st["n_partial"] == 0 and st["addsub_partial"] == 3 * n_out


def test_checking_plan_preconditions_on_the_host():
    """A checking plan keeps the layer's signs: the signs a call passes must be
    the ones the plan was compiled from (Sec. 2.2, a plan fixed offline), scales
    below 2^20, inputs and plaintext words below 2^50."""
    layer = synth.make_layer(synth.LayerConfig("chk", N=64, L=2, n_in=6, n_out=3, T=12, g=3, ternary=0.5),
                             3, moduli=synth.ntt_primes(64, 2))
    ctx = fiona.Ctx(layer.N, layer.L, layer.moduli)
    plan = fiona.Plan.from_layer(ctx, layer, flags=HOST | fiona.FIONA_PLAN_CHECK_INPUTS)
    x, pt = synth.input_values(layer), synth.pt_values(layer)
    ok = fiona.plan_check_inputs
    assert ok(plan, layer.mem_sign, layer.scales, x, pt) == 0
    assert ok(plan, layer.mem_sign, layer.scales) == 0                     # signs and scales only
    nz = int(np.nonzero(layer.mem_sign)[0][0])
    for change in (lambda s: s.__setitem__(nz, -s[nz]), lambda s: s.__setitem__(nz, 0),
                   lambda s: s.__setitem__(int(np.nonzero(layer.mem_sign == 0)[0][0]), 1)):
        s2 = layer.mem_sign.copy()
        change(s2)
        assert ok(plan, s2, layer.scales, x, pt) == fiona.FIONA_ERR_PRECONDITION
    sc = layer.scales.copy()
    sc[-1] = 1 << 20
    assert ok(plan, layer.mem_sign, sc) == fiona.FIONA_ERR_PRECONDITION
    x2 = x.copy()
    x2[1, 1, 1, 5] = np.uint64(1 << 50)
    assert ok(plan, layer.mem_sign, layer.scales, x2, pt) == fiona.FIONA_ERR_PRECONDITION
    pt2 = pt.copy()
    pt2[-1, -1, -1] = np.uint64(2 ** 64 - 1)
    assert ok(plan, layer.mem_sign, layer.scales, x, pt2) == fiona.FIONA_ERR_PRECONDITION
    # a plan made without the flag keeps no signs
    plain = fiona.Plan.from_layer(ctx, layer, flags=HOST)
    assert ok(plain, layer.mem_sign, layer.scales) == fiona.FIONA_ERR_ARG


@pytest.mark.parametrize("n_in,passes", [(159, 1), (160, 2), (256, 2), (320, 3), (1000, 8)])
def test_input_passes(n_in, passes):
    """Layers with more inputs than one tile's LDS holds run in passes over
    input ranges of at most 128; every raw term and member lands in exactly
    one pass, and a group spanning ranges becomes one use per range."""
    cfg = synth.LayerConfig("wide", N=64, L=1, n_in=n_in, n_out=5, T=-(-2 * n_in // 16) * 16, g=16, ternary=0.6, pool=3)
    lay = synth.make_layer(cfg, 2, moduli=synth.ntt_primes(64, 1))
    ctx = fiona.Ctx(lay.N, lay.L, lay.moduli)
    st = fiona.Plan.from_layer(ctx, lay, flags=HOST).stats()
    assert st["input_passes"] == passes
    assert st["ct_terms"] == lay.ct_terms and st["n_pmult"] == lay.n_pm and st["n_member"] == lay.n_member
    assert st["lds_bytes"] <= 160 * 1024
    per = -(-n_in // passes)
    # uses: every group once per input range its nonzero members touch
    uses = 0
    for q in range(lay.n_group):
        m0, m1 = int(lay.grp_mem_off[q]), int(lay.grp_mem_off[q + 1])
        nz = lay.mem_input[m0:m1][lay.mem_sign[m0:m1] != 0]
        uses += len(set(int(i) // per for i in nz))
    assert st["n_use"] == uses


def test_input_passes_skip_unread_ranges():
    """Input ranges that no term reads get no pass (320 inputs, terms on the
    first 64 only: one pass)."""
    cfg = synth.LayerConfig("wide_sparse", N=100, L=2, n_in=320, n_out=5, T=64, g=8, ternary=0.5)
    lay = synth.make_layer(cfg, 5, moduli=synth.ntt_primes(128, 2))
    ctx = fiona.Ctx(lay.N, lay.L, lay.moduli)
    st = fiona.Plan.from_layer(ctx, lay, flags=HOST).stats()
    assert st["input_passes"] == 1 and st["ct_terms"] == lay.ct_terms


@pytest.mark.parametrize("seed", range(64))
def test_random_layer_plans(seed):
    """Random layer descriptions (random_layers.py) compile on the host under
    their flags; the counts match the description and the launch fits."""
    lay = random_layers.random_layer(seed)
    flags, _ = random_layers.random_flags(seed)
    ctx = fiona.Ctx(lay.N, lay.L, lay.moduli)
    st = fiona.Plan.from_layer(ctx, lay, flags=HOST | flags).stats()
    assert st["ct_terms"] == lay.ct_terms and st["n_pmult"] == lay.n_pm and st["n_member"] == lay.n_member
    nz = int(np.count_nonzero(lay.mem_sign))
    assert st["n_member_nonzero"] == nz and st["pmult_per_contribution"] == lay.n_pm + nz
    assert 1 <= st["input_passes"] <= max(1, -(-lay.n_in // 128))
    if lay.n_in <= 159:   # FIONA_MAX_INPUTS: one tile of every input in LDS
        assert st["input_passes"] == 1
    assert st["lds_bytes"] <= 160 * 1024 and st["waves"] in (8, 16)
    if flags & fiona.FIONA_PLAN_PER_CONTRIBUTION:
        assert st["pmult_grouped"] == st["pmult_per_contribution"]
