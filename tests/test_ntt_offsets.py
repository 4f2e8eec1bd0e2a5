"""Host replay of every memory access of the NTT passes (no device).

fiona_check_ntt_offsets lays a rescaler or rotator out at fake device
addresses, records one call's launches instead of issuing them, and
recomputes every global access of every workgroup and thread with the
kernels' own offset helpers.  Each access must fall inside the buffer that
holds its descriptor's base (the twiddle tables each on their own), offsets
must stay below 2^32 bytes, and every descriptor's end must be its buffer's
end.  Every fake buffer starts with bit 31 of its low address half set, and
the replay rebuilds each descriptor base from its two halves as the kernels
do (a signed low half would spill into the high half).

The shapes are those of the GPU tests and of bench.py: rings 2^8 .. 2^17,
L up to 16, several limbs per launch and one limb per launch, the shared
input order of pass A, the transposed outputs, 1 .. 256 rotations.
"""
import os

import pytest

import synth
import paper_2609_35352_amd as fiona

pytestmark = pytest.mark.skipif(not os.path.exists(fiona.LIB_PATH), reason="libfiona.so not built")

RESCALE = [  # N, L, max_ct, n_ct
    (256, 2, 3, 2), (1 << 12, 3, 4, 3), (1 << 13, 5, 3, 2), (1 << 11, 4, 2, 1), (1 << 17, 2, 2, 1),
    (256, 5, 16384, 3), (256, 5, 10000, 3), (256, 3, 32767, 32767), (1 << 12, 3, 1, 1),
    (1 << 16, 8, 4, 4), (1 << 16, 16, 4, 4), (1 << 16, 8, 128, 5),
    (1 << 16, 8, 128, 128), (1 << 16, 10, 24, 24), (1 << 16, 12, 96, 96), (1 << 16, 16, 128, 128),
]
ROTATE = [  # N, L, max_rot, n_rot
    (256, 1, 2, 2), (1024, 3, 3, 3), (1 << 12, 4, 4, 4), (2048, 10, 1, 1), (1 << 17, 2, 2, 2),
    (256, 2, 256, 256), (256, 2, 70, 70), (256, 2, 1, 1), (2048, 2, 1, 1),
    (1 << 16, 8, 63, 63), (1 << 16, 10, 23, 23), (1 << 16, 10, 3, 3), (1 << 16, 12, 31, 31),
    (1 << 16, 16, 127, 127), (1 << 16, 16, 4, 4),
]


@pytest.mark.parametrize("N,L,max_ct,n_ct", RESCALE)
def test_rescale_accesses_in_bounds(N, L, max_ct, n_ct):
    rc, msg = fiona.check_ntt_offsets("rescale", N, L, synth.ntt_primes(N, L), max_ct, n_ct)
    assert rc == 0, msg


@pytest.mark.parametrize("N,L,max_rot,n_rot", ROTATE)
def test_rotate_accesses_in_bounds(N, L, max_rot, n_rot):
    rc, msg = fiona.check_ntt_offsets("rotate", N, L, synth.ntt_primes(N, L + 1), max_rot, n_rot)
    assert rc == 0, msg


@pytest.mark.parametrize("op,N,L,cap,n", [("rescale", 256, 2, 3, 2), ("rescale", 1 << 16, 8, 128, 128),
                                           ("rotate", 256, 2, 2, 2), ("rotate", 1 << 16, 8, 63, 63)])
def test_replay_finds_an_overrun(op, N, L, cap, n):
    """The output buffer taken one word short: the replay reports the store
    that reaches past it (the last word of the output is written)."""
    mods = synth.ntt_primes(N, L if op == "rescale" else L + 1)
    rc, msg = fiona.check_ntt_offsets(op, N, L, mods, cap, n, out_shrink=8)
    assert rc == fiona.FIONA_ERR_BOUNDS and "out_cts" in msg and "bytes up to" in msg, msg


def test_replay_parameter_errors():
    q = synth.ntt_primes(256, 3)
    assert fiona.check_ntt_offsets("rescale", 256, 2, q, 2, 3)[0] == -1            # n_ct > max_ct
    assert fiona.check_ntt_offsets("rescale", 384, 2, q, 2, 1)[0] == -3            # N not a power of two
    assert fiona.check_ntt_offsets("rotate", 256, 2, q, 300, 1)[0] == -3           # max_rot > 256
