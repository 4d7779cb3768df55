"""Parity of the library's kernel-to-bubble packer (enc_schedule_kernels, host
code) with the packing oracle: identical intervals and start offsets on seeded
random timelines, the exhaustive-enumeration pin applied to the library
directly, and the documented argument errors."""

import ctypes
import random

import pytest

from oracle import schedule as S
from paper_2408_03505_amd import binding as B


def _lib_pack(kus, comm, ius, bub):
    where, off, _ = B.enc_schedule_kernels(kus, ius, bub, comm)
    return where, off


def test_library_matches_oracle_on_random_timelines():
    rng = random.Random(2408)
    for case in range(2000):
        n, m = rng.randint(0, 40), rng.randint(0, 60)
        kus = [rng.choice([0.0, rng.uniform(1, 400), rng.uniform(1, 60)]) for _ in range(n)]
        comm = [rng.random() < 0.15 for _ in range(n)]
        ius = [rng.choice([rng.uniform(100, 500), rng.uniform(0, 3000), 0.0]) for _ in range(m)]
        bub = [rng.random() < 0.6 for _ in range(m)]
        want = S.schedule_kernels(kus, comm, ius, bub)
        got = _lib_pack(kus, comm, ius, bub)
        assert got == want, case


def test_library_passes_the_enumeration_pin():
    from test_schedule_pins import _check_against_brute_force, _random_case
    rng = random.Random(7)
    for _ in range(1000):
        _check_against_brute_force(_lib_pack, *_random_case(rng))


def test_return_value_counts_placed_kernels():
    assert B.enc_schedule_kernels([1, 9, 1], [5, 5], [1, 1])[2] == 1
    assert B.enc_schedule_kernels([], [5], [1])[2] == 0


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), -1.0])
def test_bad_durations_are_rejected(bad):
    with pytest.raises(B.EncError) as e:
        B.enc_schedule_kernels([1.0, bad], [5.0], [1])
    assert e.value.status == B.ENC_ERR_INVALID
    with pytest.raises(B.EncError) as e:
        B.enc_schedule_kernels([1.0], [bad], [1])
    assert e.value.status == B.ENC_ERR_INVALID


def test_null_arrays_and_negative_counts_are_rejected():
    L = B.lib()
    out = (ctypes.c_int * 2)()
    k = (ctypes.c_double * 2)(1.0, 2.0)
    assert L.enc_schedule_kernels(None, None, 2, None, None, 0, ctypes.cast(out, ctypes.c_void_p), None) \
        == B.ENC_ERR_INVALID
    assert L.enc_schedule_kernels(ctypes.cast(k, ctypes.c_void_p), None, -1, None, None, 0, None, None) \
        == B.ENC_ERR_INVALID
    assert L.enc_schedule_kernels(ctypes.cast(k, ctypes.c_void_p), None, 2, None, None, 3,
                                  ctypes.cast(out, ctypes.c_void_p), None) == B.ENC_ERR_INVALID
    assert b"interval_us" in L.enc_last_error()
