"""Philox4x32-10 against the Random123 known-answer vectors (SC'11 generator)."""
import numpy as np
import pytest

from oracle.philox import philox4x32_10, philox4x32_10_np
import synth

# (counter, key) -> output, from the Random123 distribution's kat_vectors.
KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,out", KAT)
def test_oracle_philox_kat(ctr, key, out):
    assert philox4x32_10(ctr, key) == out


@pytest.mark.parametrize("ctr,key,out", KAT)
def test_vectorised_philox_kat(ctr, key, out):
    res = philox4x32_10_np(*[np.array([c]) for c in ctr], *key)
    assert tuple(int(r[0]) for r in res) == out


@pytest.mark.parametrize("ctr,key,out", KAT)
def test_input_generator_philox_kat(ctr, key, out):
    assert synth.philox(ctr, key) == out


def test_vectorised_matches_scalar_on_many_counters():
    rng = np.random.default_rng(0)
    c = rng.integers(0, 2**32, size=(4, 64), dtype=np.uint64)
    vec = philox4x32_10_np(c[0], c[1], c[2], c[3], 0x1234, 0xABCDEF01)
    for i in range(64):
        assert tuple(int(v[i]) for v in vec) == philox4x32_10(tuple(int(x) for x in c[:, i]), (0x1234, 0xABCDEF01))
