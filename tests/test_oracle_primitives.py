"""Pins of the two hash primitives the oracle uses as library steps.

The known-answer vectors come from published sources (tests/golden, each file
names its source); the pure-Python XXH64 is a second implementation written
from the published algorithm, so a wrong library (or a wrong reading of the
algorithm on the GPU side later) cannot agree with both."""
import ast
import hashlib
import os

import numpy as np
import pytest

from oracle import taliesin_ref as ref
from tests.sha256_spec import sha256 as spec_sha256
from tests.xxh64_spec import xxh64 as spec_xxh64

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _kat(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield [p.strip() for p in line.split("|")]


def _spec_bytes(s):
    if s.startswith("REPEAT "):
        _, lit, cnt = s.split(" ")
        return ast.literal_eval(lit) * int(cnt)
    return ast.literal_eval(s)


def test_xxh64_known_answers():
    n = 0
    for data, seed, want in _kat("xxh64_kat.txt"):
        d = ast.literal_eval(data)
        assert ref.xxh64(d, int(seed)) == int(want, 16)
        assert spec_xxh64(d, int(seed)) == int(want, 16)
        n += 1
    assert n >= 6


def test_sha256_known_answers():
    n = 0
    for data, want in _kat("sha256_kat.txt"):
        d = _spec_bytes(data)
        assert hashlib.sha256(d).hexdigest() == want
        if len(d) < 10000:  # the pure-Python SHA-256 is slow
            assert spec_sha256(d).hex() == want
        n += 1
    assert n >= 4


def test_sha256_library_matches_spec_all_padding_lengths():
    # every padding case: lengths around the 55/56/64-byte boundaries, one to
    # three message blocks
    rng = np.random.default_rng(7)
    for n in list(range(0, 130)) + [183, 184, 191, 192, 200]:
        d = rng.integers(0, 256, n, dtype=np.uint8).tobytes()
        assert hashlib.sha256(d).digest() == spec_sha256(d), n


@pytest.mark.parametrize("seed", [0, 1, 63, 2**32 + 5, 2**64 - 1])
def test_xxh64_library_matches_spec_all_lengths(seed):
    # every tail path: 0..7 single bytes, a 4-byte word, 8-byte words, stripes
    rng = np.random.default_rng(seed % 1000)
    for n in list(range(0, 80)) + [127, 128, 129, 255, 256, 1024, 1031]:
        d = rng.integers(0, 256, n, dtype=np.uint8).tobytes()
        assert ref.xxh64(d, seed) == spec_xxh64(d, seed), n
