"""Pins of the oracle's SHA-256 (FIPS 180-4) against the standard's published
example values and an independent library implementation (hashlib)."""
import hashlib
import os

import numpy as np
import pytest

import oracle


def _fips_vectors(golden_dir):
    out = []
    for line in open(os.path.join(golden_dir, "sha256_fips180_4.txt")):
        if line.startswith("#") or not line.strip():
            continue
        spec, dig = line.split()
        if spec == "empty":
            msg = b""
        elif spec.startswith("ascii:"):
            msg = spec[len("ascii:"):].encode()
        else:
            _, count, ch = spec.split(":")
            msg = ch.encode() * int(count)
        out.append((spec, msg, dig))
    return out


def test_fips_example_vectors(golden_dir):
    vecs = _fips_vectors(golden_dir)
    assert len(vecs) == 5
    for spec, msg, dig in vecs:
        assert oracle.sha256(msg).hex() == dig, spec


def test_constants_derived_from_primes_match_standard(golden_dir):
    k, h0 = oracle.sha256_constants()
    table = {}
    for line in open(os.path.join(golden_dir, "sha256_constants_fips180_4.txt")):
        if line.startswith("#") or not line.strip():
            continue
        name, *vals = line.split()
        table[name] = [int(v, 16) for v in vals]
    assert list(h0) == table["H0"]
    assert k[0] == table["K0"][0] and k[1] == table["K1"][0] and k[63] == table["K63"][0]
    assert len(set(k.tolist())) == 64


@pytest.mark.parametrize("length", list(range(0, 200)) + [447, 448, 511, 512, 1000, 4128])
def test_matches_hashlib_across_padding_boundaries(length):
    rng = np.random.default_rng(1000 + length)
    msg = rng.integers(0, 256, size=length, dtype=np.uint8).tobytes()
    assert oracle.sha256(msg) == hashlib.sha256(msg).digest()
