"""Pins of the oracle's Gaussian-noise generator (CPU only).

* Philox4x32-10 words against the known-answer vectors published with the
  generator (tests/golden/philox4x32_10_kat.json), and against rocRAND's
  independent implementation of it (its header-only engine, compiled here for
  the host) on many counters.
* The uniform mapping and Box-Muller transform against their definitions and
  the standard normal law (moments, Kolmogorov-Smirnov).
"""
import json
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest
from scipy import stats

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
KAT = os.path.join(HERE, "golden", "philox4x32_10_kat.json")


def _kat():
    return [([int(x, 16) for x in v["counter"]], [int(x, 16) for x in v["key"]], [int(x, 16) for x in v["out"]])
            for v in json.load(open(KAT))["vectors"]]


def test_philox_known_answer_vectors():
    for ctr, key, out in _kat():
        got = [int(w) for w in oracle.philox4x32_10(ctr, key)]
        assert got == out, (ctr, key)
    # the library's counter layout: block q of (seed, tensor, step) is the
    # counter (q lo, q hi, tensor, step) under the key (seed lo, seed hi)
    for ctr, key, out in _kat():
        seed, q = key[0] | (key[1] << 32), ctr[0] | (ctr[1] << 32)
        words = oracle.philox_words(seed, ctr[2], ctr[3], q, 1)
        assert [int(w) for w in np.asarray(words).reshape(-1)] == out


@pytest.fixture(scope="module")
def rocrand_ref():
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    hdr = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"
    if not (os.path.exists(hipcc) and os.path.exists(hdr)):
        pytest.skip("hipcc / rocRAND headers not available")
    d = tempfile.mkdtemp(prefix="philox_ref_")
    exe = os.path.join(d, "philox_ref")
    subprocess.run([hipcc, "-O1", "-x", "hip", "--offload-arch=gfx950",
                    os.path.join(HERE, "philox_rocrand_ref.cpp"), "-o", exe],
                   check=True, capture_output=True)

    def run(seed, subseq, q0, nq):
        out = subprocess.run([exe, str(seed), str(subseq), str(q0), str(nq)], check=True,
                             capture_output=True, text=True).stdout.split()
        return np.array([int(x, 16) for x in out], dtype=np.uint64).reshape(nq, 4)
    yield run
    shutil.rmtree(d, ignore_errors=True)


@pytest.mark.parametrize("seed,tensor_id,step,q0", [
    (0, 0, 0, 0), (1, 0, 0, 0), (0xFFFFFFFFFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0),
    (0x0123456789ABCDEF, 3, 11, 1000), (5, 144, 0, (1 << 32) - 2), (2, 7, 1, 123456789012)])
def test_philox_words_match_rocrand(rocrand_ref, seed, tensor_id, step, q0):
    nq = 6
    ref = rocrand_ref(seed, tensor_id | (step << 32), q0, nq)
    got = oracle.philox_words(seed, tensor_id, step, q0, nq).astype(np.uint64)
    np.testing.assert_array_equal(got, ref)


def test_uniform_mapping_is_exact_and_open():
    x = np.array([0, 1, 511, 512, 0xFFFFFFFF, 0x80000000], dtype=np.uint64)
    u = oracle.uniforms_from_words(x)
    assert u[0] == 2.0 ** -24 and u[1] == 2.0 ** -24 and u[2] == 2.0 ** -24
    assert u[3] == 3 * 2.0 ** -24
    assert u[4] == 1 - 2.0 ** -24
    assert u[5] == 0.5 + 2.0 ** -24
    assert np.all(u.astype(np.float32).astype(np.float64) == u)       # representable in fp32


def test_box_muller_special_points():
    z0, z1 = oracle.box_muller(np.exp(-0.5), 0.0)        # radius 1, angle 0
    assert abs(z0 - 1.0) < 1e-15 and abs(z1) < 1e-15
    z0, z1 = oracle.box_muller(np.exp(-2.0), 0.25)       # radius 2, angle pi/2
    assert abs(z0) < 1e-15 and abs(z1 - 2.0) < 1e-15


def test_noise_layout_uses_word_pairs():
    w = oracle.philox_words(9, 4, 2, 0, 3)
    u = oracle.uniforms_from_words(w)
    z = oracle.noise(10, 9, 4, 2)
    a, b = oracle.box_muller(u[:, 0], u[:, 1])
    c, d = oracle.box_muller(u[:, 2], u[:, 3])
    ref = np.stack([a, b, c, d], 1).reshape(-1)[:10]
    np.testing.assert_array_equal(z, ref)


def test_noise_is_standard_normal():
    z = oracle.noise(1 << 20, seed=2024, tensor_id=3, step=0)
    n = z.size
    assert abs(z.mean()) < 5 / np.sqrt(n)
    assert abs(z.var() - 1.0) < 5 * np.sqrt(2.0 / n)
    assert stats.kstest(z, "norm").pvalue > 1e-3
    # streams of different tensors / steps are uncorrelated
    z2 = oracle.noise(1 << 20, seed=2024, tensor_id=4, step=0)
    z3 = oracle.noise(1 << 20, seed=2024, tensor_id=3, step=1)
    assert abs(np.corrcoef(z, z2)[0, 1]) < 5 / np.sqrt(n)
    assert abs(np.corrcoef(z, z3)[0, 1]) < 5 / np.sqrt(n)


def test_add_noise_scale_and_zero_std():
    G = np.arange(12.0).reshape(3, 4)
    np.testing.assert_array_equal(oracle.add_noise(G, 0.0, 1, 0, 0), G)
    z = oracle.noise(12, 1, 0, 0).reshape(3, 4)
    np.testing.assert_allclose(oracle.add_noise(G, 0.8, 1, 0, 0), G + 0.8 * z, rtol=1e-15)


def test_noise_at_selects_from_noise():
    z = oracle.noise(1003, seed=77, tensor_id=5, step=2)
    idx = np.array([[0, 1, 2, 3], [4, 999, 1002, 17]])
    np.testing.assert_array_equal(oracle.noise_at(idx, 77, 5, 2), z[idx])
    big = np.array([(1 << 33) + 5, 7])                   # counter blocks beyond 2^32 elements
    w = oracle.philox_words(77, 5, 2, ((1 << 33) + 5) // 4, 1)
    u = oracle.uniforms_from_words(w)
    assert oracle.noise_at(big, 77, 5, 2)[0] == oracle.box_muller(u[0, 0], u[0, 1])[1]
