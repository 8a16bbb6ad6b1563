"""Pins of the oracle sampler: Philox4x32-10 against rocRAND's independent
implementation (its open-source header, built for the host), statistical checks
of the uniform and Gumbel draws, and the greedy / top-k limits."""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest
from scipy import stats

from oracle import log_softmax, philox4x32_10, philox_uniform24, sample_token, topk_set
from oracle.philox import gumbel_keys, split_seed, vocab_words

ROCRAND_HDR = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"

_KAT_SRC = r"""
#include <cstdio>
#include <cstdlib>
#include <rocrand/rocrand_philox4x32_10.h>
// Prints rocRAND's Philox4x32-10 block for each (seed, c0, c1, c2, c3) given on argv.
int main(int argc, char** argv) {
  for (int a = 1; a + 4 < argc; a += 5) {
    unsigned long long seed = strtoull(argv[a], 0, 0);
    unsigned long long c[4];
    for (int j = 0; j < 4; ++j) c[j] = strtoull(argv[a + 1 + j], 0, 0);
    // the subsequence index fills counter words 2,3
    rocrand_device::philox4x32_10_engine e(seed, c[2] | (c[3] << 32), 0);
    // skipping n blocks (4n outputs) fills counter words 0,1; chunks avoid 64-bit overflow
    unsigned long long n = c[0] | (c[1] << 32);
    while (n) {
      unsigned long long s = n > (1ull << 61) ? (1ull << 61) : n;
      e.discard(s * 4ull);
      n -= s;
    }
    uint4 r = e.next4();
    printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
"""


@pytest.fixture(scope="module")
def rocrand_philox():
    if not os.path.exists(ROCRAND_HDR):
        pytest.skip("rocRAND headers not present")
    cxx = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    d = tempfile.mkdtemp()
    src, exe = os.path.join(d, "kat.cpp"), os.path.join(d, "kat")
    open(src, "w").write(_KAT_SRC)
    r = subprocess.run([cxx, "-x", "c++", "--offload-host-only", "-O1", src, "-o", exe],
                       capture_output=True, text=True)
    if r.returncode != 0:
        r = subprocess.run(["g++", "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", src,
                            "-o", exe], capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip("cannot build the rocRAND host probe: " + r.stderr[-400:])

    def run(cases):
        args = []
        for seed, c in cases:
            args += [str(seed)] + [str(int(x)) for x in c]
        out = subprocess.run([exe] + args, capture_output=True, text=True, check=True).stdout
        return np.array([[int(t) for t in ln.split()] for ln in out.strip().splitlines()],
                        np.uint64)
    yield run
    shutil.rmtree(d, ignore_errors=True)


def test_philox_matches_rocrand(rocrand_philox):
    rng = np.random.default_rng(0)
    cases = [(0, (0, 0, 0, 0)), (2**64 - 1, (2**32 - 1,) * 4)]
    for _ in range(30):
        seed = int(rng.integers(0, 2**63)) * 2 + int(rng.integers(0, 2))
        ctr = tuple(int(x) for x in rng.integers(0, 2**32, 4, dtype=np.uint64))
        cases.append((seed, ctr))
    ref = rocrand_philox(cases)
    ours = np.concatenate([philox4x32_10(np.array([c], np.uint64), split_seed(s)) for s, c in cases])
    np.testing.assert_array_equal(ours.astype(np.uint64), ref)


def test_vocab_word_layout():
    seed, step, seq, V = 0x1234_5678_9ABC_DEF0, 17, 5, 10
    w = vocab_words(seed, step, seq, V)
    blk = philox4x32_10(np.array([[2, step, seq, 0]], np.uint64), split_seed(seed))[0]
    np.testing.assert_array_equal(w[8:10], blk[:2])


def test_uniform24_range_and_uniformity():
    w = philox4x32_10(np.stack([np.arange(50000), np.zeros(50000), np.ones(50000),
                                np.zeros(50000)], 1).astype(np.uint64), (3, 4)).reshape(-1)
    u = philox_uniform24(w)
    assert u.min() > 0 and u.max() < 1
    k = np.round(u * 2**24)
    assert np.all(k % 2 == 1)
    assert np.all(philox_uniform24(np.array([0, 2**32 - 1], np.uint32)) == [2**-24, 1 - 2**-24])
    assert stats.kstest(u, "uniform").pvalue > 1e-4
    bits = np.unpackbits(w.view(np.uint8))
    assert abs(bits.mean() - 0.5) < 0.002


def test_gumbel_max_frequencies_match_softmax():
    V, n = 16, 100_000
    rng = np.random.default_rng(7)
    z = rng.standard_normal(V) * 1.5
    # n independent draws: steps 0..n-1 of one sequence
    nblk = V // 4
    ctr = np.zeros((n * nblk, 4), np.uint64)
    ctr[:, 0] = np.tile(np.arange(nblk), n)
    ctr[:, 1] = np.repeat(np.arange(n), nblk)
    ctr[:, 2] = 3
    u = philox_uniform24(philox4x32_10(ctr, split_seed(42)).reshape(n, V))
    tok = np.argmax(z[None, :] - np.log(-np.log(u)), axis=1)
    counts = np.bincount(tok, minlength=V)
    p = np.exp(log_softmax(z))
    chi = stats.chisquare(counts, p * n)
    assert chi.pvalue > 1e-4
    # the single-step path of the sampler draws the same keys
    g0 = gumbel_keys(42, 5, 3, V)
    np.testing.assert_allclose(g0, -np.log(-np.log(u[5])), rtol=1e-15)


def test_topk_set_brute_force():
    rng = np.random.default_rng(1)
    l = rng.integers(-3, 4, 40).astype(np.float64)   # many ties
    for k in (1, 5, 17, 40):
        brute = [i for _, i in sorted((-l[i], i) for i in range(40))][:k]
        assert list(topk_set(l, k)) == brute
    assert len(topk_set(l, 0)) == 40


def test_greedy_limits_and_logp():
    rng = np.random.default_rng(2)
    l = rng.standard_normal(300)
    l[[17, 200]] = l.max() + 1.0          # a tie at the top: lowest id wins
    tok, lp, _ = sample_token(l, 0.0, 0, 1, 0, 0)
    assert tok == 17
    assert abs(lp - log_softmax(l)[17]) < 1e-14
    # top_k = 1 with any temperature picks the greedy token
    for T in (0.5, 1.0, 3.0):
        assert sample_token(l, T, 1, 9, 3, 2)[0] == 17
    # temperature -> 0 reduces to greedy
    l2 = rng.standard_normal(300)
    assert sample_token(l2, 1e-9, 0, 5, 1, 1)[0] == int(np.argmax(l2))
    # logp is the full-vocabulary log-softmax of z = l / T
    tok, lp, _ = sample_token(l2, 0.8, 50, 5, 1, 1)
    assert abs(lp - log_softmax(l2 / 0.8)[tok]) < 1e-13
    assert tok in set(topk_set(l2, 50))


def test_log_softmax_properties():
    rng = np.random.default_rng(3)
    z = rng.standard_normal((4, 1000)) * 10
    ls = log_softmax(z)
    np.testing.assert_allclose(np.exp(ls).sum(axis=1), 1.0, rtol=0, atol=1e-12)
    assert np.all(ls <= 0)
    np.testing.assert_allclose(log_softmax(z + 123.0), ls, rtol=0, atol=1e-11)
