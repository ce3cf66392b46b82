"""The seeded input generators against their published definitions (CPU only)."""
import numpy as np
import pytest
from scipy import stats

from workloads import configs, gen


def test_splitmix64_published_vectors():
    # Sequential SplitMix64 from state 0 (Steele, Lea & Flood 2014; reference outputs).
    assert gen.splitmix64_sequence(0, 3) == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    # the counter form draws the same sequence
    d = gen.draws_u64(0, 0, 3)
    assert [int(x) for x in d] == gen.splitmix64_sequence(0, 3)


def test_uniform53_range_and_moments():
    u = gen.uniform53(gen.stream_key(1, 0, 5), 0, 200_000)
    assert u.min() >= 0.0 and u.max() < 1.0
    assert abs(u.mean() - 0.5) < 5 * (1 / np.sqrt(12 * 200_000))


def test_normals_moments():
    z = gen.normal_f32(gen.stream_key(2, 0, 5), 400_000, 0.01).astype(np.float64)
    assert abs(z.mean()) < 5 * 0.01 / np.sqrt(400_000)
    assert abs(z.std() - 0.01) < 1e-4
    assert stats.kstest(z / 0.01, "norm").pvalue > 1e-4


@pytest.mark.parametrize("s", [1.0, 1.1, 1.3])
def test_zipf_chi_square(s):
    V, n = 50, 200_000
    ids = gen.zipf_ids(gen.stream_key(3, 0, gen.PURPOSE_IDS), n, V, s)
    assert ids.min() >= 0 and ids.max() < V
    obs = np.bincount(ids, minlength=V)
    exp = gen.zipf_pmf(V, s) * n
    assert stats.chisquare(obs, exp).pvalue > 1e-4


def test_uniform_ids_expected_unique_count():
    # E[U] = V (1 - (1 - 1/V)^T) for T uniform draws over V ids.
    V, T = 1 << 20, 65536
    ids = gen.uniform_ids(gen.stream_key(51, 0, gen.PURPOSE_IDS), T, V)
    U = np.unique(ids).size
    EU = V * (1 - (1 - 1 / V) ** T)
    assert abs(U - EU) < 5 * np.sqrt(EU * (1 - EU / V) + 1)


def test_bf16_round_to_nearest_even():
    bits = np.array([0x3F800000, 0x3F808000, 0x3F818000, 0x3F808001, 0x3F80FFFF, 0xBF808000, 0x7F7FFFFF],
                    dtype=np.uint32)
    x = bits.view(np.float32)
    assert gen.bf16_round(x).tolist() == [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0x3F81, 0xBF80, 0x7F80]
    # widening is exact and rounding a bf16 value is the identity
    h = np.arange(0, 0x7F80, 7, dtype=np.uint16)
    assert np.array_equal(gen.bf16_round(gen.bf16_bits_to_f32(h)), h)


def test_owner_maps():
    assert gen.owner_mod(10, 3).tolist() == [0, 1, 2, 0, 1, 2, 0, 1, 2, 0]
    assert gen.owner_range(10, 3).tolist() == [0, 0, 0, 0, 1, 1, 1, 1, 2, 2]
    assert gen.owner_range(32768, 4).tolist()[8191:8193] == [0, 1]


def test_workload_shapes_small():
    spec = configs.WORKLOADS["tiny"].tables[0]
    ids, g = configs.make_batch(spec, 0)
    assert ids.shape == (512,) and g.shape == (512, 64) and g.dtype == np.float32
    ids2, _ = configs.make_batch(spec, 0)
    assert np.array_equal(ids, ids2)  # seeded
    spec4 = configs.WORKLOADS["lm_large_vocab_bf16"].tables[0]
    g4 = configs.make_grads(spec4, 0, T=8)
    assert g4.dtype == np.uint16 and g4.shape == (8, 1024)


def test_compiled_normals_match_reference():
    key = gen.stream_key(9, 3, gen.PURPOSE_GRADS)
    for n in (0, 1, 2, 7, 10001):
        a = gen.normal_f32(key, n, 0.5)
        b = gen.normal_f32_reference(key, n, 0.5)
        assert a.shape == b.shape
        # same definition; libm and numpy may differ in the last fp64 bit
        assert np.all(np.abs(a.astype(np.float64) - b) <= np.spacing(np.abs(b)))
