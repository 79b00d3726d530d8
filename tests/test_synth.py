"""The seeded input generator: SplitMix64 against its published outputs and
the distributions' basic properties."""

import numpy as np

import synth


def test_splitmix64_published_outputs():
    # the first outputs of splitmix64 seeded with 0 (Vigna's reference code)
    assert int(synth.splitmix64(np.uint64(0))) == 0xE220A8397B1DCDAF
    assert int(synth.splitmix64(synth.GAMMA)) == 0x6E789E6AA1B965F4
    assert int(synth.splitmix64(np.uint64((2 * 0x9E3779B97F4A7C15) % 2 ** 64))) == \
        0x06C45D188009454F


def test_sampled_values_match_full_generation():
    for dist, kw in (("uniform_int", {"lo": -5, "hi": 9}),
                     ("normal_f32", {}), ("uniform_u32_mat", {})):
        full = synth.generate(dist, 2111, 6, 50, **kw)
        part = synth.sample(dist, 2111, [0, 3, 5], [1, 17, 49], **kw)
        assert np.array_equal(full[[0, 3, 5]][:, [1, 17, 49]], part)


def test_threaded_generation_is_identical():
    a = synth.generate("normal_f32", 3, 40, 4096, threads=1)
    b = synth.generate("normal_f32", 3, 40, 4096, threads=8)
    assert np.array_equal(a, b)


def test_distributions():
    x = synth.generate("uniform_int", 1, 4, 20000, lo=-1000, hi=1000)
    assert x.dtype == np.int32 and x.min() == -1000 and x.max() == 1000
    z = synth.generate("normal_f32", 2, 4, 50000)
    assert z.dtype == np.float32
    assert abs(float(z.mean())) < 0.02 and abs(float(z.std()) - 1) < 0.02
    mt = synth.generate("odd_det_u32_mat", 3, 2, 100)
    det = (mt[..., 0].astype(np.uint64) * mt[..., 3]
           - mt[..., 1].astype(np.uint64) * mt[..., 2]) & np.uint64(1)
    assert (det == 1).all()
