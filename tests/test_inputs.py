"""The seeded generator: determinism, thread independence, rounding, recipe."""

import numpy as np

from paper_2609_18077_amd import inputs


def test_bf16_rounding_matches_definition():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -0.0, 3.0e38, 1.0 + 2 ** -9], np.float32)
    b = inputs.f32_to_bf16_bits(x)
    assert list(b) == [0x3F80, 0x3F80, 0x3F82, 0x8000, 0x7F62, 0x3F80]


def test_deterministic_and_chunked():
    a = inputs.bf16_tensor(5, 1, (3, inputs.CHUNK // 64 + 7, 1, 128))
    b = inputs.bf16_tensor(5, 1, (3, inputs.CHUNK // 64 + 7, 1, 128))
    assert np.array_equal(a, b)
    c = inputs.bf16_tensor(6, 1, (3, inputs.CHUNK // 64 + 7, 1, 128))
    assert not np.array_equal(a, c)
    # first chunk is the plain PCG64 stream of SeedSequence([seed, tensor, 0])
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([5, 1, 0])))
    ref = g.standard_normal(1000, dtype=np.float32)
    assert np.array_equal(a.reshape(-1)[:1000], inputs.f32_to_bf16_bits(ref))


def test_rms_norm_recipe():
    x = inputs.bf16_tensor(2, 0, (1, 64, 3, 128), rms_norm=True)
    f = (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    rms = np.sqrt((f * f).mean(-1))
    assert np.allclose(rms, 1.0, atol=1e-2)


def test_workload_table():
    w = inputs.WORKLOADS
    assert w["wan13b_480p"].n_rot == 32760 == w["wan13b_480p"].Lq
    assert w["wan14b_720p"].n_rot == 75600
    assert w["hunyuan_joint"].n_rot == 118800 and w["hunyuan_joint"].Lq == 119056
    assert list(inputs.kv_valid_len(w["hunyuan_joint"])) == [118980]
    lv = inputs.kv_valid_len(w["cross_text"])
    assert lv.shape == (2,) and np.all((lv >= 64) & (lv <= 512))
    assert w["tiny"].scale == float(np.float32(1 / np.sqrt(128)))
