"""The seeded input generator: determinism, encodings and workload shape."""
import numpy as np
import pytest
import torch

import synth


def test_rows_independent_of_thread_count_and_regenerable():
    a, _ = synth.gaussian_rows(3, 2, 257, 64, "bf16", threads=1)
    b, _ = synth.gaussian_rows(3, 2, 257, 64, "bf16", threads=7)
    np.testing.assert_array_equal(a, b)
    c, _ = synth.gaussian_rows(3, 2, 0, 64, "bf16", row_ids=np.array([200, 5, 5]))
    np.testing.assert_array_equal(c, a[[200, 5, 5]])
    d, _ = synth.gaussian_rows(3, 2, 57, 64, "bf16", first=200)
    np.testing.assert_array_equal(d, a[200:])


def test_unit_norm_rows():
    x, _ = synth.gaussian_rows(1, 2, 100, 768, "f32")
    n = np.linalg.norm(x.astype(np.float64), axis=1)
    np.testing.assert_allclose(n, 1.0, atol=1e-6)
    # roughly Gaussian coordinates: variance 1/d
    assert abs(x.var() * 768 - 1.0) < 0.05


def test_bf16_encoding_is_rne_of_fp32():
    f, _ = synth.gaussian_rows(4, 2, 50, 128, "f32")
    b, _ = synth.gaussian_rows(4, 2, 50, 128, "bf16")
    ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(b, ref)


def test_fp8_encoding_is_rne_with_row_scale():
    f, _ = synth.gaussian_rows(5, 2, 64, 256, "f32")
    c, s = synth.gaussian_rows(5, 2, 64, 256, "fp8")
    amax = np.abs(f).max(axis=1)
    np.testing.assert_array_equal(s, (amax / np.float32(448.0)).astype(np.float32))
    v = f.astype(np.float64) / s.astype(np.float64)[:, None]
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(c, ref)
    assert c.max() != 0x7F and not np.any(c == 0xFF)   # never NaN


@pytest.mark.parametrize("v", [0.0, -0.0, 1e-12, 2.0 ** -10, 3 * 2.0 ** -10, 0.0625, 447.0,
                               448.0, 460.0, -1.0625, 2.0 ** -6 - 2.0 ** -11])
def test_e4m3_encode_points(v):
    lib = synth._load()
    got = lib.syn_e4m3_encode(v)
    ref = int(torch.tensor([min(v, 448.0)], dtype=torch.float64).to(torch.float8_e4m3fn)
              .view(torch.uint8)[0])
    assert got == ref


def test_tiny_layout_has_20_distinct_ids():
    w = synth.make("tiny")
    assert w.R == 32 and len(set(w.keys.tolist())) == 20
    per = w.template_ids.reshape(4, 8)
    for row in per:
        assert set([0, 1, 2, 3]) <= set(row.tolist())
    # duplicates carry identical vectors
    for t in range(4):
        rows = w.q_req[w.template_ids == t]
        assert np.all(rows == rows[0])


@pytest.mark.parametrize("name", ["ridge1m", "dedup256k", "mfma4m", "fp8_20m"])
def test_zipf_unique_count_near_closed_form(name):
    w = synth.make(name, with_corpus=False)
    nu = len(set(w.keys.tolist()))
    e = synth.expected_unique(w.cfg)
    # the distinct count concentrates tightly (sum of weakly dependent Bernoullis)
    assert abs(nu - e) < 6 * np.sqrt(e) + 5, (nu, e)
    assert w.R == w.cfg.n_requests


def test_keys_distinct_per_template():
    w = synth.make("mfma4m", with_corpus=False)
    pairs = set(zip(w.template_ids.tolist(), w.keys.tolist()))
    assert len(pairs) == len(set(w.template_ids.tolist())) == len(set(w.keys.tolist()))


def test_dedup_keys_are_row_ids():
    w = synth.make("dedup256k", with_corpus=False)
    assert w.keys.min() >= 0 and w.keys.max() < 200_000
