"""The seeded input generator: determinism, storage encoding and the
distributions the workloads state.  CPU only."""
import numpy as np
import torch

import fusedsub_data as fd


def test_bf16_encoding_matches_library_cast():
    rng = np.random.default_rng(0)
    v = np.concatenate([rng.standard_normal(50000) * 3, [0.0, -0.0, np.inf, -np.inf, 1e-40]])
    ref = torch.from_numpy(v.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy()
    np.testing.assert_array_equal(fd.f32_to_bf16_bits(v).view(np.int16), ref)
    back = fd.bf16_bits_to_f64(fd.f32_to_bf16_bits(v))
    np.testing.assert_array_equal(back, torch.from_numpy(ref).view(torch.bfloat16).double().numpy())


def test_seed_determinism_and_distinct_seeds():
    a = fd.softmax_inputs(3, 16, 64)
    b = fd.softmax_inputs(3, 16, 64)
    c = fd.softmax_inputs(4, 16, 64)
    np.testing.assert_array_equal(a["x"].data, b["x"].data)
    np.testing.assert_array_equal(a["mask"].data, b["mask"].data)
    assert not np.array_equal(a["x"].data, c["x"].data)


def test_softmax_mask_rate_and_no_empty_row():
    d = fd.softmax_inputs(0, 512, 512, p_masked=0.1)
    m = d["mask"].f64()
    assert set(np.unique(m)) <= {0.0, -np.inf}
    frac = np.isinf(m).mean()
    assert 0.095 < frac < 0.105
    d = fd.softmax_inputs(0, 64, 4, p_masked=0.9)
    assert (~np.isinf(d["mask"].f64())).any(axis=1).all()


def test_byte_mask_has_the_pattern_of_the_additive_mask():
    a = fd.softmax_inputs(5, 300, 96, "bf16")
    b = fd.softmax_inputs(5, 300, 96, "bf16", mask_dtype="u8")
    np.testing.assert_array_equal(a["x"].data, b["x"].data)
    assert b["mask"].dtype == "u8" and b["mask"].data.dtype == np.uint8
    np.testing.assert_array_equal(b["mask"].data != 0, np.isinf(a["mask"].f64()))
    vals = b["mask"].data[b["mask"].data != 0]
    assert vals.min() >= 1 and len(np.unique(vals)) > 100   # many byte values, not just 1
    np.testing.assert_array_equal(b["mask"].f64(), b["mask"].data.astype(np.float64))


def test_distributions():
    d = fd.layernorm_inputs(1, 256, 1024)
    assert abs(d["x"].f64().std() - 1.0) < 0.01
    assert abs(d["gamma"].f64().mean() - 1.0) < 0.02
    assert abs(d["gamma"].f64().std() - 0.1) < 0.01
    p = fd.pointwise_inputs(1, 256, 1024)
    b = p["bias"].f64()
    assert b.min() >= -0.5 and b.max() < 0.5
    assert p["scale"] == float(np.float32(0.7))
    e = fd.epilogue_inputs(2, 64, 4096)
    s = e["col_scale"].f64()
    assert s.min() >= 0.5 and s.max() < 1.5
    assert abs(e["c"].f64().std() - 0.0256) < 0.001
