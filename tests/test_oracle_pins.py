"""Pins of the float64 oracle against values and identities fixed by the
paper's definitions and by mathematics -- never against the oracle itself
re-typed.  CPU only.

Each group is built so that a plausible mistake in the oracle (a dropped
term, a wrong sign or constant, a wrong axis, a swapped order of operations)
fails at least one test; the mistake each test catches is named in it.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from conftest import read_golden

GOLD = read_golden("normal_cdf.txt")
PHI = {float(z): float(v) for k, z, v in GOLD if k == "phi"}
ERF = {float(z): float(v) for k, z, v in GOLD if k == "erf"}


# ---------------------------------------------------------------------------
# activations
# ---------------------------------------------------------------------------
class TestGelu:
    def test_table_values(self):
        # GELU(z) = z * Phi(z); catches erf(z/2) or erf(z) for erf(z/sqrt 2),
        # a missing factor 1/2 and a missing "1 +".
        for z, phi in PHI.items():
            assert oracle.gelu_erf(z) == pytest.approx(z * phi, abs=2e-15)
            assert oracle.gelu_erf(-z) == pytest.approx(-z * (1.0 - phi), abs=2e-15)

    def test_erf_table(self):
        from scipy.special import erf
        for z, v in ERF.items():
            assert erf(z) == pytest.approx(v, abs=1e-15)

    def test_zero_and_odd_part(self):
        assert oracle.gelu_erf(0.0) == 0.0
        z = np.linspace(-6, 6, 1001)
        # Phi(z) + Phi(-z) = 1  =>  GELU(z) - GELU(-z) = z
        np.testing.assert_allclose(oracle.gelu_erf(z) - oracle.gelu_erf(-z), z,
                                   rtol=0, atol=1e-14)

    def test_tails(self):
        assert oracle.gelu_erf(12.0) == 12.0
        g = oracle.gelu_erf(-12.0)
        assert g <= 0.0 and g > -1e-30


class TestSigmoid:
    def test_closed_forms(self):
        assert oracle.sigmoid(0.0) == 0.5
        for k in (2.0, 3.0, 7.0, 99.0):       # sigma(ln k) = k / (k + 1)
            assert oracle.sigmoid(math.log(k)) == pytest.approx(k / (k + 1), rel=1e-15)
            assert oracle.sigmoid(-math.log(k)) == pytest.approx(1 / (k + 1), rel=1e-14)

    def test_symmetry_and_extremes(self):
        t = np.linspace(-30, 30, 601)
        np.testing.assert_allclose(oracle.sigmoid(-t), 1 - oracle.sigmoid(t), atol=1e-15)
        assert oracle.sigmoid(-1000.0) == 0.0
        assert oracle.sigmoid(1000.0) == 1.0


# ---------------------------------------------------------------------------
# a1 pointwise chain
# ---------------------------------------------------------------------------
class TestPointwise:
    def test_order_scale_bias_act_residual(self):
        x = np.array([[1.0]])
        # scale before bias: 1*2 + 1 = 3 (not (1+1)*2 = 4)
        y = oracle.pointwise_chain(x, np.array([1.0]), None, 2.0, "none")
        assert y[0, 0] == 3.0
        # residual after the activation: GELU(1) + 1 = Phi(1) + 1 (not GELU(2))
        y = oracle.pointwise_chain(np.array([[0.0]]), np.array([1.0]), np.array([[1.0]]),
                                   1.0, "gelu_erf")
        assert y[0, 0] == pytest.approx(PHI[1.0] + 1.0, abs=2e-15)

    def test_bias_broadcasts_per_column(self):
        x = np.zeros((2, 3))
        b = np.array([1.0, 2.0, 3.0])
        y = oracle.pointwise_chain(x, b, None, 1.0, "none")
        np.testing.assert_array_equal(y, [[1, 2, 3], [1, 2, 3]])

    def test_zero_scale_bias_gives_residual(self):
        rng = np.random.default_rng(0)
        x, r = rng.standard_normal((4, 5)), rng.standard_normal((4, 5))
        y = oracle.pointwise_chain(x, np.zeros(5), r, 0.0, "gelu_erf")
        np.testing.assert_array_equal(y, r)

    def test_acts(self):
        x = np.array([[-2.0, -0.5, 0.0, 0.5, 2.0]])
        np.testing.assert_array_equal(oracle.pointwise_chain(x, None, None, 1.0, "relu"),
                                      [[0, 0, 0, 0.5, 2.0]])
        np.testing.assert_allclose(
            oracle.pointwise_chain(x, None, None, 1.0, "sigmoid"),
            [[1 / (1 + math.exp(2)), 1 / (1 + math.exp(0.5)), 0.5,
              1 / (1 + math.exp(-0.5)), 1 / (1 + math.exp(-2))]], rtol=1e-15)


class TestPointwiseProgram:
    def test_empty_program_is_identity(self):
        x = np.array([[1.5, -2.0, 0.0]])
        np.testing.assert_array_equal(oracle.pointwise_program(x, []), x)

    def test_order_is_the_listed_order(self):
        x = np.array([[3.0]])
        assert oracle.pointwise_program(x, [("scale", 2), ("shift", 1)])[0, 0] == 7.0
        assert oracle.pointwise_program(x, [("shift", 1), ("scale", 2)])[0, 0] == 8.0

    def test_linear_mul_hardtanh_gelu_chain(self):
        # the paper's fused group (a multiply, a hardtanh, a GELU after a
        # linear layer) on values whose results the normal table gives:
        # 3 * 0.5 = 1.5 clamps to 1 -> Phi(1); 1 * 0.5 = 0.5 passes ->
        # 0.5 Phi(0.5); -1 * 0.5 -> -0.5 Phi(-0.5) = -0.5 (1 - Phi(0.5));
        # -8 * 0.5 = -4 clamps to -1 -> -(1 - Phi(1))
        x = np.array([[3.0, 1.0, -1.0, -8.0]])
        y = oracle.pointwise_program(x, [("scale", 0.5), ("clamp", -1, 1), ("gelu_erf",)])
        want = [PHI[1.0], 0.5 * PHI[0.5], -0.5 * (1 - PHI[0.5]), -(1 - PHI[1.0])]
        np.testing.assert_allclose(y[0], want, rtol=0, atol=1e-15)

    def test_clamp_leaky_relu_and_relu(self):
        x = np.array([[-2.0, -0.5, 0.0, 0.5, 2.0]])
        np.testing.assert_array_equal(oracle.pointwise_program(x, [("clamp", -1, 1)]),
                                      [[-1, -0.5, 0, 0.5, 1]])
        np.testing.assert_allclose(oracle.pointwise_program(x, [("leaky_relu", 0.1)]),
                                   [[-0.2, -0.05, 0, 0.5, 2.0]], rtol=1e-15)
        np.testing.assert_array_equal(oracle.pointwise_program(x, [("relu",)]),
                                      [[0, 0, 0, 0.5, 2.0]])

    def test_tanh_and_silu_closed_forms(self):
        # tanh(ln(3) / 2) = (3 - 1) / (3 + 1) = 1/2 and tanh is odd;
        # silu(ln 3) = ln 3 * 3/4 (sigmoid(ln 3) = 3/4), silu(0) = 0,
        # silu(-ln 3) = -ln 3 / 4
        l3 = math.log(3.0)
        y = oracle.pointwise_program(np.array([[l3 / 2, -l3 / 2, 0.0]]), [("tanh",)])
        np.testing.assert_allclose(y[0], [0.5, -0.5, 0.0], rtol=1e-15, atol=1e-16)
        y = oracle.pointwise_program(np.array([[l3, 0.0, -l3]]), [("silu",)])
        np.testing.assert_allclose(y[0], [0.75 * l3, 0.0, -0.25 * l3], rtol=1e-15)
        y = oracle.pointwise_program(np.array([[l3]]), [("sigmoid",)])
        assert y[0, 0] == pytest.approx(0.75, rel=1e-15)

    def test_vectors_broadcast_per_column_and_residual_per_element(self):
        x = np.array([[1.0, 2.0], [3.0, 4.0]])
        b = np.array([10.0, 20.0])
        c = np.array([2.0, -1.0])
        r = np.array([[1.0, 0.0], [-1.0, 5.0]])
        y = oracle.pointwise_program(x, [("add_bias",), ("mul_column",), ("add_residual",)],
                                     bias=b, col=c, residual=r)
        np.testing.assert_array_equal(y, [[23.0, -22.0], [25.0, -19.0]])
        y = oracle.pointwise_program(x, [("mul_residual",)], residual=r)
        np.testing.assert_array_equal(y, [[1.0, 0.0], [-3.0, 20.0]])

    def test_rejects_unknown_or_malformed_operations(self):
        with pytest.raises(ValueError):
            oracle.pointwise_program(np.zeros((1, 1)), [("softplus",)])
        with pytest.raises(ValueError):
            oracle.pointwise_program(np.zeros((1, 1)), [("clamp", -1)])


# ---------------------------------------------------------------------------
# a2 row softmax
# ---------------------------------------------------------------------------
class TestSoftmax:
    def test_known_row_and_scale(self):
        # exp of [0, ln2, ln3] is [1, 2, 3]: softmax = [1/6, 2/6, 3/6].  The
        # logits are given doubled with scale 1/2, so a divide-by-scale or a
        # dropped scale fails.
        x = np.array([[0.0, 2 * math.log(2), 2 * math.log(3)]])
        y = oracle.row_softmax(x, None, 0.5)
        np.testing.assert_allclose(y, [[1 / 6, 2 / 6, 3 / 6]], rtol=1e-14)

    def test_large_logits_do_not_overflow(self):
        # exp(1000) overflows float64: the max must be subtracted first
        y = oracle.row_softmax(np.array([[1000.0, 1000.0 + math.log(3)]]), None, 1.0)
        np.testing.assert_allclose(y, [[0.25, 0.75]], rtol=1e-13)

    def test_rows_sum_to_one_along_last_axis(self):
        rng = np.random.default_rng(1)
        x = rng.standard_normal((5, 7)) * 3
        y = oracle.row_softmax(x, None, 0.125)
        np.testing.assert_allclose(y.sum(axis=1), 1.0, atol=1e-14)
        assert not np.allclose(y.sum(axis=0), 1.0)

    def test_shift_invariance(self):
        rng = np.random.default_rng(2)
        x = rng.standard_normal((6, 9)) * 3
        c = rng.standard_normal((6, 1)) * 100
        np.testing.assert_allclose(oracle.row_softmax(x + c, None, 1.0),
                                   oracle.row_softmax(x, None, 1.0), atol=1e-13)

    def test_mask_uniform_and_pairs(self):
        ninf = -np.inf
        x = np.array([[5.0, 5.0, 5.0, 5.0], [1.0, 2.0, 3.0, 4.0]])
        mask = np.array([[0.0, ninf, 0.0, 0.0], [ninf, 0.0, ninf, 0.0]])
        y = oracle.row_softmax(x, mask, 1.0)
        np.testing.assert_allclose(y[0], [1 / 3, 0, 1 / 3, 1 / 3], rtol=1e-15)
        # two unmasked entries: logistic of the difference
        np.testing.assert_allclose(y[1], [0, 1 / (1 + math.e ** 2), 0, 1 / (1 + math.e ** -2)],
                                   rtol=1e-14)
        assert y[0, 1] == 0.0 and y[1, 0] == 0.0 and y[1, 2] == 0.0

    def test_byte_mask_keeps_the_zero_bytes_only(self):
        # brute force: the softmax of a row under a byte mask is the softmax
        # of its kept entries alone (zero bytes), placed back, with exact
        # zeros at the nonzero bytes -- whatever their value (1, 7, 255)
        rng = np.random.default_rng(4)
        x = rng.standard_normal((3, 8)) * 2
        m = np.array([[0, 1, 0, 255, 0, 0, 7, 0],
                      [1, 1, 1, 1, 1, 1, 1, 0],
                      [0, 0, 0, 0, 0, 0, 0, 0]], dtype=np.uint8)
        add = oracle.byte_mask_additive(m)
        assert add.dtype == np.float64
        np.testing.assert_array_equal(np.isinf(add), m != 0)
        assert np.all(add[m == 0] == 0.0) and np.all(add[m != 0] < 0)
        y = oracle.row_softmax(x, add, 0.5)
        for r in range(3):
            keep = [j for j in range(8) if m[r, j] == 0]
            e = [math.exp(0.5 * x[r, j]) for j in keep]
            want = np.zeros(8)
            for j, v in zip(keep, e):
                want[j] = v / sum(e)
            np.testing.assert_allclose(y[r], want, rtol=1e-14, atol=0)
        assert np.all(y[m != 0] == 0.0)
        np.testing.assert_array_equal(y[1], [0, 0, 0, 0, 0, 0, 0, 1])
        np.testing.assert_array_equal(y[2], oracle.row_softmax(x[2:], None, 0.5)[0])

    def test_fully_masked_row_is_zero(self):
        y = oracle.row_softmax(np.ones((1, 3)), np.full((1, 3), -np.inf), 1.0)
        np.testing.assert_array_equal(y, 0.0)

    def test_causal_square(self):
        rng = np.random.default_rng(3)
        s = 6
        x = rng.standard_normal((2 * s, s))       # two heads stacked as rows
        y = oracle.row_softmax(x, None, 1.0, causal_q_len=s)
        for r in range(2 * s):
            t = r % s
            assert np.all(y[r, t + 1:] == 0.0)
            assert y[r, :t + 1].sum() == pytest.approx(1.0, abs=1e-15)
        np.testing.assert_array_equal(y[0], [1, 0, 0, 0, 0, 0])     # row 0 one-hot
        np.testing.assert_array_equal(y[s], [1, 0, 0, 0, 0, 0])
        d = x[1, 0] - x[1, 1]
        np.testing.assert_allclose(y[1, :2], [1 / (1 + math.exp(-d)), 1 / (1 + math.exp(d))],
                                   rtol=1e-14)

    def test_causal_rectangular_offset(self):
        # q_len 2 queries over 5 keys: query i sees keys 0 .. i + 3
        m = oracle.causal_mask(4, 5, 2)
        np.testing.assert_array_equal(m, [[0, 0, 0, 0, 1], [0, 0, 0, 0, 0],
                                          [0, 0, 0, 0, 1], [0, 0, 0, 0, 0]])


# ---------------------------------------------------------------------------
# a3 LayerNorm + residual
# ---------------------------------------------------------------------------
class TestLayerNorm:
    def test_hand_example(self):
        # h = [1,2,3,4]: mean 2.5, biased variance 1.25 (unbiased would be 5/3)
        y, h = oracle.layernorm_residual(np.array([[1.0, 2.0, 3.0, 4.0]]), None, None, None, 0.0)
        v = 1.5 / math.sqrt(1.25)
        np.testing.assert_allclose(y, [[-v, -v / 3, v / 3, v]], rtol=1e-15)

    def test_two_elements_biased_variance_and_affine(self):
        y, _ = oracle.layernorm_residual(np.array([[1.0, 3.0]]), None, None, None, 0.0)
        np.testing.assert_array_equal(y, [[-1.0, 1.0]])
        y, _ = oracle.layernorm_residual(np.array([[1.0, 3.0]]), None,
                                         np.array([2.0, 3.0]), np.array([5.0, 7.0]), 0.0)
        np.testing.assert_array_equal(y, [[3.0, 10.0]])       # gamma then beta, per column

    def test_eps_inside_sqrt(self):
        # variance of the normalised row is var / (var + eps) exactly
        rng = np.random.default_rng(4)
        h = rng.standard_normal((3, 64))
        eps = 0.25
        y, _ = oracle.layernorm_residual(h, None, None, None, eps)
        var = np.var(h, axis=1)
        np.testing.assert_allclose(y.mean(axis=1), 0.0, atol=1e-15)
        np.testing.assert_allclose(np.var(y, axis=1), var / (var + eps), rtol=1e-13)

    def test_constant_row_gives_beta_and_residual_is_added(self):
        rng = np.random.default_rng(5)
        x = rng.standard_normal((2, 8))
        beta = rng.standard_normal(8)
        gamma = rng.standard_normal(8)
        y, h = oracle.layernorm_residual(x, 3.0 - x, gamma, beta, 1e-5)
        np.testing.assert_allclose(h, 3.0, atol=1e-15)
        np.testing.assert_allclose(y, np.broadcast_to(beta, (2, 8)), atol=1e-10)

    def test_scale_invariance_eps0(self):
        rng = np.random.default_rng(6)
        h = rng.standard_normal((4, 33))
        a, _ = oracle.layernorm_residual(h, None, None, None, 0.0)
        b, _ = oracle.layernorm_residual(7.5 * h, None, None, None, 0.0)
        np.testing.assert_allclose(a, b, atol=1e-13)

    def test_round_to_bf16_known_values(self):
        f = oracle.round_to_bf16
        assert f(1.0 + 2 ** -8) == 1.0                      # tie -> even (down)
        assert f(1.0 + 3 * 2 ** -8) == 1.0 + 2 ** -6        # tie -> even (up)
        assert f(1.0 + 2 ** -8 + 2 ** -20) == 1.0 + 2 ** -7  # above the tie
        assert f(-(1.0 + 2 ** -8)) == -1.0
        assert f(2.0 ** -133) == 2.0 ** -133               # smallest subnormal
        assert f(2.0 ** -135) == 0.0
        assert f(3.0e38 * 2) == np.inf

    def test_round_to_bf16_matches_library_cast(self):
        rng = np.random.default_rng(7)
        v = np.concatenate([rng.standard_normal(20000).astype(np.float32),
                            (rng.standard_normal(2000) * 1e-39).astype(np.float32),
                            np.float32(1.0) + np.float32(2.0 ** -8) * np.arange(64,
                                                                              dtype=np.float32)])
        ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
        np.testing.assert_array_equal(oracle.round_to_bf16(v.astype(np.float64)), ref)

    def test_residual_store_is_rounded_fp32_sum(self):
        rng = np.random.default_rng(8)
        xb = torch.from_numpy(rng.standard_normal(5000).astype(np.float32)).to(torch.bfloat16)
        rb = torch.from_numpy(rng.standard_normal(5000).astype(np.float32)).to(torch.bfloat16)
        ref = (xb.float() + rb.float()).to(torch.bfloat16).double().numpy()
        got = oracle.residual_store_bf16(xb.double().numpy(), rb.double().numpy())
        np.testing.assert_array_equal(got, ref)


# ---------------------------------------------------------------------------
# a4 GEMM epilogue + row reduction
# ---------------------------------------------------------------------------
class TestEpilogue:
    def test_max_and_logsumexp_reductions(self):
        # C + b then * s, act, then the row's max or log-sum-exp: with
        # relu over [-1, ln 3 - 1] + 1 -> [0, ln 3], max ln 3 and LSE log 4;
        # sigmoid of 0 everywhere -> max 1/2 and LSE 1/2 + log(cols)
        c = np.array([[-1.0, math.log(3.0) - 1.0]])
        b, s = np.array([1.0, 1.0]), np.array([1.0, 1.0])
        assert oracle.gemm_epilogue_reduce(c, b, s, "relu", "max")[0] == pytest.approx(
            math.log(3.0), rel=1e-15)
        assert oracle.gemm_epilogue_reduce(c, b, s, "relu", "logsumexp")[0] == pytest.approx(
            math.log(4.0), rel=1e-15)
        z = oracle.gemm_epilogue_reduce(np.zeros((2, 64)), None, None, "sigmoid", "logsumexp")
        np.testing.assert_allclose(z, 0.5 + math.log(64.0), rtol=1e-15)
        assert (oracle.gemm_epilogue_reduce(np.zeros((2, 64)), None, None, "sigmoid", "max")
                == 0.5).all()

    def test_zero_input_gives_half_count(self):
        out = oracle.gemm_epilogue_reduce(np.zeros((3, 8192)), np.zeros(8192), np.ones(8192),
                                          "sigmoid", "sum")
        np.testing.assert_array_equal(out, 4096.0)

    def test_hand_example_and_bias_axis(self):
        l3 = math.log(3)
        c = np.array([[l3, 0.0], [0.0, -l3]])
        np.testing.assert_allclose(oracle.gemm_epilogue_reduce(c, None, None, "sigmoid", "sum"),
                                   [1.25, 0.75], rtol=1e-15)
        # per-column bias on a 2x3 matrix: every row sees [ln3, 0, -ln3]
        out = oracle.gemm_epilogue_reduce(np.zeros((2, 3)), np.array([l3, 0.0, -l3]),
                                          None, "sigmoid", "sum")
        np.testing.assert_allclose(out, [1.5, 1.5], rtol=1e-15)

    def test_bias_before_scale(self):
        # (1 + 1) * 2 = 4 -> sigma(4); 1*2 + 1 = 3 would give sigma(3)
        out = oracle.gemm_epilogue_reduce(np.array([[1.0]]), np.array([1.0]), np.array([2.0]),
                                          "sigmoid", "sum")
        assert out[0] == pytest.approx(1 / (1 + math.exp(-4)), rel=1e-15)

    def test_sign_flip_symmetry_and_mean(self):
        rng = np.random.default_rng(9)
        c = rng.standard_normal((4, 100)) * 0.03
        b = rng.uniform(-0.5, 0.5, 100)
        s = rng.uniform(0.5, 1.5, 100)
        o = oracle.gemm_epilogue_reduce(c, b, s, "sigmoid", "sum")
        o2 = oracle.gemm_epilogue_reduce(-c, -b, s, "sigmoid", "sum")
        np.testing.assert_allclose(o + o2, 100.0, atol=1e-12)
        np.testing.assert_allclose(oracle.gemm_epilogue_reduce(c, b, s, "sigmoid", "mean"),
                                   o / 100, rtol=1e-15)

    def test_identity_act_is_weighted_row_sum(self):
        c = np.array([[1.0, 2.0, 3.0], [4.0, 5.0, 6.0]])
        out = oracle.gemm_epilogue_reduce(c, np.array([1.0, 0.0, -1.0]),
                                          np.array([1.0, 10.0, 100.0]), "none", "sum")
        np.testing.assert_array_equal(out, [2 + 20 + 200, 5 + 50 + 500])


# ---------------------------------------------------------------------------
# a5 stitched block
# ---------------------------------------------------------------------------
def _tiny_params(rng, hid, mlp, std=0.3):
    p = {
        "w_qkv": rng.standard_normal((hid, 3 * hid)) * std,
        "b_qkv": rng.standard_normal(3 * hid) * std,
        "w_o": rng.standard_normal((hid, hid)) * std,
        "b_o": rng.standard_normal(hid) * std,
        "w_1": rng.standard_normal((hid, mlp)) * std,
        "b_1": rng.standard_normal(mlp) * std,
        "w_2": rng.standard_normal((mlp, hid)) * std,
        "b_2": rng.standard_normal(hid) * std,
        "ln1_gamma": 1 + 0.1 * rng.standard_normal(hid),
        "ln1_beta": 0.1 * rng.standard_normal(hid),
        "ln2_gamma": 1 + 0.1 * rng.standard_normal(hid),
        "ln2_beta": 0.1 * rng.standard_normal(hid),
    }
    return p


class TestBlock:
    S, H, NH, F = 7, 8, 2, 12

    def test_causality(self):
        rng = np.random.default_rng(10)
        p = _tiny_params(rng, self.H, self.F)
        x = rng.standard_normal((self.S, self.H))
        y = oracle.block_forward_sequence(x, p, self.NH, 1e-5)["out"]
        for t in range(self.S - 1):
            x2 = x.copy()
            x2[t + 1:] = rng.standard_normal((self.S - t - 1, self.H)) * 5
            y2 = oracle.block_forward_sequence(x2, p, self.NH, 1e-5)["out"]
            np.testing.assert_allclose(y2[:t + 1], y[:t + 1], atol=1e-12)
            assert not np.allclose(y2[t + 1:], y[t + 1:])

    def test_token0_attends_to_itself(self):
        rng = np.random.default_rng(11)
        p = _tiny_params(rng, self.H, self.F)
        x = rng.standard_normal((self.S, self.H))
        r = oracle.block_forward_sequence(x, p, self.NH, 1e-5, keep=("qkv", "o"))
        np.testing.assert_allclose(r["o"][0], r["qkv"][0, 2 * self.H:], atol=1e-14)

    def test_zero_branches_give_identity(self):
        rng = np.random.default_rng(12)
        p = _tiny_params(rng, self.H, self.F)
        for k in ("w_o", "b_o", "w_2", "b_2"):
            p[k] = np.zeros_like(p[k])
        x = rng.standard_normal((self.S, self.H))
        np.testing.assert_array_equal(oracle.block_forward_sequence(x, p, self.NH, 1e-5)["out"], x)

    def test_uniform_attention_is_prefix_mean_through_permuted_wo(self):
        # q = 0 -> all scores 0 -> uniform causal attention -> o_t = mean(v_0..v_t).
        # Wv = I and Wo = a cyclic shift (not symmetric), so a transposed Wo or a
        # misplaced head lands in the wrong columns.
        rng = np.random.default_rng(13)
        H = self.H
        p = _tiny_params(rng, H, self.F)
        p["w_qkv"][:, :H] = 0.0
        p["b_qkv"][:H] = 0.0
        p["w_qkv"][:, 2 * H:] = np.eye(H)
        p["b_qkv"][2 * H:] = 0.0
        shift = np.roll(np.eye(H), 1, axis=1)       # column j of out = column j-1 of in
        p["w_o"] = shift
        p["b_o"] = np.zeros(H)
        x = rng.standard_normal((self.S, H))
        r = oracle.block_forward_sequence(x, p, self.NH, 1e-5, keep=("a", "att"))
        prefix = np.cumsum(r["a"], axis=0) / np.arange(1, self.S + 1)[:, None]
        np.testing.assert_allclose(r["att"], np.roll(prefix, 1, axis=1), atol=1e-13)

    def test_score_scale_is_inverse_sqrt_head_dim(self):
        # q_t = c * e_0 (bias only), k_t picks a[t, 0] into head 0's first dim,
        # v = a: head 0 probabilities are softmax over s <= t of c*w*a[s,0]/sqrt(dh).
        rng = np.random.default_rng(14)
        H, NH = self.H, self.NH
        dh = H // NH
        p = _tiny_params(rng, H, self.F)
        c, w = 3.0, 2.0
        p["w_qkv"][:, :H] = 0.0
        p["b_qkv"][:H] = 0.0
        p["b_qkv"][0] = c
        p["w_qkv"][:, H:2 * H] = 0.0
        p["b_qkv"][H:2 * H] = 0.0
        p["w_qkv"][0, H] = w
        p["w_qkv"][:, 2 * H:] = np.eye(H)
        p["b_qkv"][2 * H:] = 0.0
        x = rng.standard_normal((self.S, H))
        r = oracle.block_forward_sequence(x, p, NH, 1e-5, keep=("a", "o"))
        a = r["a"]
        for t in range(self.S):
            logits = [c * w * a[s, 0] / math.sqrt(dh) for s in range(t + 1)]
            mx = max(logits)
            e = [math.exp(l - mx) for l in logits]
            z = sum(e)
            expect = sum(e[s] / z * a[s, :dh] for s in range(t + 1))
            np.testing.assert_allclose(r["o"][t, :dh], expect, atol=1e-13)

    def test_mlp_wiring(self):
        # attention branch off; W1 = [I | 0], W2 = [I ; 0]:
        # out = x + GELU(LN2(x) + b1[:H]) + b2  (b1 inside the activation)
        rng = np.random.default_rng(15)
        H, F = self.H, self.F
        p = _tiny_params(rng, H, F)
        p["w_o"][:] = 0.0
        p["b_o"][:] = 0.0
        p["w_1"] = np.zeros((H, F))
        p["w_1"][:, :H] = np.eye(H)
        p["b_1"] = rng.standard_normal(F)
        p["w_2"] = np.zeros((F, H))
        p["w_2"][:H, :] = np.eye(H)
        x = rng.standard_normal((self.S, H))
        ln, _ = oracle.layernorm_residual(x, None, p["ln2_gamma"], p["ln2_beta"], 1e-5)
        expect = x + oracle.gelu_erf(ln + p["b_1"][:H]) + p["b_2"]
        np.testing.assert_allclose(oracle.block_forward_sequence(x, p, self.NH, 1e-5)["out"],
                                   expect, atol=1e-14)

    def test_second_residual_carries_attention(self):
        # MLP branch off: out = h1 = x + att
        rng = np.random.default_rng(16)
        p = _tiny_params(rng, self.H, self.F)
        p["w_2"][:] = 0.0
        p["b_2"][:] = 0.0
        x = rng.standard_normal((self.S, self.H))
        r = oracle.block_forward_sequence(x, p, self.NH, 1e-5, keep=("att", "h1", "out"))
        assert np.abs(r["att"]).max() > 0.1
        np.testing.assert_allclose(r["out"], x + r["att"], atol=1e-14)
        np.testing.assert_array_equal(r["out"], r["h1"])

    def test_sequence_selection_of_a_batch(self):
        # block_forward(sequences=[3, 0]) stacks sequence 3, then sequence 0,
        # each as computed alone; attention never crosses sequences, so
        # changing sequence 1 changes nothing of them; the default is every
        # sequence in order
        rng = np.random.default_rng(17)
        p = _tiny_params(rng, self.H, self.F)
        x = rng.standard_normal((4, self.S, self.H))
        keep = ("a", "probs", "att", "out")
        sel = oracle.block_forward(x, p, self.NH, 1e-5, sequences=[3, 0], keep=keep)
        for k in keep:
            assert sel[k].shape[0] == 2
            for i, b in enumerate((3, 0)):
                alone = oracle.block_forward_sequence(x[b], p, self.NH, 1e-5, keep=(k,))[k]
                np.testing.assert_array_equal(sel[k][i], alone)
        x2 = x.copy()
        x2[1] = rng.standard_normal((self.S, self.H)) * 3
        sel2 = oracle.block_forward(x2, p, self.NH, 1e-5, sequences=[3, 0], keep=("out",))
        np.testing.assert_array_equal(sel2["out"], sel["out"])
        full = oracle.block_forward(x, p, self.NH, 1e-5)["out"]
        assert full.shape == (4, self.S, self.H)
        np.testing.assert_array_equal(full[[3, 0]], sel["out"])
        assert not np.allclose(full[1], full[2])


# ---------------------------------------------------------------------------
# RMSNorm + residual
# ---------------------------------------------------------------------------
class TestRMSNorm:
    def test_hand_example(self):
        # h = [3, 4]: mean square 12.5 -> y = h / sqrt(12.5) (no mean subtraction)
        y, _ = oracle.rmsnorm_residual(np.array([[3.0, 4.0]]), None, None, 0.0)
        np.testing.assert_allclose(y, [[3 / math.sqrt(12.5), 4 / math.sqrt(12.5)]], rtol=1e-15)

    def test_unit_rms_and_scale_invariance(self):
        rng = np.random.default_rng(20)
        h = rng.standard_normal((4, 64)) + 2.0
        y, _ = oracle.rmsnorm_residual(h, None, None, 0.0)
        np.testing.assert_allclose((y * y).mean(axis=1), 1.0, rtol=1e-14)
        y2, _ = oracle.rmsnorm_residual(5.0 * h, None, None, 0.0)
        np.testing.assert_allclose(y, y2, atol=1e-14)
        assert np.all(y.mean(axis=1) > 0.5)          # the mean is not removed

    def test_eps_gamma_and_residual(self):
        x = np.array([[1.0, 1.0, 1.0, 1.0]])
        y, h = oracle.rmsnorm_residual(x, -x + 2.0, np.array([1.0, 2.0, 3.0, 4.0]), 12.0)
        np.testing.assert_array_equal(h, 2.0)
        # mean square 4, eps 12 -> 2 / sqrt(16) = 0.5, times gamma
        np.testing.assert_allclose(y, [[0.5, 1.0, 1.5, 2.0]], rtol=1e-15)


# ---------------------------------------------------------------------------
# row reductions
# ---------------------------------------------------------------------------
class TestRowReduce:
    def test_closed_forms(self):
        x = np.arange(12, dtype=np.float64).reshape(3, 4)
        np.testing.assert_array_equal(oracle.row_reduce(x, "sum"), [6, 22, 38])
        np.testing.assert_array_equal(oracle.row_reduce(x, "mean"), [1.5, 5.5, 9.5])
        np.testing.assert_array_equal(oracle.row_reduce(x, "max"), [3, 7, 11])
        # sum of 1..n = n(n+1)/2 along the last axis only
        y = np.tile(np.arange(1, 101, dtype=np.float64), (2, 1))
        np.testing.assert_array_equal(oracle.row_reduce(y, "sum"), [5050, 5050])

    def test_argmax_ties_and_nan(self):
        x = np.array([[1.0, 3.0, 3.0, 2.0],        # tie -> lowest index
                      [-5.0, -5.0, -5.0, -5.0],     # all equal -> 0
                      [0.0, np.nan, 9.0, np.nan],   # first NaN
                      [-np.inf, -np.inf, -1.0, 7.0]])
        np.testing.assert_array_equal(oracle.row_argmax(x), [1, 0, 1, 3])

    def test_argmax_matches_brute_force_comparisons(self):
        rng = np.random.default_rng(21)
        x = rng.integers(-3, 4, size=(50, 17)).astype(np.float64)   # many ties
        got = oracle.row_argmax(x)
        for i in range(50):
            best = 0
            for j in range(1, 17):
                if x[i, j] > x[i, best]:
                    best = j
            assert got[i] == best


# ---------------------------------------------------------------------------
# layout transform
# ---------------------------------------------------------------------------
    def test_logsumexp_closed_forms(self):
        l3 = math.log(3.0)
        x = np.array([[0.0, l3, -np.inf],          # log(1 + 3) = log 4
                      [5.0, 5.0, 5.0],             # 5 + log 3
                      [1000.0, 1000.0, -1000.0],   # no overflow: 1000 + log 2
                      [-np.inf, -np.inf, -np.inf], # empty sum: -inf
                      [1.0, np.inf, 0.0],          # +inf
                      [np.nan, 0.0, 1.0]])         # NaN
        y = oracle.row_reduce(x, "logsumexp")
        np.testing.assert_allclose(y[:3], [math.log(4.0), 5.0 + l3, 1000.0 + math.log(2.0)],
                                   rtol=1e-15)
        assert y[3] == -np.inf and y[4] == np.inf and np.isnan(y[5])

    def test_logsumexp_shift_and_bounds(self):
        # lse(x + c) = lse(x) + c, and max <= lse <= max + log(cols)
        rng = np.random.default_rng(8)
        x = rng.standard_normal((6, 50)) * 4
        y = oracle.row_reduce(x, "logsumexp")
        np.testing.assert_allclose(oracle.row_reduce(x + 7.5, "logsumexp"), y + 7.5, rtol=1e-14)
        assert np.all(x.max(axis=1) <= y) and np.all(y <= x.max(axis=1) + math.log(50))

class TestStridedCopy:
    def test_head_split_is_a_numpy_transpose(self):
        # [tokens, 3, heads, dh] -> [3, heads, tokens, dh]; catches swapped
        # strides, a wrong source or destination batch stride
        t, nh, dh = 6, 4, 3
        src = np.arange(t * 3 * nh * dh, dtype=np.int64)
        got = oracle.strided_copy(src, np.zeros(src.size, np.int64), rows=t, cols=dh,
                                  batch=3 * nh, ld_src=3 * nh * dh, stride_src=dh, ld_dst=dh,
                                  stride_dst=t * dh)
        want = src.reshape(t, 3, nh, dh).transpose(1, 2, 0, 3).reshape(-1)
        np.testing.assert_array_equal(got, want)

    def test_split_then_merge_round_trips(self):
        t, nh, dh = 5, 3, 4
        h = nh * dh
        src = np.random.default_rng(4).standard_normal(t * h)
        heads = oracle.strided_copy(src, np.zeros(t * h), rows=t, cols=dh, batch=nh, ld_src=h,
                                    stride_src=dh, ld_dst=dh, stride_dst=t * dh)
        back = oracle.strided_copy(heads, np.zeros(t * h), rows=t, cols=dh, batch=nh,
                                   ld_src=dh, stride_src=t * dh, ld_dst=h, stride_dst=dh)
        np.testing.assert_array_equal(back, src)
        assert not np.array_equal(heads, src)              # the split really moved data

    def test_gaps_keep_their_values_and_bits(self):
        # padding between rows and batches is not written; bit patterns
        # (here including a NaN payload) are copied unchanged
        src = np.arange(1, 13, dtype=np.uint16)
        src[5] = 0x7FC1
        dst = np.full(40, 0xAAAA, dtype=np.uint16)
        got = oracle.strided_copy(src, dst, rows=2, cols=3, batch=2, ld_src=3, stride_src=6,
                                  ld_dst=5, stride_dst=20)
        want = dst.copy()
        for b in range(2):
            for r in range(2):
                for c in range(3):
                    want[b * 20 + r * 5 + c] = src[b * 6 + r * 3 + c]
        np.testing.assert_array_equal(got, want)
        assert got[39] == 0xAAAA and got[3] == 0xAAAA

    def test_zero_source_stride_broadcasts(self):
        src = np.array([7.0, 8.0])
        got = oracle.strided_copy(src, np.zeros(6), rows=1, cols=2, batch=3, ld_src=2,
                                  stride_src=0, ld_dst=2, stride_dst=2)
        np.testing.assert_array_equal(got, [7, 8, 7, 8, 7, 8])


# ---------------------------------------------------------------------------
# causal softmax trimmed to row blocks
# ---------------------------------------------------------------------------
class TestCausalWrittenWidth:
    def test_hand_worked_widths(self):
        # square, block 2: positions 0..5 write 2, 2, 4, 4, 6, 6 columns
        np.testing.assert_array_equal(oracle.causal_written_width(6, 6, 6, 2), [2, 2, 4, 4, 6, 6])
        # rows wrap every q_len rows (two heads of 3 positions)
        np.testing.assert_array_equal(oracle.causal_written_width(6, 3, 3, 2), [2, 2, 3, 2, 2, 3])
        # rectangular: 6 extra leading columns visible to every row
        np.testing.assert_array_equal(oracle.causal_written_width(4, 10, 4, 2), [8, 8, 10, 10])

    def test_special_blocks(self):
        # block 1 writes exactly the live columns (the causal limit + 1)
        rows, cols, q = 7, 9, 5
        live = (~oracle.causal_mask(rows, cols, q)).sum(axis=1)
        np.testing.assert_array_equal(oracle.causal_written_width(rows, cols, q, 1), live)
        # a block at least as long as the row writes every column
        np.testing.assert_array_equal(oracle.causal_written_width(5, 8, 5, 8), [8] * 5)

    def test_live_columns_always_written(self):
        for rows, cols, q, b in ((64, 64, 64, 16), (30, 40, 10, 4), (12, 5, 7, 2)):
            w = oracle.causal_written_width(rows, cols, q, b)
            live = ~oracle.causal_mask(rows, cols, q)
            last_live = np.where(live.any(axis=1), cols - 1 - np.argmax(live[:, ::-1], axis=1), -1)
            assert np.all(w > last_live)           # every live column lies below w
            assert np.all(w <= cols)
