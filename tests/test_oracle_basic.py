"""Pins of the fp64 reference checker: binary16 rounding, tree bookkeeping,
dequantisation / packing, GEMM, SwiGLU, RMSNorm and RoPE.

Every expectation here comes from something other than the checker itself:
numpy's binary16 conversion, brute-force enumeration, transitive closure by
boolean matrix products, numpy float64 matmul, or closed forms.
"""
import itertools

import numpy as np
import pytest

import gen
import oracle
from gen.workloads import CONFIGS


# --------------------------------------------------------------- binary16


def test_f16_decode_all_patterns_match_numpy():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = oracle.f16_array_to_f64(bits)
    fin = np.isfinite(ref)
    assert np.array_equal(got[fin], ref[fin])
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert np.array_equal(got[np.isinf(ref)], ref[np.isinf(ref)])


def _np_f16_bits(x):
    return np.asarray(x, dtype=np.float64).astype(np.float16).view(np.uint16)


def test_f16_round_matches_numpy_on_ties_subnormals_and_random():
    rng = np.random.default_rng(7)
    # exact midpoints between consecutive finite fp16 values (ties -> even)
    finite = np.arange(0, 0x7C00, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float64)
    mids = (finite[:-1] + finite[1:]) / 2
    vals = np.concatenate([
        mids, -mids[::97], finite, -finite[::53],
        rng.standard_normal(20000) * np.exp(rng.uniform(-25, 12, 20000)),
        np.nextafter(mids[::31], np.inf), np.nextafter(mids[::29], -np.inf),
        [0.0, -0.0, 65504.0, 65519.99, 65520.0, 1e6, -1e6, 2.0 ** -25, 2.0 ** -26, 2.0 ** -24,
         3 * 2.0 ** -26, np.inf, -np.inf],
    ])
    got = oracle.f64_array_to_f16(vals)
    ref = _np_f16_bits(vals)
    assert np.array_equal(got, ref)
    assert oracle.f64_to_f16(float("nan")) & 0x7C00 == 0x7C00


# ------------------------------------------------------------------- tree


def _all_increasing_trees(T):
    """Every parent array with parent[0] = -1 and 0 <= parent[i] < i."""
    for choice in itertools.product(*[range(i) for i in range(1, T)]):
        yield np.array((-1,) + choice, dtype=np.int32)


def _closure_reference(parent):
    """Ancestor-or-self matrix by transitive closure of the child->parent relation."""
    T = len(parent)
    A = np.eye(T, dtype=bool)
    for i in range(1, T):
        A[i, parent[i]] = True
    R = A.copy()
    for _ in range(T):
        R = (R.astype(np.int64) @ A.astype(np.int64)) > 0
    return R


@pytest.mark.parametrize("T", [1, 2, 3, 4, 5, 6, 7])
def test_tree_exhaustive_vs_transitive_closure(T):
    for parent in _all_increasing_trees(T):
        depth, anc = oracle.tree(parent)
        R = _closure_reference(parent)
        assert np.array_equal(anc.astype(bool), R)
        # depth = number of strict ancestors
        assert np.array_equal(depth, R.sum(axis=1) - 1)


def test_tree_chain_mask_is_lower_triangular():
    for T in (1, 2, 8, 64):
        parent = np.arange(-1, T - 1, dtype=np.int32)
        depth, anc = oracle.tree(parent)
        assert np.array_equal(anc, np.tril(np.ones((T, T), np.uint8)))
        assert np.array_equal(depth, np.arange(T))


@pytest.mark.parametrize("parent", [[0], [-1, 1], [-1, 0, 3], [-1, -1], [-1, 0, 2], [5, -1]])
def test_tree_rejects_invalid_parent_arrays(parent):
    assert not oracle.tree_valid(parent)
    with pytest.raises(ValueError):
        oracle.tree(parent)


@pytest.mark.parametrize("name", list(CONFIGS))
def test_generated_trees_have_the_configured_shape(name):
    cfg = CONFIGS[name]
    parent, accepted = gen.workloads.make_tree(cfg)
    depth, anc = oracle.tree(parent)
    assert len(parent) == cfg.T
    assert depth.max() + 1 == cfg.levels
    children = np.bincount(parent[1:], minlength=cfg.T)
    assert children.max() <= cfg.branching
    assert children[accepted] == 0  # a leaf
    if cfg.deepest_leaf:
        assert depth[accepted] + 1 == cfg.levels


# ------------------------------------------------------------ dequant/GEMM


def _pack(qint):
    """Boundary packing: two nibbles per byte, low nibble = even k."""
    qint = np.asarray(qint, np.uint8)
    return (qint[:, 0::2] | (qint[:, 1::2] << 4)).astype(np.uint8)


def _make_w(qint, scales_f, zeros):
    N, K = qint.shape
    return {"qweight": _pack(qint), "scales": _np_f16_bits(scales_f).reshape(N, K // 128),
            "zeros": np.asarray(zeros, np.uint8).reshape(N, K // 128), "K": K, "N": N}


def _dense(qint, scales_f, zeros):
    N, K = qint.shape
    s = np.repeat(np.asarray(scales_f, np.float16).astype(np.float64).reshape(N, K // 128), 128, axis=1)
    z = np.repeat(np.asarray(zeros, np.float64).reshape(N, K // 128), 128, axis=1)
    return (qint.astype(np.float64) - z) * s


def _rand_w(rng, N, K):
    qint = rng.integers(0, 16, size=(N, K))
    sc = rng.uniform(0.002, 0.05, size=(N, K // 128))
    zz = rng.integers(0, 16, size=(N, K // 128))
    return qint, sc, zz


def test_gemm_one_hot_rows_reproduce_dequantised_columns_exactly():
    rng = np.random.default_rng(1)
    N, K = 24, 256
    qint, sc, zz = _rand_w(rng, N, K)
    W = _make_w(qint, sc, zz)
    ks = [0, 1, 2, 3, 127, 128, 129, 254, 255]
    x = np.zeros((len(ks), K), np.float16)
    for m, k0 in enumerate(ks):
        x[m, k0] = 1.0
    y = oracle.w4a16_gemm(W, x.view(np.uint16))
    dense = _dense(qint, sc, zz)
    for m, k0 in enumerate(ks):
        assert np.array_equal(y[m], _np_f16_bits(dense[:, k0]))
        for n in range(N):
            assert oracle.dequant(W, n, k0) == dense[n, k0]


def test_gemm_zero_when_q_equals_zero_point():
    rng = np.random.default_rng(2)
    N, K = 16, 384
    zz = rng.integers(0, 16, size=(N, K // 128))
    qint = np.repeat(zz, 128, axis=1)
    W = _make_w(qint, rng.uniform(0.01, 0.1, size=(N, K // 128)), zz)
    x = gen.normal_f16(5, 0, (7, K))
    y = oracle.w4a16_gemm(W, x)
    assert np.all(y.view(np.float16) == 0)


@pytest.mark.parametrize("M,N,K", [(1, 8, 128), (5, 17, 256), (16, 33, 512)])
def test_gemm_matches_numpy_float64(M, N, K):
    rng = np.random.default_rng(M * 100 + N)
    qint, sc, zz = _rand_w(rng, N, K)
    W = _make_w(qint, sc, zz)
    x = gen.normal_f16(11, M, (M, K))
    r = gen.normal_f16(12, M, (M, N))
    ref = x.view(np.float16).astype(np.float64) @ _dense(qint, sc, zz).T
    y = oracle.w4a16_gemm(W, x)
    yr = oracle.w4a16_gemm(W, x, residual=r)
    ref_b = _np_f16_bits(ref)
    ref_rb = _np_f16_bits(ref + r.view(np.float16).astype(np.float64))
    # fp64 sums in a different order may flip a rounding tie; allow one ulp
    for got, exp in ((y, ref_b), (yr, ref_rb)):
        diff = np.abs(got.astype(np.int32) - exp.astype(np.int32))
        assert diff.max() <= 1
        assert (diff == 0).mean() > 0.99


def test_gemm_is_exactly_homogeneous_under_power_of_two_scaling():
    rng = np.random.default_rng(3)
    qint, sc, zz = _rand_w(rng, 32, 256)
    W = _make_w(qint, sc, zz)
    x = gen.normal_f16(13, 0, (4, 256))
    y1 = oracle.w4a16_gemm(W, x).view(np.float16).astype(np.float64)
    x2 = (x.view(np.float16).astype(np.float64) * 2).astype(np.float16).view(np.uint16)
    y2 = oracle.w4a16_gemm(W, x2).view(np.float16).astype(np.float64)
    assert np.array_equal(2 * y1, y2)


def test_generator_quantiser_error_is_within_half_a_step():
    w = gen.normal_f16(21, 0, (64, 512), 0.0, 0.02)
    q, s, z = gen.quantize_w4(w)
    qint = np.empty((64, 512), np.int64)
    qint[:, 0::2] = q & 15
    qint[:, 1::2] = q >> 4
    dense = _dense(qint, s.view(np.float16).astype(np.float64), z)
    wf = w.view(np.float16).astype(np.float64)
    step = np.repeat(s.view(np.float16).astype(np.float64), 128, axis=1)
    assert np.all(np.abs(dense - wf) <= 0.5 * step * (1 + 1e-12) + 1e-12)
    assert q.dtype == np.uint8 and z.max() <= 15


def test_swiglu_matches_numpy_and_closed_forms():
    rng = np.random.default_rng(4)
    N, K, M = 40, 256, 6
    qg, sg, zg = _rand_w(rng, N, K)
    qu, su, zu = _rand_w(rng, N, K)
    Wg, Wu = _make_w(qg, sg, zg), _make_w(qu, su, zu)
    x = gen.normal_f16(31, 0, (M, K))
    xf = x.view(np.float16).astype(np.float64)
    g = xf @ _dense(qg, sg, zg).T
    u = xf @ _dense(qu, su, zu).T
    ref = _np_f16_bits(g / (1 + np.exp(-g)) * u)
    y = oracle.w4a16_swiglu(Wg, Wu, x)
    diff = np.abs(y.astype(np.int32) - ref.astype(np.int32))
    assert diff.max() <= 1 and (diff == 0).mean() > 0.99
    # silu(0) = 0: a zero gate (q = z) gives an exactly zero output
    Wg0 = _make_w(np.repeat(zg, 128, axis=1), sg, zg)
    assert np.all(oracle.w4a16_swiglu(Wg0, Wu, x).view(np.float16) == 0)


# ---------------------------------------------------------------- RMSNorm


def test_rmsnorm_constant_vector_closed_form():
    H = 256
    gamma = gen.normal_f16(41, 0, (H,), 1.0, 0.02)
    gf = gamma.view(np.float16).astype(np.float64)
    for c in (1.0, -3.5, 0.125, 0.0):
        x = np.full((1, H), c, np.float16).view(np.uint16)
        y = oracle.rmsnorm(x, gamma, eps=1e-5)
        expected = _np_f16_bits(c / np.sqrt(c * c + 1e-5) * gf)
        assert np.array_equal(y[0], expected)


def test_rmsnorm_matches_numpy():
    x = gen.normal_f16(42, 0, (9, 512))
    gamma = gen.normal_f16(43, 0, (512,), 1.0, 0.02)
    xf = x.view(np.float16).astype(np.float64)
    ref = xf / np.sqrt((xf * xf).mean(axis=1, keepdims=True) + 1e-5) * gamma.view(np.float16).astype(np.float64)
    diff = np.abs(oracle.rmsnorm(x, gamma).astype(np.int32) - _np_f16_bits(ref).astype(np.int32))
    assert diff.max() <= 1 and (diff == 0).mean() > 0.99


# ------------------------------------------------------------------- RoPE


def test_rope_position_zero_is_identity_and_norms_are_preserved():
    rng = np.random.default_rng(5)
    for D in (64, 128):
        v = rng.standard_normal(D)
        assert np.array_equal(oracle.rope(v, 0), v)
        for pos in (1, 17, 4096, 32831):
            r = oracle.rope(v, pos)
            h = D // 2
            assert np.allclose(r[:h] ** 2 + r[h:] ** 2, v[:h] ** 2 + v[h:] ** 2, rtol=1e-12, atol=1e-12)


def test_rope_pairs_d_with_d_plus_half_and_uses_theta_frequencies():
    D, theta = 8, 500000.0
    for pos in (1, 3, 1000):
        e0 = np.zeros(D)
        e0[0] = 1.0
        r = oracle.rope(e0, pos, theta)
        exp = np.zeros(D)
        exp[0], exp[4] = np.cos(pos), np.sin(pos)  # frequency 1 for d = 0
        assert np.allclose(r, exp, atol=1e-12)
        e3 = np.zeros(D)
        e3[3 + 4] = 1.0
        r = oracle.rope(e3, pos, theta)
        f = theta ** (-6.0 / 8.0)
        exp = np.zeros(D)
        exp[3], exp[7] = -np.sin(pos * f), np.cos(pos * f)
        assert np.allclose(r, exp, atol=1e-12)


def test_rope_scores_depend_only_on_relative_position():
    rng = np.random.default_rng(6)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    base = oracle.rope(q, 10) @ oracle.rope(k, 3)
    for shift in (1, 100, 4000):
        assert abs(oracle.rope(q, 10 + shift) @ oracle.rope(k, 3 + shift) - base) < 1e-9


# ---------------------------------------------------------------- LM head


def test_lm_head_matches_numpy_on_a_non_square_head():
    # logits = fp16(fp16(rmsnorm(h) * gamma) @ W^T) with W stored [V][H]: a
    # head read as [H][V], or a skipped normalisation, changes every value
    M, H, V = 5, 256, 48
    h = gen.normal_f16(44, 0, (M, H), 0.0, 3.0)
    gamma = gen.normal_f16(45, 0, (H,), 1.0, 0.02)
    W = gen.normal_f16(46, 0, (V, H), 0.0, 0.02)
    hf = h.view(np.float16).astype(np.float64)
    xn = hf / np.sqrt((hf * hf).mean(axis=1, keepdims=True) + 1e-5) * gamma.view(np.float16).astype(np.float64)
    xn16 = xn.astype(np.float16).astype(np.float64)
    ref = _np_f16_bits(xn16 @ W.view(np.float16).astype(np.float64).T)
    got = oracle.lm_head(h, gamma, W)
    assert got.shape == (M, V)
    diff = np.abs(got.astype(np.int32) - ref.astype(np.int32))
    assert diff.max() <= 1 and (diff == 0).mean() > 0.95


def test_lm_head_one_hot_row_reads_one_column_of_the_head():
    # a row a * e_k normalises to c * e_k, c = fp16(a / sqrt(a^2 / H + eps))
    # (gamma = 1), so its logits are exactly fp16(c * W[:, k])
    H, V = 256, 40
    W = gen.normal_f16(47, 0, (V, H), 0.0, 0.5)
    gamma = np.full(H, 1.0, np.float16).view(np.uint16)
    wf = W.view(np.float16).astype(np.float64)
    for k, a in ((0, 1.0), (37, -2.5), (255, 0.75)):
        h = np.zeros((1, H), np.float16)
        h[0, k] = a
        c = np.float64(np.float16(a / np.sqrt(a * a / H + 1e-5)))
        got = oracle.lm_head(h.view(np.uint16), gamma, W)
        assert np.array_equal(got[0], _np_f16_bits(c * wf[:, k]))
