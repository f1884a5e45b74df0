"""GPU parity of the individual kernels against the fp64 reference checker.

Bit-exact: device tree masks / depths, KV commit (every cache byte), values
copied into the cache.  Tolerance |gpu - ref| <= 2e-3 + 1e-2 |ref| (fp16
outputs): W4A16 GEMM, SwiGLU, RMSNorm, tree attention, rotated keys.
"""
import itertools

import numpy as np
import pytest

import gen
import oracle
from gen.workloads import CONFIGS, LLAMA_1B, LLAMA_8B, LLAMA_70B

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2506_11309_amd as ss
    ss.lib()
    torch.cuda.set_device(0)


import paper_2506_11309_amd as ss  # noqa: E402
from gpu_helpers import check_close, dev, down16, up, upload_w4  # noqa: E402


# ------------------------------------------------------------- tree masks


def _all_trees(T):
    for choice in itertools.product(*[range(i) for i in range(1, T)]):
        yield (-1,) + choice


def test_tree_masks_exhaustive_T8_bit_exact():
    T = 8
    parents = np.array(list(_all_trees(T)), np.int32)  # 5040 trees
    n = len(parents)
    anc = torch.zeros((n, T), dtype=torch.int64, device=dev())
    depth = torch.zeros((n, T), dtype=torch.int32, device=dev())
    status = torch.full((n,), -7, dtype=torch.int32, device=dev())
    ss.tree_masks(up(parents), anc, depth, status)
    torch.cuda.synchronize()
    a = anc.cpu().numpy().view(np.uint64)
    d = depth.cpu().numpy()
    assert np.all(status.cpu().numpy() == 0)
    for t in range(n):
        od, oa = oracle.tree(parents[t])
        bits = (oa.astype(np.uint64) << np.arange(T, dtype=np.uint64)[None, :]).sum(axis=1)
        assert np.array_equal(a[t], bits), parents[t]
        assert np.array_equal(d[t], od)


def test_tree_masks_large_random_and_invalid():
    rng = np.random.default_rng(3)
    rows = []
    for T in (64,):
        for k in range(200):
            p = np.array([-1] + [int(rng.integers(0, i)) for i in range(1, T)], np.int32)
            rows.append(p)
    rows.append(np.arange(-1, 63, dtype=np.int32))  # depth-63 chain
    bad = np.arange(-1, 63, dtype=np.int32).copy()
    bad[10] = 12  # parent after child
    rows.append(bad)
    bad2 = np.arange(-1, 63, dtype=np.int32).copy()
    bad2[0] = 0
    rows.append(bad2)
    parents = np.stack(rows)
    n, T = parents.shape
    anc = torch.zeros((n, T), dtype=torch.int64, device=dev())
    depth = torch.zeros((n, T), dtype=torch.int32, device=dev())
    status = torch.full((n,), -7, dtype=torch.int32, device=dev())
    ss.tree_masks(up(parents), anc, depth, status)
    torch.cuda.synchronize()
    a = anc.cpu().numpy().view(np.uint64)
    d = depth.cpu().numpy()
    st = status.cpu().numpy()
    for t in range(n - 2):
        od, oa = oracle.tree(parents[t])
        bits = np.zeros(T, np.uint64)
        for j in range(T):
            bits |= (oa[:, j].astype(np.uint64) << np.uint64(j))
        assert st[t] == 0 and np.array_equal(a[t], bits) and np.array_equal(d[t], od)
    assert st[-2] == ss.DEVERR_BAD_TREE and st[-1] == ss.DEVERR_BAD_TREE
    # invalid trees: self bit only, depth 0
    assert np.array_equal(a[-1], (np.uint64(1) << np.arange(T, dtype=np.uint64)))
    assert np.all(d[-1] == 0)


# --------------------------------------------------------------- commit


@pytest.mark.parametrize("name,n_layers", [("c1", 1), ("c2", 1), ("c3", 1), ("c4", 1), ("c5", 4)])
def test_kv_commit_bit_exact_all_configs(name, n_layers):
    cfg = CONFIGS[name]
    s = cfg.shape
    parent, acc = gen.workloads.make_tree(cfg)
    shape = (n_layers, s.Hkv, cfg.S_max, s.D)
    k = gen.normal_f16(77, 0, shape)
    v = gen.normal_f16(77, 1, shape)
    dk, dv = up(k), up(v)
    P = up(np.array([cfg.P], np.int32))
    ws = ss.workspace(ss.WS_HEADER_BYTES, dev())
    ss.kv_commit(dk, dv, P, up(parent), up(np.array([acc], np.int32)), n_layers=n_layers, advance=True,
                 ws=ws)
    torch.cuda.synchronize()
    L = oracle.kv_commit(k, v, cfg.P, parent, acc, n_layers=n_layers)
    assert np.array_equal(down16(dk), k)
    assert np.array_equal(down16(dv), v)
    assert int(P.item()) == cfg.P + L
    assert ss.read_device_error(ws) == 0
    if cfg.deepest_leaf:
        assert L == cfg.levels


def test_kv_commit_full_80_layer_cache():
    cfg = CONFIGS["c5"]
    s = cfg.shape
    parent, acc = gen.workloads.make_tree(cfg)
    # random bytes stand in for cache contents (the commit is a pure move)
    shape = (cfg.n_layers, s.Hkv, cfg.S_max, s.D)
    n = int(np.prod(shape))
    k = gen.u64(91, 0, n // 4).view(np.uint16).reshape(shape)
    v = gen.u64(91, 1, n // 4).view(np.uint16).reshape(shape)
    dk, dv = up(k), up(v)
    P = up(np.array([cfg.P], np.int32))
    ss.kv_commit(dk, dv, P, up(parent), up(np.array([acc], np.int32)), n_layers=cfg.n_layers)
    torch.cuda.synchronize()
    oracle.kv_commit(k, v, cfg.P, parent, acc, n_layers=cfg.n_layers)
    assert np.array_equal(down16(dk), k)
    assert np.array_equal(down16(dv), v)
    assert int(P.item()) == cfg.P  # advance off


def test_kv_commit_edge_cases_and_device_errors():
    Hkv, D, T = 2, 128, 64
    for P0, S_max in ((0, 64), (100, 164)):  # empty prefix, cache exactly full
        parent = np.arange(-1, T - 1, dtype=np.int32)
        for acc in (0, T - 1, 17):
            k = gen.normal_f16(5, acc, (Hkv, S_max, D))
            v = gen.normal_f16(6, acc, (Hkv, S_max, D))
            dk, dv = up(k), up(v)
            P = up(np.array([P0], np.int32))
            ss.kv_commit(dk, dv, P, up(parent), up(np.array([acc], np.int32)), advance=True)
            torch.cuda.synchronize()
            oracle.kv_commit(k, v, P0, parent, acc)
            assert np.array_equal(down16(dk), k) and np.array_equal(down16(dv), v)
            assert int(P.item()) == P0 + acc + 1
    # invalid accepted node / prefix / tree: nothing moves, error word set
    k = gen.normal_f16(8, 0, (Hkv, 80, D))
    parent = np.arange(-1, 8 - 1, dtype=np.int32)
    for acc, P0, par, bit in ((8, 10, parent, ss.DEVERR_BAD_ACCEPTED), (3, 73, parent, ss.DEVERR_BAD_PREFIX),
                              (3, 10, np.array([-1, 0, 5, 1, 1, 1, 1, 1], np.int32), ss.DEVERR_BAD_TREE)):
        dk, dv = up(k), up(k)
        P = up(np.array([P0], np.int32))
        ws = ss.workspace(ss.WS_HEADER_BYTES, dev())
        ss.kv_commit(dk, dv, P, up(par), up(np.array([acc], np.int32)), advance=True, ws=ws)
        err = ss.read_device_error(ws)
        assert err & bit
        assert np.array_equal(down16(dk), k) and int(P.item()) == P0


# ----------------------------------------------------------------- GEMM


def _rand_w4(seed, N, K):
    q, s, z = gen.w4_random(seed, 0, N, K, std=0.02)
    return {"qweight": q, "scales": s, "zeros": z, "K": K, "N": N}


def _gemm_case(M, K, N, seed, residual):
    W = _rand_w4(seed, N, K)
    x = gen.normal_f16(seed, 1, (M, K))
    r = gen.normal_f16(seed, 2, (M, N)) if residual else None
    t, d = upload_w4(W)
    dx = up(x)
    dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
    ws = ss.workspace(ss.gemm_workspace_bytes(M, K, N), dev())
    ss.w4a16_gemm(d, dx, dy, ws, residual=up(r) if residual else None)
    torch.cuda.synchronize()
    ref = oracle.w4a16_gemm(W, x, residual=r)
    return check_close(down16(dy), ref, f"gemm M={M} K={K} N={N}")


@pytest.mark.parametrize("M", [1, 8, 13, 16, 32, 40, 64])
def test_w4a16_gemm_small_shapes_ragged_M(M):
    _gemm_case(M, 1024, 320, seed=M, residual=(M % 2 == 0))


@pytest.mark.parametrize("M,K,N", [(1, 1024, 2048), (5, 1920, 2048), (8, 2048, 3072), (13, 8192, 2048),
                                   (16, 4096, 4096), (16, 1152, 4096)])
def test_w4a16_gemm_k_split_workgroups(M, K, N):
    """Up to 16 rows and at most 32 MB of weights (the 8B down projection,
    29 MB, runs in the config-shape test): one workgroup per column tile, 4
    (K < 2048) or 8 waves splitting K into unequal group ranges where G is
    not a multiple of the wave count (K = 1152, 1920), partials added in wave
    order; with and without residual, ragged M."""
    _gemm_case(M, K, N, seed=M * 7 + K, residual=(M % 2 == 1))


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4"])
def test_w4a16_gemm_config_shapes(name):
    cfg = CONFIGS[name]
    s = cfg.shape
    M = cfg.T
    for K, N in ((s.H, s.n_qkv), (s.Hq * s.D, s.H), (s.F, s.H)):
        _gemm_case(M, K, N, seed=1000 + K + N, residual=True)


def test_w4a16_gemm_deterministic_and_split_consistent():
    K, N, M = 8192, 1024, 32
    W = _rand_w4(9, N, K)
    x = gen.normal_f16(9, 1, (M, K))
    t, d = upload_w4(W)
    dx = up(x)
    outs = []
    for _ in range(3):
        dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
        ws = ss.workspace(ss.gemm_workspace_bytes(M, K, N), dev())
        ss.w4a16_gemm(d, dx, dy, ws)
        torch.cuda.synchronize()
        outs.append(down16(dy))
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])
    check_close(outs[0], oracle.w4a16_gemm(W, x), "gemm det")


@pytest.mark.parametrize("M,K,N,swiglu", [(32, 8192, 10240, False), (13, 2048, 4096, False), (64, 4096, 14336, True)])
def test_w4a16_split_blocks_reuse_one_workspace(M, K, N, swiglu):
    """Column blocks split between workgroups (partials summed in workgroup
    order): five calls on one workspace give bit-identical results within
    tolerance of the oracle and leave the workspace header zero."""
    W = _rand_w4(17, N, K)
    t, d = upload_w4(W)
    x = gen.normal_f16(17, 1, (M, K))
    dx = up(x)
    if swiglu:
        Wu = _rand_w4(18, N, K)
        tu, du = upload_w4(Wu)
        ws = ss.workspace(ss.swiglu_workspace_bytes(M, K, N), dev())
        ref = oracle.w4a16_swiglu(W, Wu, x)
    else:
        r = gen.normal_f16(17, 2, (M, N))
        ws = ss.workspace(ss.gemm_workspace_bytes(M, K, N), dev())
        ref = oracle.w4a16_gemm(W, x, residual=r)
    outs = []
    for _ in range(5):
        dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
        if swiglu:
            ss.w4a16_swiglu(d, du, dx, dy, ws)
        else:
            ss.w4a16_gemm(d, dx, dy, ws, residual=up(r))
        torch.cuda.synchronize()
        outs.append(down16(dy))
        header = ws[:ss.WS_HEADER_BYTES].cpu().numpy()
        assert not header.any(), "workspace header not left zero"
    for o in outs[1:]:
        assert np.array_equal(outs[0], o)
    check_close(outs[0], ref, f"split blocks M={M} K={K} N={N}")


@pytest.mark.parametrize("name", ["c1", "c3"])
def test_w4a16_swiglu_config_shapes(name):
    cfg = CONFIGS[name]
    s = cfg.shape
    M, K, N = cfg.T, s.H, s.F if name == "c1" else 4096
    Wg, Wu = _rand_w4(11, N, K), _rand_w4(12, N, K)
    x = gen.normal_f16(13, 0, (M, K))
    tg, dg = upload_w4(Wg)
    tu, du = upload_w4(Wu)
    dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
    ws = ss.workspace(ss.swiglu_workspace_bytes(M, K, N), dev())
    ss.w4a16_swiglu(dg, du, up(x), dy, ws)
    torch.cuda.synchronize()
    check_close(down16(dy), oracle.w4a16_swiglu(Wg, Wu, x), f"swiglu {name}")


def _w4_rows(W, rows):
    """The int4 matrix restricted to output rows (columns of y) `rows`."""
    return {"qweight": W["qweight"][rows], "scales": W["scales"][rows], "zeros": W["zeros"][rows],
            "K": W["K"], "N": len(rows)}


@pytest.mark.parametrize("M", [32, 9, 64, 47])
def test_w4a16_swiglu_70b_width(M):
    """SwiGLU at the 70B FFN width (K = 8192, N = 28672), checked against the
    oracle on every column of four 112-column stretches (first, second, a
    middle one, last) and on 256 random columns."""
    K, N = 8192, 28672
    Wg, Wu = _rand_w4(21, N, K), _rand_w4(22, N, K)
    x = gen.normal_f16(23, 0, (M, K))
    tg, dg = upload_w4(Wg)
    tu, du = upload_w4(Wu)
    dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
    ws = ss.workspace(ss.swiglu_workspace_bytes(M, K, N), dev())
    ss.w4a16_swiglu(dg, du, up(x), dy, ws)
    torch.cuda.synchronize()
    y = down16(dy)
    blk = 7 * 16
    cols = np.concatenate([np.arange(b * blk, (b + 1) * blk) for b in (0, 1, 128, N // blk - 1)]
                          + [np.random.default_rng(24).choice(N, 256, replace=False)])
    ref = oracle.w4a16_swiglu(_w4_rows(Wg, cols), _w4_rows(Wu, cols), x)
    check_close(y[:, cols], ref, f"swiglu 70b width M={M}")


def _swiglu_sampled_case(M, K, N, seed):
    """Two calls agree bit for bit; sampled columns (the first and last 64,
    256 random ones) against the oracle."""
    Wg, Wu = _rand_w4(seed, N, K), _rand_w4(seed + 1, N, K)
    x = gen.normal_f16(33, M, (M, K))
    tg, dg = upload_w4(Wg)
    tu, du = upload_w4(Wu)
    outs = []
    for _ in range(2):
        dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
        ws = ss.workspace(ss.swiglu_workspace_bytes(M, K, N), dev())
        ss.w4a16_swiglu(dg, du, up(x), dy, ws)
        torch.cuda.synchronize()
        outs.append(down16(dy))
    assert np.array_equal(outs[0], outs[1])
    cols = np.concatenate([np.arange(64), np.arange(N - 64, N),
                           np.random.default_rng(34).choice(np.arange(64, N - 64), 256, replace=False)])
    ref = oracle.w4a16_swiglu(_w4_rows(Wg, cols), _w4_rows(Wu, cols), x)
    check_close(outs[0][:, cols], ref, f"swiglu M={M} K={K} N={N}")


@pytest.mark.parametrize("M,K,N", [(1, 4096, 14336), (8, 2048, 8192), (5, 8192, 7168), (8, 1152, 2048),
                                   (3, 1920, 4096)])
def test_w4a16_swiglu_k_split_workgroups(M, K, N):
    """Fused SwiGLU at up to 8 rows and at most 32 MB per matrix (the 1B FFN,
    the 8B FFN at one row, one GPU's share of the 70B FFN under 4-way tensor
    parallelism): one workgroup per column tile reads its gate and up tiles,
    4 waves split K (unequal group ranges at K = 1152 and 1920)."""
    _swiglu_sampled_case(M, K, N, seed=41 + M)


@pytest.mark.parametrize("M,K,N", [(16, 4096, 14336), (9, 4096, 14336), (17, 4096, 14336), (32, 4096, 14336),
                                   (9, 2048, 8192), (31, 2048, 8192)])
def test_w4a16_swiglu_two_column_blocks(M, K, N):
    """SwiGLU at the 8B and 1B FFN widths above 8 rows, where the gate and
    up tiles of a column run in different waves of one workgroup: sampled
    columns (the first and last 64, 256 random ones) against the oracle, and
    two calls agree bit for bit."""
    _swiglu_sampled_case(M, K, N, seed=31 + M)


@pytest.mark.parametrize("M,K,N,ldx,swiglu", [
    # norm inside the K-split GEMM: 2 groups per wave, then up to 4
    (8, 2048, 3072, 2048, False), (1, 2048, 3072, 2048, False), (6, 1024, 2048, 1032, False),
    (8, 1152, 2048, 1280, False), (5, 1920, 2048, 1920, False), (13, 4096, 6144, 4096, False),
    (16, 1152, 2048, 1288, False), (16, 4096, 4096, 4096, False),
    # norm kernel, then the K-split GEMM (8 and 16 groups per wave)
    (7, 8192, 2560, 8192, False), (3, 16384, 2048, 16384, False),
    (17, 2048, 3072, 2048, False), (32, 8192, 1024, 8200, False),  # norm kernel, then stream-K
    (4, 1024, 2048, 1024, True), (8, 2048, 8192, 2048, True), (3, 1920, 4096, 2056, True),  # in the SwiGLU
    (9, 2048, 8192, 2048, True)])                                  # norm kernel, then the SwiGLU
def test_rmsnorm_then_projection_matches_oracle(M, K, N, ldx, swiglu):
    """RMSNorm followed by the QKV-style projection or the fused SwiGLU,
    against the reference's fp16 rmsnorm then its fp64 product: where each
    workgroup holds all of K and each wave at most 4 groups the norm runs
    inside the GEMM (row sums first, then the operand normalised as the
    norm kernel does it; each row's 16-byte chunks loaded in a
    row-dependent order), else as its own kernel; both within the GEMM
    tolerance, with strided rows (ldx > K, also not a multiple of 16 bytes
    apart), ragged M and unequal K ranges per wave (K = 1152, 1920); two
    calls agree bit for bit."""
    seed = 50 + M + K % 1000
    x = gen.normal_f16(seed, 0, (M, ldx), 0.0, 2.0)
    gamma = gen.normal_f16(seed, 1, (K,), 1.0, 0.2)
    W = _rand_w4(seed + 1, N, K)
    t, d = upload_w4(W)
    xn = oracle.rmsnorm(np.ascontiguousarray(x[:, :K]), gamma)
    if swiglu:
        Wu = _rand_w4(seed + 2, N, K)
        tu, du = upload_w4(Wu)
        ws = ss.workspace(ss.swiglu_workspace_bytes(M, K, N), dev())
        ref = oracle.w4a16_swiglu(W, Wu, xn)
    else:
        ws = ss.workspace(ss.gemm_workspace_bytes(M, K, N), dev())
        ref = oracle.w4a16_gemm(W, xn)
    dx, dg = up(x), up(gamma)
    outs = []
    for _ in range(2):
        dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
        if swiglu:
            ss.rmsnorm_w4a16_swiglu(d, du, dx, dg, dy, ws)
        else:
            ss.rmsnorm_w4a16_gemm(d, dx, dg, dy, ws)
        torch.cuda.synchronize()
        outs.append(down16(dy))
    assert np.array_equal(outs[0], outs[1])
    check_close(outs[0], ref, f"rmsnorm then {'swiglu' if swiglu else 'gemm'} M={M} K={K} N={N}")
    # the normalised operand is rounded where the two-kernel chain rounds it
    # (fp16 of (x * inv) * gamma): against the norm kernel followed by the
    # plain entry point the outputs differ only through the last bits of
    # inv (an fp16 ulp of a rare normalised value, or of an output), far
    # inside what rounding x * gamma instead would produce
    xn_d = torch.zeros((M, K), dtype=torch.int16, device=dev())
    ss.rmsnorm(dx[:, :K], dg, xn_d)
    dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
    if swiglu:
        ss.w4a16_swiglu(d, du, xn_d, dy, ws)
    else:
        ss.w4a16_gemm(d, xn_d, dy, ws)
    torch.cuda.synchronize()
    chain = down16(dy).view(np.float16).astype(np.float64)
    diff = np.abs(outs[0].view(np.float16).astype(np.float64) - chain)
    assert np.all(diff <= 5e-4 + 1e-3 * np.abs(chain)), diff.max()


@pytest.mark.parametrize("M,K,N", [(1, 1024, 1024), (8, 2048, 512), (13, 1024, 2048), (32, 8192, 1024),
                                   (40, 4096, 1024), (64, 2048, 1024)])
def test_w4a16_gemm_valu_variant_matches_oracle(M, K, N):
    """The vector-ALU comparison variant computes the same product (with a
    residual) within the tolerance, deterministically."""
    W = _rand_w4(21 + M, N, K)
    x = gen.normal_f16(21, M, (M, K))
    res = gen.normal_f16(22, M, (M, N))
    t, d = upload_w4(W)
    outs = []
    for _ in range(2):
        dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
        ws = ss.workspace(ss.gemm_valu_workspace_bytes(M, K, N), dev())
        ss.w4a16_gemm_valu(d, up(x), dy, ws, residual=up(res))
        torch.cuda.synchronize()
        outs.append(down16(dy))
    assert np.array_equal(outs[0], outs[1])
    err, rel = check_close(outs[0], oracle.w4a16_gemm(W, x, residual=res), f"valu gemm M={M} K={K} N={N}")
    print(f"valu gemm M={M} K={K} N={N}: max abs err {err:.3g}, rel {rel:.3g}")


def test_w4a16_gemm_rejects_bad_arguments():
    W = _rand_w4(1, 64, 256)
    t, d = upload_w4(W)
    ws = ss.workspace(ss.gemm_workspace_bytes(8, 256, 64), dev())
    x = torch.zeros((65, 256), dtype=torch.int16, device=dev())
    y = torch.zeros((65, 64), dtype=torch.int16, device=dev())
    with pytest.raises(ss.SwiftSpecError) as e:
        ss.w4a16_gemm(d, x, y, ws)
    assert e.value.status == ss.UNSUPPORTED
    small = ss.workspace(1024, dev())
    with pytest.raises(ss.SwiftSpecError) as e:
        ss.w4a16_gemm(d, x[:8], y[:8], small)
    assert e.value.status == ss.WORKSPACE_TOO_SMALL


# -------------------------------------------------------------- RMSNorm


@pytest.mark.parametrize("M,H", [(1, 2048), (13, 4096), (64, 8192), (3, 96), (2, 16384), (5, 8224), (2, 20480)])
def test_rmsnorm(M, H):
    x = gen.normal_f16(20 + M, 0, (M, H))
    g = gen.normal_f16(21, 0, (H,), 1.0, 0.02)
    out = torch.zeros((M, H), dtype=torch.int16, device=dev())
    ss.rmsnorm(up(x), up(g), out)
    torch.cuda.synchronize()
    check_close(down16(out), oracle.rmsnorm(x, g), "rmsnorm")


# ------------------------------------------------------------ attention


def _attn_case(cfg, seed=0, P=None, parent=None, q=None, k=None, v=None, kc=None, vc=None):
    s = cfg.shape
    T = cfg.T
    P = cfg.P if P is None else P
    S_max = cfg.S_max
    if parent is None:
        parent, _ = gen.workloads.make_tree(cfg)
    q = gen.normal_f16(seed, 0, (T, s.Hq * s.D), 0.0, 1.8) if q is None else q
    k = gen.normal_f16(seed, 1, (T, s.Hkv * s.D), 0.0, 1.8) if k is None else k
    v = gen.normal_f16(seed, 2, (T, s.Hkv * s.D)) if v is None else v
    if kc is None:
        kc = np.zeros((s.Hkv, S_max, s.D), np.uint16)
        vc = np.zeros((s.Hkv, S_max, s.D), np.uint16)
        kc[:, :P] = gen.normal_f16(seed, 3, (s.Hkv, P, s.D))
        vc[:, :P] = gen.normal_f16(seed, 4, (s.Hkv, P, s.D))
    dkc, dvc = up(kc), up(vc)
    out = torch.zeros((T, s.Hq * s.D), dtype=torch.int16, device=dev())
    ws = ss.workspace(ss.tree_attention_workspace_bytes(T, s.Hq, s.Hkv, s.D, S_max), dev())
    rope = up(ss.rope_table(500000.0, S_max, s.D))
    ss.tree_attention(up(q), up(k), up(v), dkc, dvc, up(np.array([P], np.int32)), up(parent), s.Hq,
                      s.Hkv, s.D, rope, out, ws)
    torch.cuda.synchronize()
    assert ss.read_device_error(ws) == 0
    okc, ovc = kc.copy(), vc.copy()
    ref = oracle.tree_attention(q, k, v, okc, ovc, P, parent, s.Hq, s.Hkv, s.D)
    return out, dkc, dvc, ref, okc, ovc


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_tree_attention_config_shapes(name):
    cfg = CONFIGS[name]
    P = cfg.P
    out, dkc, dvc, ref, okc, ovc = _attn_case(cfg, seed=cfg.index)
    check_close(down16(out), ref, f"attention {name}")
    gk, gv = down16(dkc), down16(dvc)
    assert np.array_equal(gk[:, :P], okc[:, :P]) and np.array_equal(gv, ovc)
    check_close(gk[:, P:P + cfg.T], okc[:, P:P + cfg.T], "rotated tree keys")


def test_tree_attention_edge_cases():
    from gen.workloads import WorkloadConfig
    # empty prefix, single-node tree, chain of 64, prefix not a multiple of the key tile
    cases = [WorkloadConfig(61, "e1", LLAMA_8B, P=0, T=5, levels=3, branching=2),
             WorkloadConfig(62, "e2", LLAMA_1B, P=77, T=1, levels=1, branching=1),
             WorkloadConfig(63, "e3", LLAMA_70B, P=130, T=64, levels=64, branching=1),
             WorkloadConfig(64, "e4", LLAMA_8B, P=1000, T=33, levels=7, branching=4),
             # 104 query rows per KV head in 16-row waves: the 7th wave half
             # empty, the 8th wholly past the rows
             WorkloadConfig(65, "e5", LLAMA_70B, P=2000, T=13, levels=5, branching=3)]
    for cfg in cases:
        out, dkc, dvc, ref, okc, ovc = _attn_case(cfg, seed=cfg.index)
        check_close(down16(out), ref, f"attention {cfg.name}")


@pytest.mark.parametrize("shape,P,T", [("1b", 16391, 64), ("8b", 16400, 33), ("70b", 16384, 17)])
def test_tree_attention_long_prefix_eight_wave_workgroups(shape, P, T):
    """More than 128 query rows per KV head and a prefix that may reach 16K
    keys: workgroups of 8 waves (256 rows), one per compute unit, 32 parts;
    prefixes not a multiple of the 32-key stage, trees of 17 to 64 nodes."""
    from gen.workloads import WorkloadConfig
    sh = {"1b": LLAMA_1B, "8b": LLAMA_8B, "70b": LLAMA_70B}[shape]
    cfg = WorkloadConfig(70 + T, f"long-{shape}", sh, P=P, T=T, levels=min(T, 9), branching=3)
    out, dkc, dvc, ref, okc, ovc = _attn_case(cfg, seed=cfg.index)
    check_close(down16(out), ref, f"attention {cfg.name}")
    check_close(down16(dkc)[:, P:P + T], okc[:, P:P + T], "rotated tree keys")


def test_tree_attention_non_ancestor_perturbation_is_bitwise_invisible():
    cfg = CONFIGS["c2"]
    s = cfg.shape
    parent, _ = gen.workloads.make_tree(cfg)
    depth, anc = oracle.tree(parent)
    q = gen.normal_f16(1, 0, (cfg.T, s.Hq * s.D), 0.0, 1.8)
    k = gen.normal_f16(1, 1, (cfg.T, s.Hkv * s.D), 0.0, 1.8)
    v = gen.normal_f16(1, 2, (cfg.T, s.Hkv * s.D))
    base = _attn_case(cfg, seed=1, parent=parent, q=q, k=k, v=v)[0].cpu().numpy()
    i = int(np.argmax(depth))
    others = ~anc[i].astype(bool)
    noise = gen.normal_f16(99, 0, q.shape)
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    q2[others] = noise[others]
    k2[others] = noise[others][:, :s.Hkv * s.D]
    v2[others] = noise[others][:, s.Hkv * s.D:2 * s.Hkv * s.D]
    pert = _attn_case(cfg, seed=1, parent=parent, q=q2, k=k2, v=v2)[0].cpu().numpy()
    assert np.array_equal(base[i], pert[i])


def test_tree_attention_invalid_tree_or_prefix_sets_error_and_writes_nothing():
    cfg = CONFIGS["c1"]
    s = cfg.shape
    T = cfg.T
    for P, parent, bit in ((cfg.P, np.array([-1, 0, 0, 5, 1, 1, 1, 1], np.int32), ss.DEVERR_BAD_TREE),
                           (cfg.P + 1, gen.workloads.make_tree(cfg)[0], ss.DEVERR_BAD_PREFIX)):
        kc = torch.zeros((s.Hkv, cfg.S_max, s.D), dtype=torch.int16, device=dev())
        vc = torch.zeros_like(kc)
        out = torch.full((T, s.Hq * s.D), 7, dtype=torch.int16, device=dev())
        ws = ss.workspace(ss.tree_attention_workspace_bytes(T, s.Hq, s.Hkv, s.D, cfg.S_max), dev())
        qkv = torch.ones((T, s.n_qkv), dtype=torch.int16, device=dev())
        rope = up(ss.rope_table(500000.0, cfg.S_max, s.D))
        ss.tree_attention(qkv, qkv[:, s.Hq * s.D:], qkv[:, (s.Hq + s.Hkv) * s.D:], kc, vc,
                          up(np.array([P], np.int32)), up(parent), s.Hq, s.Hkv, s.D, rope, out, ws)
        assert ss.read_device_error(ws) & bit
        assert torch.all(out == 7) and torch.all(kc == 0) and torch.all(vc == 0)


# ------------------------------------------------------- layouts (bit-exact)


def test_prepack_is_a_bit_exact_rearrangement():
    K, N = 512, 192
    W = _rand_w4(31, N, K)
    t, d = upload_w4(W)
    packed = t[3].cpu().numpy()
    G = K // 128
    qp = packed[:K * N // 2].reshape(N // 16, G, 64, 16)
    szp = packed[K * N // 2:].view(np.uint32).reshape(N // 16, G, 16)
    q, s_, z = W["qweight"], W["scales"], W["zeros"]
    for tile in range(N // 16):
        for g in range(G):
            for lane in range(64):
                n, kq = tile * 16 + lane % 16, lane // 16
                assert np.array_equal(qp[tile, g, lane], q[n, g * 64 + kq * 16:g * 64 + kq * 16 + 16])
            for c in range(16):
                n = tile * 16 + c
                assert szp[tile, g, c] == int(s_[n, g]) | (int(z[n, g]) << 16)


def test_prepared_activation_layout_is_bit_exact():
    M, K = 21, 256
    x = gen.normal_f16(32, 0, (M, K))
    xp = torch.zeros(ss.prepared_bytes(M, K), dtype=torch.uint8, device=dev())
    ss.prepare_activations(up(x), xp)
    torch.cuda.synchronize()
    got = xp.cpu().numpy().view(np.uint16)
    G = K // 128
    exp = np.zeros(((M + 15) // 16, G, 4, 64, 8), np.uint16)
    order = [0, 4, 2, 6, 8, 12, 10, 14]
    xf = x.view(np.float16)
    for m in range(M):
        for k0 in range(0, K, 32):
            g, kq = k0 // 128, (k0 % 128) // 32
            lane = kq * 16 + m % 16
            for f in range(4):
                base = k0 + 16 * (f % 2) + (f // 2)  # even k for f < 2, odd k for f >= 2
                vals = np.array([xf[m, base + o] for o in order], np.float16)
                exp[m // 16, g, f, lane] = vals.view(np.uint16)
    assert np.array_equal(got.reshape(exp.shape), exp)


def test_prepared_gemm_entry_matches_plain_entry_bitwise():
    M, K, N = 24, 1024, 256
    W = _rand_w4(33, N, K)
    t, d = upload_w4(W)
    x = gen.normal_f16(34, 0, (M, K))
    dx = up(x)
    y1 = torch.zeros((M, N), dtype=torch.int16, device=dev())
    y2 = torch.zeros_like(y1)
    ws = ss.workspace(ss.gemm_workspace_bytes(M, K, N), dev())
    ss.w4a16_gemm(d, dx, y1, ws)
    xp = torch.zeros(ss.prepared_bytes(M, K), dtype=torch.uint8, device=dev())
    ss.prepare_activations(dx, xp)
    ss.w4a16_gemm_prepared(d, xp, M, y2, ws)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
