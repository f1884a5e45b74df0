"""GPU parity of the kernel paths the benchmark times outside the five layer
configurations, and of the W4A16 GEMMs over the whole fp16 input range.

* Full fp16 range: activation rows carrying values up to +-65504 at even
  and at odd k (the two nibble positions of a packed weight byte), through
  the plain GEMM, the vector-ALU variant, the fused SwiGLU and the 70B down
  projection, against the oracle at |gpu - ref| <= 2e-3 + 1e-2 |ref|.
* Template instances reached only at the 80-layer shape or by the
  tensor-parallel shard benchmark: four 16-row tiles with two column tiles
  per wave (M = 64, K = 28672), three tiles (M = 40, K = 16384), the
  one-tile SwiGLU whose column blocks are split between workgroups and summed
  by the fix-up kernel (M = 8, K = 8192, N = 7168), the other shard GEMMs,
  and the attention over 16 query / 2 KV heads at a tree of 8 tokens with
  prefixes of 500, 1000 and 4096 keys.
"""
import numpy as np
import pytest

import gen
import oracle
from gen.workloads import LayerShape, WorkloadConfig

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

SPIKES = np.array([65504.0, -65504.0, 30000.0, -20000.0, 8192.0, -4096.0, 4095.0, -12288.0], np.float16)


def _w4(seed, N, K, std=0.02):
    q, s, z = gen.w4_random(seed, 0, N, K, std=std)
    return {"qweight": q, "scales": s, "zeros": z, "K": K, "N": N}


def _rows(W, cols):
    return {"qweight": W["qweight"][cols], "scales": W["scales"][cols], "zeros": W["zeros"][cols],
            "K": W["K"], "N": len(cols)}


def _spiked(seed, M, K, per_row=2):
    """N(0, 1) fp16 rows, each with `per_row` entries replaced by values from
    SPIKES, alternately at an even and an odd k; row 0 keeps its spikes at
    k = 0 and k = 1 (the first low and high nibble of a weight byte)."""
    x = gen.normal_f16(seed, 0, (M, K)).view(np.float16).copy()
    rng = np.random.default_rng(seed)
    for m in range(M):
        for j in range(per_row):
            k = 2 * int(rng.integers(0, K // 2)) + (j % 2)
            if m == 0:
                k = j % 2
            x[m, k] = SPIKES[(m + j) % len(SPIKES)]
    return x.view(np.uint16)


def _gemm(W, x, residual=None, valu=False):
    M, K = x.shape
    N = W["N"]
    t, d = upload_w4(W)
    dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
    r = up(residual) if residual is not None else None
    if valu:
        ws = ss.workspace(ss.gemm_valu_workspace_bytes(M, K, N), dev())
        ss.w4a16_gemm_valu(d, up(x), dy, ws, residual=r)
    else:
        ws = ss.workspace(ss.gemm_workspace_bytes(M, K, N), dev())
        ss.w4a16_gemm(d, up(x), dy, ws, residual=r)
    torch.cuda.synchronize()
    return down16(dy)


def _swiglu(Wg, Wu, x):
    M, K = x.shape
    N = Wg["N"]
    tg, dg = upload_w4(Wg)
    tu, du = upload_w4(Wu)
    dy = torch.zeros((M, N), dtype=torch.int16, device=dev())
    ws = ss.workspace(ss.swiglu_workspace_bytes(M, K, N), dev())
    ss.w4a16_swiglu(dg, du, up(x), dy, ws)
    torch.cuda.synchronize()
    return down16(dy)


def _sample_cols(N, seed, edge=64, n=256):
    rng = np.random.default_rng(seed)
    return np.concatenate([np.arange(edge), np.arange(N - edge, N),
                           rng.choice(np.arange(edge, N - edge), n, replace=False)])


# ------------------------------------------------------- full fp16 range


@pytest.mark.parametrize("M,K,N,valu", [(21, 1024, 320, False), (32, 8192, 1024, False), (64, 2048, 1024, False),
                                        (8, 4096, 512, False), (13, 1024, 320, True), (40, 2048, 512, True)])
def test_gemm_accepts_the_whole_fp16_range(M, K, N, valu):
    W = _w4(300 + M, N, K)
    x = _spiked(301 + M, M, K)
    res = gen.normal_f16(302, M, (M, N))
    got = _gemm(W, x, res, valu=valu)
    ref = oracle.w4a16_gemm(W, x, residual=res)
    assert np.all(np.isfinite(ref.view(np.float16)))
    err, rel = check_close(got, ref, f"spiked gemm M={M} K={K} N={N} valu={valu}")
    print(f"spiked gemm M={M} K={K} N={N} valu={valu}: max |ref| "
          f"{np.abs(ref.view(np.float16).astype(np.float64)).max():.0f}, max abs err {err:.3g}, rel {rel:.3g}")


@pytest.mark.parametrize("M,K,N", [(32, 8192, 28672), (8, 4096, 14336), (64, 8192, 28672), (8, 8192, 7168)])
def test_swiglu_accepts_the_whole_fp16_range(M, K, N):
    # small weights keep silu(g) * u finite at spikes of 65504
    Wg, Wu = _w4(310 + M, N, K, std=0.0004), _w4(311 + M, N, K, std=0.0004)
    x = _spiked(312 + M, M, K)
    got = _swiglu(Wg, Wu, x)
    cols = _sample_cols(N, 313)
    ref = oracle.w4a16_swiglu(_rows(Wg, cols), _rows(Wu, cols), x)
    assert np.all(np.isfinite(ref.view(np.float16)))
    err, rel = check_close(got[:, cols], ref, f"spiked swiglu M={M} K={K} N={N}")
    print(f"spiked swiglu M={M} K={K} N={N}: max |ref| "
          f"{np.abs(ref.view(np.float16).astype(np.float64)).max():.1f}, max abs err {err:.3g}, rel {rel:.3g}")


@pytest.mark.parametrize("M", [32, 64])
def test_down_projection_70b_with_spiked_input(M):
    """The 70B down projection (K = 28672, N = 8192, + residual) fed an FFN
    activation with large entries; M = 64 is the 80-layer step's instance
    (four 16-row tiles, two column tiles per wave)."""
    K, N = 28672, 8192
    W = _w4(320, N, K)
    x = _spiked(321 + M, M, K, per_row=4)
    res = gen.normal_f16(322, M, (M, N))
    got = _gemm(W, x, res)
    cols = _sample_cols(N, 323)
    ref = oracle.w4a16_gemm(_rows(W, cols), x, residual=np.ascontiguousarray(res[:, cols]))
    assert np.all(np.isfinite(ref.view(np.float16)))
    err, rel = check_close(got[:, cols], ref, f"spiked down M={M}")
    print(f"spiked down M={M}: max abs err {err:.3g}, rel {rel:.3g}")


# ---------------------------------------- instances of the long-K plans


@pytest.mark.parametrize("M,K,N", [(64, 28672, 8192), (40, 16384, 512), (16, 16384, 1024)])
def test_gemm_two_tiles_per_wave_long_k(M, K, N):
    """Two column tiles per wave at K >= 16384: the 80-layer step's down
    projection (64 rows, 16-row tiles x 4), 40 rows (x 3) and 16 rows (x 1),
    with residual; sampled columns where N is large."""
    W = _w4(330 + M, N, K)
    x = gen.normal_f16(331, M, (M, K))
    res = gen.normal_f16(332, M, (M, N))
    got = _gemm(W, x, res)
    cols = _sample_cols(N, 333) if N > 1024 else np.arange(N)
    ref = oracle.w4a16_gemm(_rows(W, cols), x, residual=np.ascontiguousarray(res[:, cols]))
    err, rel = check_close(got[:, cols], ref, f"long-K gemm M={M} K={K} N={N}")
    print(f"long-K gemm M={M} K={K} N={N}: max abs err {err:.3g}, rel {rel:.3g}")


# ------------------------- one GPU's share of the 70B TP4 shard (batch 8)


@pytest.mark.parametrize("name,K,N,res", [("qkv", 8192, 2560, False), ("o_proj", 2048, 8192, True),
                                          ("down", 7168, 8192, True)])
def test_tp4_shard_gemms(name, K, N, res):
    M = 8
    W = _w4(340 + K // 1024, N, K)
    x = gen.normal_f16(341, K // 1024, (M, K))
    r = gen.normal_f16(342, K // 1024, (M, N)) if res else None
    outs = [_gemm(W, x, r) for _ in range(2)]
    assert np.array_equal(outs[0], outs[1])
    err, rel = check_close(outs[0], oracle.w4a16_gemm(W, x, residual=r), f"tp4 {name}")
    print(f"tp4 {name} (M 8, K {K}, N {N}): max abs err {err:.3g}, rel {rel:.3g}")


@pytest.mark.parametrize("M", [8, 12])
def test_tp4_shard_swiglu(M):
    """K = 8192, N = 7168.  M = 8 (the shard's batch): one workgroup per
    16-column tile, gate and up tile together, K split across 4 waves.
    M = 12 (past the K-split SwiGLU's 8 rows): 112 column blocks of 64,
    fewer than the compute units, so stream-K splits them between
    workgroups and the fix-up kernel sums the gate and up partials in order
    before silu(g) * u."""
    K, N = 8192, 7168
    Wg, Wu = _w4(350, N, K), _w4(351, N, K)
    x = gen.normal_f16(352, M, (M, K))
    outs = [_swiglu(Wg, Wu, x) for _ in range(2)]
    assert np.array_equal(outs[0], outs[1])
    err, rel = check_close(outs[0], oracle.w4a16_swiglu(Wg, Wu, x), f"tp4 swiglu M={M}")
    print(f"tp4 swiglu (M {M}, K 8192, N 7168): max abs err {err:.3g}, rel {rel:.3g}")


@pytest.mark.parametrize("P", [500, 1000, 4096])
def test_tp4_shard_attention(P):
    """16 query / 2 KV heads, D = 128, a tree of 8 tokens (spine of 4,
    branching <= 2), prefix of P keys: outputs within tolerance, the
    appended rotated keys within tolerance, values bit-exact, the prefix
    untouched."""
    shape = LayerShape(H=2048, Hq=16, Hkv=2, D=128, F=7168)
    cfg = WorkloadConfig(90 + P % 89, f"tp4_ctx{P}", shape, P=P, T=8, levels=4, branching=2)
    T, S_max = cfg.T, cfg.S_max
    parent = np.asarray(gen.tree(T, 4, 2, 2506), np.int32)
    q = gen.normal_f16(360, P, (T, shape.Hq * shape.D), 0.0, 1.8)
    k = gen.normal_f16(361, P, (T, shape.Hkv * shape.D), 0.0, 1.8)
    v = gen.normal_f16(362, P, (T, shape.Hkv * shape.D))
    kc = np.zeros((shape.Hkv, S_max, shape.D), np.uint16)
    vc = np.zeros_like(kc)
    kc[:, :P] = gen.normal_f16(363, P, (shape.Hkv, P, shape.D))
    vc[:, :P] = gen.normal_f16(364, P, (shape.Hkv, P, shape.D))
    dkc, dvc = up(kc), up(vc)
    out = torch.zeros((T, shape.Hq * shape.D), dtype=torch.int16, device=dev())
    ws = ss.workspace(ss.tree_attention_workspace_bytes(T, shape.Hq, shape.Hkv, shape.D, S_max), dev())
    rope = up(ss.rope_table(500000.0, S_max, shape.D))
    ss.tree_attention(up(q), up(k), up(v), dkc, dvc, up(np.array([P], np.int32)), up(parent), shape.Hq,
                      shape.Hkv, shape.D, rope, out, ws)
    torch.cuda.synchronize()
    assert ss.read_device_error(ws) == 0
    okc, ovc = kc.copy(), vc.copy()
    ref = oracle.tree_attention(q, k, v, okc, ovc, P, parent, shape.Hq, shape.Hkv, shape.D)
    err, rel = check_close(down16(out), ref, f"tp4 attention ctx {P}")
    gk, gv = down16(dkc), down16(dvc)
    assert np.array_equal(gk[:, :P], kc[:, :P]) and np.array_equal(gv, ovc)
    check_close(gk[:, P:P + T], okc[:, P:P + T], "tp4 rotated tree keys")
    print(f"tp4 attention ctx {P}: max abs err {err:.3g}, rel {rel:.3g}")
