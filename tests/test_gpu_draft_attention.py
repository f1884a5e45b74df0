"""GPU checks of the draft model's tree attention with the non-square mask
(swiftspec_draft_tree_attention) against the oracle: Llama-3.2-1B- and
Llama-3-8B-shaped heads (D = 64 and 128), the Fig. 4 sizes (a tree cache of
6 nodes, 4 leaves), full 64-node caches with 64 leaves, an empty prefix and
an empty tree cache; outputs and rotated key rows within the kernel
tolerance, value rows and every other cache row bit-exact; invalid forests
and prefixes leave output and cache untouched and set the error word."""
import numpy as np
import pytest

import gen
import oracle
from gen.workloads import LLAMA_1B, LLAMA_8B

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
from gpu_helpers import check_close, dev, down16, up  # noqa: E402


def _case(shape, P, N, w, seed, extra=3):
    rng = np.random.default_rng(seed)
    cp = np.array([-1 if (j == 0 or rng.random() < 0.25) else int(rng.integers(0, j)) for j in range(N)], np.int32)
    lp = np.array([int(rng.integers(-1, N)) for _ in range(w)], np.int32)
    S_max = P + N + w + extra
    q = gen.normal_f16(seed, 0, (w, shape.Hq * shape.D), 0.0, 1.8)
    k = gen.normal_f16(seed, 1, (w, shape.Hkv * shape.D), 0.0, 1.8)
    v = gen.normal_f16(seed, 2, (w, shape.Hkv * shape.D))
    kc = gen.normal_f16(seed, 3, (shape.Hkv, S_max, shape.D))
    vc = gen.normal_f16(seed, 4, (shape.Hkv, S_max, shape.D))
    return cp, lp, q, k, v, kc, vc, S_max


def _run(shape, P, cp, lp, q, k, v, kc, vc, S_max):
    w = len(lp)
    dkc, dvc = up(kc), up(vc)
    out = torch.full((w, shape.Hq * shape.D), 0x1234, dtype=torch.int16, device=dev())
    ws = ss.workspace(ss.tree_attention_workspace_bytes(w, shape.Hq, shape.Hkv, shape.D, S_max), dev())
    rope = up(ss.rope_table(500000.0, S_max, shape.D))
    ss.draft_tree_attention(up(q), up(k), up(v), dkc, dvc, up(np.array([P], np.int32)),
                            up(cp) if len(cp) else None, up(lp), shape.Hq, shape.Hkv, rope, out, ws)
    torch.cuda.synchronize()
    return down16(out), down16(dkc), down16(dvc), ss.read_device_error(ws)


@pytest.mark.parametrize("shape,P,N,w", [(LLAMA_1B, 512, 6, 4), (LLAMA_1B, 2048, 40, 8), (LLAMA_8B, 1000, 64, 64),
                                         (LLAMA_8B, 0, 0, 8), (LLAMA_1B, 77, 0, 1), (LLAMA_8B, 4096, 17, 13),
                                         (LLAMA_1B, 0, 64, 5)])
def test_draft_attention_matches_oracle(shape, P, N, w):
    seed = P + 7 * N + w
    cp, lp, q, k, v, kc, vc, S_max = _case(shape, P, N, w, seed)
    out, gk, gv, err = _run(shape, P, cp, lp, q, k, v, kc, vc, S_max)
    assert err == 0
    okc, ovc = kc.copy(), vc.copy()
    ref = oracle.draft_tree_attention(q, k, v, okc, ovc, P, cp, lp, shape.Hq, shape.Hkv, shape.D)
    check_close(out, ref, f"draft attention P={P} N={N} w={w}")
    new = slice(P + N, P + N + w)
    check_close(gk[:, new], okc[:, new], "rotated new keys")
    assert np.array_equal(gv, ovc)
    keep = np.ones(S_max, bool)
    keep[new] = False
    assert np.array_equal(gk[:, keep], kc[:, keep])


def test_draft_attention_invalid_data():
    shape = LLAMA_1B
    cp, lp, q, k, v, kc, vc, S_max = _case(shape, 100, 8, 4, 5)
    for bad_cp, bad_lp, P, bit in ((np.array([-1, 0, 5, 1, 1, 2, 0, 3], np.int32), lp, 100, ss.DEVERR_BAD_TREE),
                                   (cp, np.array([0, 8, 1, -1], np.int32), 100, ss.DEVERR_BAD_TREE),
                                   (cp, lp, S_max - 8 - 4 + 1, ss.DEVERR_BAD_PREFIX)):
        out, gk, gv, err = _run(shape, P, bad_cp, bad_lp, q, k, v, kc, vc, S_max)
        assert err & bit
        assert np.all(out.view(np.int16) == 0x1234)
        assert np.array_equal(gk, kc) and np.array_equal(gv, vc)
