"""GPU parity of the final RMSNorm + fp16 LM head against the fp64 reference
checker: full outputs on small shapes (ragged M, vocabulary not a multiple of
a workgroup's 128 rows) and sampled vocabulary rows at the 80-layer
configuration's full size (M = 64, H = 8192, V = 128256), tolerance
|gpu - ref| <= 2e-3 + 1e-2 |ref|."""
import numpy as np
import pytest

import gen
import oracle
from gen.workloads import CONFIGS, make_final_norm, make_lm_head

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


def _run(h, gamma, W):
    M, H = h.shape
    V = W.shape[0]
    logits = torch.zeros((M, V), dtype=torch.int16, device=dev())
    ws = ss.workspace(ss.lm_head_workspace_bytes(M, H, V), dev())
    ss.lm_head(up(h), up(gamma), up(W), logits, ws)
    torch.cuda.synchronize()
    return down16(logits)


@pytest.mark.parametrize("M,H,V", [(1, 256, 16), (13, 512, 320), (32, 1024, 1040), (64, 384, 272)])
def test_lm_head_small_shapes(M, H, V):
    h = gen.normal_f16(71, M, (M, H))
    gamma = gen.normal_f16(72, M, (H,), 1.0, 0.02)
    W = gen.normal_f16(73, M, (V, H), 0.0, 0.02)
    got = _run(h, gamma, W)
    ref = oracle.lm_head(h, gamma, W)
    err, rel = check_close(got, ref, f"lm_head M={M} H={H} V={V}")
    print(f"lm_head M={M} H={H} V={V}: max abs err {err:.3g}, max rel err (|r|>=0.2) {rel:.3g}")


def test_lm_head_full_size_sampled_rows():
    cfg = CONFIGS["c5"]
    H, V, M = cfg.shape.H, cfg.vocab, cfg.T
    h = gen.normal_f16(cfg.seeds()["activations"], 7, (M, H))
    gamma = make_final_norm(cfg)
    W = make_lm_head(cfg)
    got = _run(h, gamma, W)
    del W
    rng = np.random.default_rng(5)
    rows = np.concatenate([[0, 1, V - 129, V - 128, V - 1], rng.choice(V, 59, replace=False)])
    ref = oracle.lm_head(h, gamma, make_lm_head(cfg, rows))
    err, rel = check_close(got[:, rows], ref, "lm_head c5 sampled rows")
    print(f"lm_head c5 (64 x 8192 x 128256), {len(rows)} sampled rows: max abs err {err:.3g}, rel {rel:.3g}")
    assert np.isfinite(got.view(np.float16).astype(np.float32)).all()


def test_lm_head_rejects_bad_arguments():
    h = torch.zeros((4, 256), dtype=torch.int16, device=dev())
    g = torch.zeros((256,), dtype=torch.int16, device=dev())
    W = torch.zeros((24, 256), dtype=torch.int16, device=dev())
    out = torch.zeros((4, 24), dtype=torch.int16, device=dev())
    ws = ss.workspace(ss.lm_head_workspace_bytes(4, 256, 24), dev())
    with pytest.raises(RuntimeError):
        ss.lm_head(h, g, W, out, ws)  # V % 16 != 0
    with pytest.raises(RuntimeError):
        ss.lm_head(h, g, W[:16], out, ss.workspace(16, dev()))  # workspace too small
