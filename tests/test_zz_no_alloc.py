"""The allocation-free tree attention (swiftspec_tree_attention_noalloc,
partials in the library's own device array) against the workspace entry
point swiftspec_tree_attention on the same inputs: outputs and caches bit for
bit, device errors in the caller's word, two calls in a row with the second
one smaller (the array keeps the first call's contents), and shapes beyond
the array refused before any launch."""
import numpy as np
import pytest

import gen
from gen.workloads import CONFIGS

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
from gpu_helpers import dev, down16, up  # noqa: E402


def _inputs(cfg, seed):
    s = cfg.shape
    T, P, S_max = cfg.T, cfg.P, cfg.S_max
    parent, _ = gen.workloads.make_tree(cfg)
    q = gen.normal_f16(seed, 0, (T, s.Hq * s.D), 0.0, 1.8)
    k = gen.normal_f16(seed, 1, (T, s.Hkv * s.D), 0.0, 1.8)
    v = gen.normal_f16(seed, 2, (T, s.Hkv * s.D))
    kc = np.zeros((s.Hkv, S_max, s.D), np.uint16)
    vc = np.zeros_like(kc)
    kc[:, :P] = gen.normal_f16(seed, 3, (s.Hkv, P, s.D))
    vc[:, :P] = gen.normal_f16(seed, 4, (s.Hkv, P, s.D))
    rope = ss.rope_table(500000.0, S_max, s.D)
    return parent, q, k, v, kc, vc, rope


def _run(cfg, seed, noalloc, parent=None, P=None):
    s = cfg.shape
    par, q, k, v, kc, vc, rope = _inputs(cfg, seed)
    par = par if parent is None else parent
    P = cfg.P if P is None else P
    dkc, dvc = up(kc), up(vc)
    out = torch.full((cfg.T, s.Hq * s.D), 7, dtype=torch.int16, device=dev())
    args = (up(q), up(k), up(v), dkc, dvc, up(np.array([P], np.int32)), up(np.asarray(par, np.int32)), s.Hq, s.Hkv,
            s.D, up(rope), out)
    if noalloc:
        err = torch.zeros(1, dtype=torch.int32, device=dev())
        ss.tree_attention_noalloc(*args, error=err)
        torch.cuda.synchronize()
        e = int(err.item())
    else:
        ws = ss.workspace(ss.tree_attention_workspace_bytes(cfg.T, s.Hq, s.Hkv, s.D, cfg.S_max), dev())
        ss.tree_attention(*args, ws)
        torch.cuda.synchronize()
        e = ss.read_device_error(ws)
    return down16(out), down16(dkc), down16(dvc), e


def test_noalloc_attention_matches_the_workspace_entry_on_two_calls():
    # the 70B layer (T 32, P 4096, 8 KV heads), then the smaller 1B layer
    for name in ("c3", "c1"):
        cfg = CONFIGS[name]
        ref = _run(cfg, cfg.index, noalloc=False)
        got = _run(cfg, cfg.index, noalloc=True)
        assert ref[3] == 0 and got[3] == 0
        for a, b in zip(ref[:3], got[:3]):
            assert np.array_equal(a, b), name
        assert not np.all(got[0] == 7)


def test_noalloc_attention_reports_device_errors_in_the_callers_word():
    cfg = CONFIGS["c1"]
    bad = np.array([-1, 0, 0, 5, 1, 1, 1, 1], np.int32)
    out, kc, vc, e = _run(cfg, 5, noalloc=True, parent=bad)
    assert e & ss.DEVERR_BAD_TREE
    assert np.all(out == 7)
    out, kc, vc, e = _run(cfg, 5, noalloc=True, P=cfg.P + 1)
    assert e & ss.DEVERR_BAD_PREFIX
    assert np.all(out == 7)


def test_noalloc_attention_refuses_partials_beyond_its_array():
    # 1024 KV heads of a 64-token tree: 2048 split partials of 16.6 KB
    T, Hq, Hkv, D, P = 64, 1024, 1024, 128, 256
    q = torch.zeros((T, Hq * D), dtype=torch.int16, device=dev())
    kc = torch.zeros((Hkv, P + T, D), dtype=torch.int16, device=dev())
    out = torch.zeros_like(q)
    rope = up(ss.rope_table(500000.0, P + T, D))
    with pytest.raises(ss.SwiftSpecError) as e:
        ss.tree_attention_noalloc(q, q, q, kc, kc, up(np.array([P], np.int32)),
                                  up(np.arange(-1, T - 1, dtype=np.int32)), Hq, Hkv, D, rope, out)
    assert e.value.status == ss.WORKSPACE_TOO_SMALL
