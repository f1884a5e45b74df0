"""GPU checks of the whole verification step (Alg. 1 batch verify over every
decoder layer, then final RMSNorm and LM head) at the 80-layer Llama-3-70B
configuration's shape (T = 64, P = 8192, H = 8192, vocabulary 128256):

* two layers + head from the seeded host recipe against the reference chain
  (end to end, with the propagation bound the one-layer test uses; the head
  on the reference's own final hidden state under the kernel tolerance), the
  KV commit of both layers bit-exact on the reference's caches;
* the full 80 layers (weights drawn on the device) captured as one HIP
  graph: replays bit-identical to the eager step, which is bit-identical to
  calling the per-layer and LM-head entry points one by one."""
import numpy as np
import pytest

import oracle
from gen.workloads import CONFIGS, make_activations, make_final_norm, make_kv_prefix, make_layer_weights, \
    make_lm_head

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
from gpu_helpers import DeviceStep, check_close, dev, down16, up  # noqa: E402


def test_step_two_layers_and_head_match_oracle():
    cfg = CONFIGS["c5"]
    s = cfg.shape
    n = 2
    st = DeviceStep(cfg, n, source="host")
    x = make_activations(cfg)
    hidden = up(x)
    st.enqueue(hidden)
    torch.cuda.synchronize()
    assert ss.read_device_error(st.ws) == 0
    out, logits = down16(hidden), down16(st.logits)
    # reference chain over the same seeded inputs
    dims = {"H": s.H, "Hq": s.Hq, "Hkv": s.Hkv, "D": s.D, "F": s.F, "S_max": cfg.S_max}
    okc, ovc = [], []
    h = x
    for l in range(n):
        kc, vc = make_kv_prefix(cfg, l)
        h = oracle.verify_layer(dims, make_layer_weights(cfg, l), kc, vc, h, cfg.P, st.parent_h)
        okc.append(kc)
        ovc.append(vc)
    r64 = h.view(np.float16).astype(np.float64)
    e2e = np.abs(out.view(np.float16).astype(np.float64) - r64)
    print(f"2-layer step: end-to-end max abs err {e2e.max():.3g}, output rms {np.sqrt(np.mean(r64 ** 2)):.3g}")
    assert np.all(e2e <= 0.05 + 0.02 * np.abs(r64)), e2e.max()
    V = cfg.vocab
    rng = np.random.default_rng(11)
    rows = np.concatenate([[0, 1, V - 1], rng.choice(V, 61, replace=False)])
    gamma = make_final_norm(cfg)
    ref_logits = oracle.lm_head(h, gamma, make_lm_head(cfg, rows))
    check_close(logits[:, rows], ref_logits, "step logits (end to end)", atol=0.05, rtol=0.02)
    # the head as a stage: fed the reference's final hidden state
    lg = torch.zeros((cfg.T, V), dtype=torch.int16, device=dev())
    ws = ss.workspace(ss.lm_head_workspace_bytes(cfg.T, s.H, V), dev())
    ss.lm_head(up(h), st.final_norm, st.lm_w, lg, ws)
    torch.cuda.synchronize()
    err, rel = check_close(down16(lg)[:, rows], ref_logits, "LM head stage")
    print(f"LM head stage: max abs err {err:.3g}, rel {rel:.3g}")
    # commit of both layers in one launch, on the reference's caches
    from gen.workloads import make_tree
    parent, acc = make_tree(cfg)
    dk, dv = up(np.stack(okc)), up(np.stack(ovc))
    dP = up(np.array([cfg.P], np.int32))
    ss.kv_commit(dk, dv, dP, st.parent, up(np.array([acc], np.int32)), n_layers=n, advance=True, ws=st.ws)
    torch.cuda.synchronize()
    k_all, v_all = np.stack(okc), np.stack(ovc)
    L = oracle.kv_commit(k_all, v_all, cfg.P, parent, acc, n_layers=n)
    assert np.array_equal(down16(dk), k_all) and np.array_equal(down16(dv), v_all)
    assert int(dP.item()) == cfg.P + L


def test_step_80_layers_graph_replay_and_composition_bitwise():
    cfg = CONFIGS["c5"]
    s = cfg.shape
    st = DeviceStep(cfg, cfg.n_layers, source="device")
    from gen import device as gdev
    x = gdev.normal_f16_device(cfg.seeds()["activations"], 0, (cfg.T, s.H), device=dev())
    hidden = x.clone()
    st.enqueue(hidden)
    torch.cuda.synchronize()
    assert ss.read_device_error(st.ws) == 0
    eager_h, eager_l = down16(hidden), down16(st.logits)
    assert np.isfinite(eager_l.view(np.float16)).all() and np.isfinite(eager_h.view(np.float16)).all()
    # per-layer entry points one by one
    h2 = x.clone()
    lws = ss.workspace(ss.verify_layer_workspace_bytes(st.dims, cfg.T), dev())
    for d in st.layer_descs:
        ss.verify_layer(d, st.dims, h2, st.P, st.parent, st.rope, lws)
    lg2 = torch.zeros_like(st.logits)
    ss.lm_head(h2, st.final_norm, st.lm_w, lg2, ss.workspace(ss.lm_head_workspace_bytes(cfg.T, s.H, cfg.vocab),
                                                              dev()))
    torch.cuda.synchronize()
    assert np.array_equal(down16(h2), eager_h) and np.array_equal(down16(lg2), eager_l)
    # one graph for the whole step; replays with eager work in between
    stream = torch.cuda.Stream()
    g = ss.Graph()
    with torch.cuda.stream(stream):
        g.begin(stream)
        st.enqueue(hidden, stream=stream)
        g.end(stream)
    for rep in range(3):
        st.logits.zero_()
        with torch.cuda.stream(stream):
            hidden.copy_(x)
            g.launch(stream)
        stream.synchronize()
        assert np.array_equal(down16(hidden), eager_h), f"replay {rep}"
        assert np.array_equal(down16(st.logits), eager_l), f"replay {rep}"
        h3 = x.clone()
        ss.verify_layer(st.layer_descs[0], st.dims, h3, st.P, st.parent, st.rope, lws)
        torch.cuda.synchronize()
