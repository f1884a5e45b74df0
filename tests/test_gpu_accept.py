"""GPU checks of greedy acceptance (swiftspec_greedy_accept) against the
oracle, bit-exact (integer outputs from the same fp16 logits):

* synthetic logits with planted ties, padded leading dimensions, random
  trees and draft tokens planted to match, over tree sizes 1..64 and
  vocabularies from 7 to 128256 entries (two calls in a row share one
  workspace, so the ticket counter must come back to zero);
* an invalid tree: the error bit, choices still written, nothing else;
* the closing step at the 80-layer configuration's shape (two layers, LM
  head over 128256 rows): verify, accept and commit on one stream, eagerly
  and as one HIP graph, against the oracle's acceptance on the step's own
  logits and its commit on the step's own caches."""
import numpy as np
import pytest

import oracle

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
from gpu_helpers import DeviceStep, dev, down16, up  # noqa: E402


def _case(T, V, pad, seed):
    rng = np.random.default_rng(seed)
    ldl = (V + 7) // 8 * 8 + 8 * pad
    lg = np.full((T, ldl), np.float16(30000.0))          # padding beyond V must be ignored
    lg[:, :V] = rng.standard_normal((T, V)).astype(np.float16)
    for i in range(0, T, 3):                              # ties: the first index must win
        j = rng.choice(V, min(V, 3), replace=False)
        lg[i, j] = np.float16(6.0)
    parent = np.array([-1] + [int(rng.integers(0, i)) for i in range(1, T)], np.int32)
    am = np.argmax(lg[:, :V].astype(np.float64), axis=1)
    tokens = rng.integers(0, V, T).astype(np.int32)
    for c in range(1, T):                                 # most children carry their parent's choice
        if rng.random() < 0.6:
            tokens[c] = am[parent[c]]
    return lg.view(np.uint16), parent, tokens


def _run(lg, parent, tokens, V, ws):
    T = len(parent)
    d_lg = up(lg)
    d_am = torch.full((T,), -7, dtype=torch.int32, device=dev())
    outs = [torch.full((1,), -7, dtype=torch.int32, device=dev()) for _ in range(3)]
    ss.greedy_accept(d_lg, up(tokens), up(parent), d_am, outs[0], outs[1], ws, path_len=outs[2], V=V)
    torch.cuda.synchronize()
    return d_am.cpu().numpy(), [int(o.item()) for o in outs]


@pytest.mark.parametrize("T,V,pad", [(1, 8, 0), (5, 1000, 1), (32, 7, 0), (64, 4099, 2), (64, 128256, 0),
                                     (17, 65, 3)])
def test_greedy_accept_matches_oracle(T, V, pad):
    ws = ss.workspace(ss.greedy_accept_workspace_bytes(T), dev())
    for rep in range(2):
        lg, parent, tokens = _case(T, V, pad, 1000 * T + V + rep)
        am, (acc, bonus, L) = _run(lg, parent, tokens, V, ws)
        r_am, r_acc, r_bonus, r_L = oracle.greedy_accept(np.ascontiguousarray(lg[:, :V]), tokens, parent)
        assert np.array_equal(am, r_am)
        assert (acc, bonus, L) == (r_acc, r_bonus, r_L), (T, V, rep)
        print(f"T={T} V={V} rep={rep}: accepted {acc} (path {L}), bonus {bonus}")
    assert ss.read_device_error(ws) == 0


def test_greedy_accept_invalid_tree():
    T, V = 9, 300
    lg, parent, tokens = _case(T, V, 0, 5)
    ws = ss.workspace(ss.greedy_accept_workspace_bytes(T), dev())
    bad = parent.copy()
    bad[4] = 6                                            # a parent after its child
    am, outs = _run(lg, bad, tokens, V, ws)
    assert ss.read_device_error(ws) == ss.DEVERR_BAD_TREE
    ref = oracle.greedy_accept(np.ascontiguousarray(lg[:, :V]), tokens, parent)
    assert np.array_equal(am, ref[0])
    assert outs == [-7, -7, -7]
    # the counter came back to zero: a valid call on the same workspace works
    am, (acc, bonus, L) = _run(lg, parent, tokens, V, ws)
    assert (acc, bonus, L) == ref[1:]


def _plant_tokens(parent, acc, am, V, seed):
    """Draft tokens under which the path root -> acc matches the target's
    choices and no other node does."""
    rng = np.random.default_rng(seed)
    T = len(parent)
    tokens = rng.integers(0, V, T).astype(np.int32)
    path = []
    j = acc
    while j != -1:
        path.append(j)
        j = int(parent[j])
    on_path = set(path)
    for c in range(1, T):
        if c in on_path:
            tokens[c] = am[parent[c]]
        elif tokens[c] == am[parent[c]]:
            tokens[c] = (tokens[c] + 1) % V
    return tokens


def test_closing_step_eager_and_graph():
    from gen.workloads import CONFIGS, make_activations
    cfg = CONFIGS["c5"]
    n = 2
    st = DeviceStep(cfg, n, source="host")
    x = up(make_activations(cfg))
    k0, v0 = st.kc.clone(), st.vc.clone()
    hidden = x.clone()
    st.enqueue(hidden)
    torch.cuda.synchronize()
    logits = down16(st.logits)
    k_pre, v_pre = down16(st.kc), down16(st.vc)
    am_ref = oracle.greedy_accept(logits, np.zeros(cfg.T, np.int32), st.parent_h)[0]
    tokens = _plant_tokens(st.parent_h, st.acc, am_ref, cfg.vocab, 3)
    r_am, r_acc, r_bonus, r_L = oracle.greedy_accept(logits, tokens, st.parent_h)
    assert r_acc == st.acc and r_L > 1
    ref_k, ref_v = k_pre.copy(), v_pre.copy()
    L = oracle.kv_commit(ref_k, ref_v, cfg.P, st.parent_h, r_acc, n_layers=n)
    assert L == r_L
    # eager: accept and commit on the step's device outputs
    d_tok = up(tokens)
    d_am = torch.zeros(cfg.T, dtype=torch.int32, device=dev())
    d_acc, d_bonus, d_len = (torch.zeros(1, dtype=torch.int32, device=dev()) for _ in range(3))
    aws = ss.workspace(ss.greedy_accept_workspace_bytes(cfg.T), dev())

    def accept_and_commit(stream=None):
        ss.greedy_accept(st.logits, d_tok, st.parent, d_am, d_acc, d_bonus, aws, path_len=d_len,
                         stream=stream)
        ss.kv_commit(st.kc, st.vc, st.P, st.parent, d_acc, n_layers=n, advance=True, ws=aws, stream=stream)

    accept_and_commit()
    torch.cuda.synchronize()
    assert ss.read_device_error(aws) == 0 and ss.read_device_error(st.ws) == 0

    def check(tag):
        assert np.array_equal(d_am.cpu().numpy(), r_am), tag
        assert (int(d_acc.item()), int(d_bonus.item()), int(d_len.item())) == (r_acc, r_bonus, r_L), tag
        assert np.array_equal(down16(st.kc), ref_k) and np.array_equal(down16(st.vc), ref_v), tag
        assert int(st.P.item()) == cfg.P + L, tag

    check("eager")
    # one graph: verify step, acceptance, commit; state restored between replays
    stream = torch.cuda.Stream()
    g = ss.Graph()
    P0 = torch.tensor([cfg.P], dtype=torch.int32, device=dev())

    def restore():
        hidden.copy_(x)
        st.kc.copy_(k0)
        st.vc.copy_(v0)
        st.P.copy_(P0)
        for t in (d_am, d_acc, d_bonus, d_len):
            t.fill_(-1)

    with torch.cuda.stream(stream):
        restore()
    stream.synchronize()
    with torch.cuda.stream(stream):
        g.begin(stream)
        st.enqueue(hidden, stream=stream)
        accept_and_commit(stream=stream)
        g.end(stream)
    for rep in range(3):
        with torch.cuda.stream(stream):
            restore()
            g.launch(stream)
        stream.synchronize()
        check(f"graph replay {rep}")
    print(f"closing step: accepted node {r_acc} (path {r_L}), bonus token {r_bonus}")
