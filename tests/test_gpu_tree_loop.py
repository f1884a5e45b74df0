"""The loop of Alg. 1 run sequentially on the GPU with synthetic draft and
target models (bench.py's tree_loop): after every iteration

* the target's acceptance equals the oracle's on the same logits rows, and
  the target cache's prefix holds exactly the committed tokens (rows moved
  by the device commit);
* the draft cache's prefix holds the committed tokens followed by the new
  root (the rows moved by the device reorganisation plus the pending
  tokens), and every tree-cache row holds the token of the node the host
  tree assigns it;
* the tree is a valid tree whose root is the target's last output token."""
import importlib.util
import os

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


def _bench():
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "bench.py")
    spec = importlib.util.spec_from_file_location("bench_mod", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("seed,p_agree,w,k,bs", [(1, 0.8, 4, 3, 8), (2, 0.95, 8, 8, 16), (3, 0.0, 2, 2, 4)])
def test_tree_loop_state_is_consistent(seed, p_agree, w, k, bs):
    bench = _bench()
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    seen = {"L": []}

    def check(st):
        lg = st["logits"].cpu().numpy().view(np.uint16)
        am, acc, bonus, L = oracle.greedy_accept(lg, st["tokens"], st["parent"])
        assert np.array_equal(st["argmax"], am)
        assert (st["accepted"], st["bonus"], st["L"]) == (acc, bonus, L)
        committed = st["committed"]
        P_t = st["P_t"]
        assert P_t == len(committed)
        assert st["tk"][0, :P_t, 0].cpu().tolist() == committed
        tree = st["tree"]
        tok, par, _, row, _ = tree.nodes()
        assert tok[0] == st["bonus"] and par[0] == -1 and all(0 <= par[v] < v for v in range(1, len(tok)))
        p_d = st["p_d"]
        assert st["dk"][0, :p_d, 0].cpu().tolist() == committed + [st["bonus"]]
        for v in range(1, len(tok)):
            if row[v] >= 0:
                assert int(st["dk"][0, p_d + row[v], 0].item()) == int(tok[v])
        seen["L"].append(L)

    out = bench.tree_loop(ss, torch, np, dev, stream, V=4096, iters=12, w=w, k=k, d=3, bs=bs, p_agree=p_agree,
                          seed=seed, check=check)
    assert len(seen["L"]) == 12
    if p_agree >= 0.8:
        assert max(seen["L"]) >= 3  # paths of several tokens were accepted
    assert out["iterations"] == 12
