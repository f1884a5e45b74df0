"""GPU checks of the draft expansion step (Sec. 3.1, maximum-likelihood tree
expansion) and of the host draft tree driving the draft cache:

* swiftspec_topk_logprobs against the oracle: tokens bit-exact (decided on
  the same fp16 logits), log-softmax values within 1e-4 absolute (fp32
  normaliser over at most 128256 terms); planted ties, equal rows, padded
  leading dimensions, vocabularies from 9 to 128256, 1 to 64 rows, k = 1..8,
  two calls in a row sharing one workspace (the row counters come back to
  zero) with bit-identical results;
* a few iterations of the draft worker's loop on one stream: leaves chosen
  by the host tree, their children from the GPU top-k over synthetic draft
  logits, re-rooting on synthetic target outputs and the draft-cache
  reorganisation on the device; tree-cache rows carry their node's token,
  so after every re-root the device rows must sit where the host tree says
  (bit-exact) and the device's new forest must equal the host's."""
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
from gpu_helpers import dev, up  # noqa: E402

LP_ATOL = 1e-4


def _logits(n, V, pad, seed, ties=True):
    rng = np.random.default_rng(seed)
    ldl = (V + 7) // 8 * 8 + 8 * pad
    lg = np.full((n, ldl), np.float16(30000.0))  # padding beyond V must be ignored
    lg[:, :V] = (rng.standard_normal((n, V)) * 2).astype(np.float16)
    if ties:
        for i in range(0, n, 2):  # equal maxima: lower index first
            j = rng.choice(V, min(V, 5), replace=False)
            lg[i, j] = np.float16(9.0)
    return lg.view(np.uint16)


def _run(lg, V, k, ws=None):
    n = lg.shape[0]
    tok = torch.zeros((n, k), dtype=torch.int32, device=dev())
    lp = torch.zeros((n, k), dtype=torch.float32, device=dev())
    if ws is None:
        ws = ss.workspace(ss.topk_logprobs_workspace_bytes(n), dev())
    ss.topk_logprobs(up(lg), tok, lp, ws, V=V)
    torch.cuda.synchronize()
    return tok.cpu().numpy(), lp.cpu().numpy(), ws


@pytest.mark.parametrize("n,V,k,pad", [(8, 128256, 8, 0), (1, 1000, 1, 1), (64, 32000, 8, 0), (3, 77, 5, 2),
                                       (5, 4099, 8, 0), (2, 9, 8, 0), (17, 128256, 3, 1), (2, 150001, 8, 1)])
def test_topk_matches_oracle(n, V, k, pad):
    lg = _logits(n, V, pad, seed=n * 1000 + V)
    tok, lp, ws = _run(lg, V, k)
    otok, olp = oracle.topk_logprobs(lg[:, :V], k)
    assert np.array_equal(tok, otok)
    err = np.abs(lp.astype(np.float64) - olp).max()
    assert err <= LP_ATOL, f"max |logprob err| {err:.3g}"
    tok2, lp2, _ = _run(lg, V, k, ws)  # the same workspace again
    assert np.array_equal(tok, tok2) and np.array_equal(lp, lp2)


def test_topk_best_entries_in_one_range():
    """All k best logits of a row inside one workgroup's range (consecutive
    indices), so one partial list supplies every entry."""
    V, k = 128256, 8
    rng = np.random.default_rng(77)
    lg = (rng.standard_normal((8, V)) * 2).astype(np.float16)
    for i in range(8):
        lg[i, 5000 * i + 100:5000 * i + 100 + k] = np.float16(10.0) + np.arange(k, dtype=np.float16) * np.float16(0.25)
    lg = lg.view(np.uint16)
    tok, lp, _ = _run(lg, V, k)
    otok, olp = oracle.topk_logprobs(lg, k)
    assert np.array_equal(tok, otok)
    assert np.abs(lp.astype(np.float64) - olp).max() <= LP_ATOL


def test_topk_equal_rows():
    V = 50000
    lg = np.full((4, V), np.float16(-1.5)).view(np.uint16)
    tok, lp, _ = _run(lg, V, 8)
    assert np.array_equal(tok, np.tile(np.arange(8, dtype=np.int32), (4, 1)))
    assert np.abs(lp + np.log(V)).max() <= LP_ATOL


def test_topk_rejects_bad_arguments():
    x = torch.zeros((4, 64), dtype=torch.int16, device=dev())
    tok = torch.zeros((4, 9), dtype=torch.int32, device=dev())
    lp = torch.zeros((4, 9), dtype=torch.float32, device=dev())
    ws = ss.workspace(ss.topk_logprobs_workspace_bytes(4), dev())
    with pytest.raises(ss.SwiftSpecError) as e:  # k > 8
        ss.topk_logprobs(x, tok, lp, ws)
    assert e.value.status == ss.UNSUPPORTED
    with pytest.raises(ss.SwiftSpecError) as e:  # workspace too small
        ss.topk_logprobs(x, tok[:, :4], lp[:, :4], ws[:100])
    assert e.value.status == ss.WORKSPACE_TOO_SMALL


def _walk_rows(tree_tok, tree_par, tree_row, verified):
    """Rows of the walked nodes (host view before the re-root)."""
    rows, v = [], 0
    for t in verified[1:]:
        kids = [c for c in range(len(tree_tok)) if tree_par[c] == v and tree_tok[c] == t]
        if not kids:
            break
        v = kids[0]
        if tree_row[v] >= 0:
            rows.append(int(tree_row[v]))
    return rows


@pytest.mark.parametrize("seed", range(3))
def test_draft_loop_keeps_device_rows_consistent(seed):
    rng = np.random.default_rng(seed)
    V, w, k, d, bs = 2048, 4, 3, 3, 8
    Hkv, D, S_max, P0 = 2, 64, 512, 40
    tree = ss.DraftTree(4096, int(rng.integers(V)))
    kc = torch.zeros((Hkv, S_max, D), dtype=torch.int16, device=dev())
    vc = torch.zeros_like(kc)
    P = torch.tensor([P0], dtype=torch.int32, device=dev())
    ws_r = ss.workspace(1 << 16, dev())
    ws_t = ss.workspace(ss.topk_logprobs_workspace_bytes(w), dev())
    tok_d = torch.zeros((w, k), dtype=torch.int32, device=dev())
    lp_d = torch.zeros((w, k), dtype=torch.float32, device=dev())
    prefix = P0
    for it in range(6):
        for _ in range(d):
            if tree.rows() + w > 64:  # the draft kernels hold at most 64 tree-cache rows
                break
            leaves, prow = tree.select_leaves(w)
            if len(leaves) == 0:
                break
            # the draft's KV rows of the selected non-root leaves: tag = token
            tok_h, _, _, row_h, _ = tree.nodes()
            for v in leaves:
                if v != 0:
                    kc[:, prefix + row_h[v], 0] = int(tok_h[v])
            lg = _logits(len(leaves), V, 0, seed * 100 + it, ties=False)
            ss.topk_logprobs(up(lg), tok_d[:len(leaves)], lp_d[:len(leaves)], ws_t)
            tree.expand(leaves, tok_d[:len(leaves)].cpu().numpy(), lp_d[:len(leaves)].cpu().numpy())
        # a synthetic target output: a root path to some node, then a child's token or a new one
        tok_h, par_h, _, row_h, _ = tree.nodes()
        v = int(rng.integers(len(tok_h)))
        path = []
        while v >= 0:
            path.append(v)
            v = int(par_h[v])
        ver = [int(tok_h[u]) for u in path[::-1]]
        kids = [c for c in range(len(tok_h)) if par_h[c] == path[0]]
        ver.append(int(tok_h[kids[0]]) if kids and rng.random() < 0.7 else V + 1)
        forest = tree.forest()
        walked = _walk_rows(tok_h, par_h, row_h, ver)
        res = tree.reroot(ver)
        N = len(forest)
        if N > 0:
            d_par = up(np.asarray(forest, np.int32))
            last = torch.tensor([res["last"]], dtype=torch.int32, device=dev())
            keep = torch.tensor([res["keep"]], dtype=torch.int32, device=dev())
            newp = torch.full((N,), -7, dtype=torch.int32, device=dev())
            nk = torch.zeros(1, dtype=torch.int32, device=dev())
            ss.kv_reorganize(kc, vc, P, d_par, last, keep, new_parent=newp, n_kept=nk, advance=True, ws=ws_r)
            torch.cuda.synchronize()
            assert int(P.item()) == prefix + res["path_rows"]
            assert [int(x) for x in kc[0, prefix:prefix + res["path_rows"], 0].cpu()] == \
                [int(tok_h[[u for u in range(len(tok_h)) if row_h[u] == r][0]]) for r in walked]
            prefix += res["path_rows"]
            n_kept = int(nk.item())
            assert n_kept == tree.rows()
            assert list(newp[:n_kept].cpu().numpy()) == list(tree.forest())
            t2, _, _, r2, _ = tree.nodes()
            for u in range(1, len(t2)):
                if r2[u] >= 0:
                    assert int(kc[0, prefix + r2[u], 0].item()) == int(t2[u])
        # pending tokens: the draft computes them into the prefix (here: tags)
        for tkn in res["pending"]:
            kc[:, prefix, 0] = tkn
            prefix += 1
        P.fill_(prefix)
        while tree.size() < bs and tree.rows() + w <= 64:
            leaves, _ = tree.select_leaves(w)
            tok_h, _, _, row_h, _ = tree.nodes()
            for v in leaves:
                if v != 0:
                    kc[:, prefix + row_h[v], 0] = int(tok_h[v])
            lg = _logits(len(leaves), V, 0, seed * 100 + 50 + it, ties=False)
            ss.topk_logprobs(up(lg), tok_d[:len(leaves)], lp_d[:len(leaves)], ws_t)
            tree.expand(leaves, tok_d[:len(leaves)].cpu().numpy(), lp_d[:len(leaves)].cpu().numpy())
        nodes, par, toks = tree.select_subgraph(bs)
        assert par[0] == -1 and all(0 <= par[j] < j for j in range(1, len(par)))
