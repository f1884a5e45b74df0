"""GPU checks of the draft-side KV reorganisation (swiftspec_kv_reorganize)
against the oracle, bit-exact: random forests up to 64 nodes over several
layers, every forest up to four nodes with every last node and both keep
settings, equality with the target commit when nothing is kept, the Fig. 5
example, and invalid device data (error word, caches untouched)."""
import itertools

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
from gpu_helpers import dev, down16, up  # noqa: E402


def _i32(x):
    return up(np.asarray(x, np.int32).reshape(-1))


def _run(k, v, P, parent, last, keep, n_layers, advance=True):
    N = len(parent)
    dk, dv = up(k), up(v)
    dP = _i32([P])
    newp = torch.full((N,), -9, dtype=torch.int32, device=dev())
    nk = torch.full((1,), -9, dtype=torch.int32, device=dev())
    ws = ss.workspace(ss.WS_HEADER_BYTES, dev())
    ss.kv_reorganize(dk, dv, dP, _i32(parent), _i32([last]), _i32([int(keep)]), new_parent=newp, n_kept=nk,
                     n_layers=n_layers, advance=advance, ws=ws)
    torch.cuda.synchronize()
    return down16(dk), down16(dv), int(dP.item()), newp.cpu().numpy(), int(nk.item()), ss.read_device_error(ws)


def _caches(n_layers, Hkv, S_max, D, seed):
    rng = np.random.default_rng(seed)
    shape = (n_layers, Hkv, S_max, D)
    return (rng.integers(0, 65535, shape).astype(np.uint16), rng.integers(0, 65535, shape).astype(np.uint16))


def _forest(rng, N, root_p=0.2):
    return np.array([-1 if (i == 0 or rng.random() < root_p) else int(rng.integers(0, i)) for i in range(N)],
                    np.int32)


@pytest.mark.parametrize("N,D,Hkv", [(64, 128, 8), (37, 64, 4), (8, 128, 8), (1, 128, 2)])
def test_reorganize_random_forests(N, D, Hkv):
    rng = np.random.default_rng(N * 7 + D)
    n_layers, P = 3, 100
    for trial in range(6):
        parent = _forest(rng, N)
        last = int(rng.integers(-1, N))
        keep = bool(trial % 3)
        k, v = _caches(n_layers, Hkv, P + N + 5, D, trial)
        gk, gv, gP, gnp, gS, err = _run(k, v, P, parent, last, keep, n_layers)
        L, rnp = oracle.kv_reorganize(k, v, P, parent, last, keep, n_layers=n_layers)
        assert err == 0
        assert np.array_equal(gk, k) and np.array_equal(gv, v), (N, trial)
        assert gP == P + L and gS == len(rnp) and np.array_equal(gnp[:gS], rnp)
        print(f"N={N} last={last} keep={keep}: path {L}, kept {gS}")


def test_reorganize_every_small_forest():
    P, Hkv, D = 5, 2, 16
    for N in range(1, 5):
        for par in itertools.product(*[range(-1, i) for i in range(N)]):
            parent = np.array(par, np.int32)
            for last in range(-1, N):
                for keep in (False, True):
                    k, v = _caches(1, Hkv, P + N + 1, D, N)
                    gk, gv, gP, gnp, gS, err = _run(k, v, P, parent, last, keep, 1)
                    L, rnp = oracle.kv_reorganize(k, v, P, parent, last, keep)
                    assert err == 0 and np.array_equal(gk, k) and np.array_equal(gv, v)
                    assert gP == P + L and np.array_equal(gnp[:gS], rnp), (par, last, keep)


def test_without_subtree_equals_commit():
    rng = np.random.default_rng(9)
    for trial in range(5):
        T = int(rng.integers(1, 65))
        parent = np.array([-1] + [int(rng.integers(0, i)) for i in range(1, T)], np.int32)
        acc = int(rng.integers(0, T))
        k, v = _caches(2, 8, 64 + T, 128, trial)
        gk, gv, gP, _, gS, err = _run(k, v, 64, parent, acc, False, 2)
        dk, dv, dP = up(k), up(v), _i32([64])
        ss.kv_commit(dk, dv, dP, _i32(parent), _i32([acc]), n_layers=2, advance=True)
        torch.cuda.synchronize()
        assert err == 0 and gS == 0
        assert np.array_equal(gk, down16(dk)) and np.array_equal(gv, down16(dv)) and gP == int(dP.item())


def test_fig5_example_on_device():
    prefix, tok = [1, 3, 7, 10], [11, 12, 13, 14, 15, 16, 17, 18]
    parent = np.array([-1, -1, 0, 0, 1, 1, 4, 4], np.int32)
    k = np.zeros((1, 1, 14, 8), np.uint16)
    k[0, 0, :4, 0] = prefix
    k[0, 0, 4:12, 0] = tok
    gk, _, gP, gnp, gS, err = _run(k, k.copy(), 4, parent, 4, True, 1)
    assert err == 0 and gP == 6
    assert list(gk[0, 0, :gP, 0]) == [1, 3, 7, 10, 12, 15]
    assert list(gk[0, 0, gP:gP + gS, 0]) == [17, 18] and list(gnp[:gS]) == [-1, -1]


def test_invalid_device_data_leaves_caches():
    k, v = _caches(2, 4, 40, 64, 1)
    bad_forest = np.array([-1, 0, 3, 1], np.int32)          # a parent after its child
    for parent, last, P, bit in ((bad_forest, 1, 10, ss.DEVERR_BAD_TREE),
                                 (np.array([-1, 0, 1, 1], np.int32), 4, 10, ss.DEVERR_BAD_ACCEPTED),
                                 (np.array([-1, 0, 1, 1], np.int32), 2, 37, ss.DEVERR_BAD_PREFIX)):
        gk, gv, gP, gnp, gS, err = _run(k, v, P, parent, last, True, 2)
        assert err & bit
        assert np.array_equal(gk, k) and np.array_equal(gv, v) and gP == P and gS == -9
