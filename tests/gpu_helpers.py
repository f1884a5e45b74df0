"""Helpers shared by the GPU parity tests: upload seeded host inputs, build
library descriptors, and compare fp16 results with the fp64 reference
checker under the tolerance |gpu - ref| <= 2e-3 + 1e-2 |ref|."""
import numpy as np
import torch

import paper_2506_11309_amd as ss

ATOL = 2e-3
RTOL = 1e-2


def dev():
    return torch.device("cuda:0")


def up(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(dev())


def down16(t):
    return t.detach().cpu().numpy().view(np.uint16)


def f64(bits):
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def check_close(got_bits, ref_bits, what=""):
    g, r = f64(got_bits), f64(ref_bits)
    assert np.all(np.isfinite(g)), f"{what}: non-finite GPU output"
    err = np.abs(g - r)
    bound = ATOL + RTOL * np.abs(r)
    bad = err > bound
    big = np.abs(r) >= 0.2
    rel = (err[big] / np.abs(r[big])).max() if big.any() else 0.0
    if bad.any():
        idx = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside tolerance; first at {tuple(idx)}:"
                             f" gpu {g[tuple(idx)]!r} ref {r[tuple(idx)]!r}; max abs err {err.max():.3g}")
    return float(err.max()), float(rel)


def upload_w4(W):
    """Upload a canonical int4 matrix and build its kernel-native copy."""
    t = (up(W["qweight"]), up(W["scales"]), up(W["zeros"]))
    d = ss.make_w4(*t)
    packed = ss.prepack_w4(d)
    return t + (packed,), d


class DeviceLayer:
    """A decoder layer's weights, caches and step inputs on the GPU."""

    def __init__(self, cfg, w, kc, vc, parent, rope_theta=500000.0):
        s = cfg.shape
        self.cfg = cfg
        self.keep = []
        self.w4 = {}
        for name in ("wqkv", "wo", "wgate", "wup", "wdown"):
            t, d = upload_w4(w[name])
            self.keep.append(t)
            self.w4[name] = d
        self.attn_norm = up(w["attn_norm"])
        self.mlp_norm = up(w["mlp_norm"])
        self.kc = up(kc)
        self.vc = up(vc)
        self.parent = up(np.asarray(parent, np.int32))
        self.P = up(np.array([cfg.P], np.int32))
        self.rope = up(ss.rope_table(rope_theta, cfg.S_max, s.D))
        self.dims = ss.make_dims(s.H, s.Hq, s.Hkv, s.D, s.F, cfg.S_max)
        self.layer = ss.make_layer(self.attn_norm, self.mlp_norm, self.w4["wqkv"], self.w4["wo"],
                                   self.w4["wgate"], self.w4["wup"], self.w4["wdown"], self.kc, self.vc)
        self.ws = ss.workspace(ss.verify_layer_workspace_bytes(self.dims, cfg.T), dev())

    def run(self, x_bits):
        h = up(x_bits)
        ss.verify_layer(self.layer, self.dims, h, self.P, self.parent, self.rope, self.ws)
        torch.cuda.synchronize()
        return h
