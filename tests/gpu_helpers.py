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


def check_close(got_bits, ref_bits, what="", atol=ATOL, rtol=RTOL):
    g, r = f64(got_bits), f64(ref_bits)
    assert np.all(np.isfinite(g)), f"{what}: non-finite GPU output"
    err = np.abs(g - r)
    bound = atol + rtol * np.abs(r)
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


class DeviceStep:
    """The whole verification step of a workload on the GPU: n_layers decoder
    layers (caches in one [n_layers][Hkv][S_max][D] allocation each for K and
    V), final RMSNorm and LM head.  source="host" uploads the seeded host
    recipe (gen.workloads, comparable with the reference); source="device"
    draws the same recipe on the GPU (gen.device; timing and self-checks
    only)."""

    def __init__(self, cfg, n_layers, source="host", rope_theta=500000.0, with_head=True):
        from gen import device as gdev
        from gen.workloads import (W_STREAMS, LAYER_STREAM_STRIDE, FINAL_NORM_STREAM, LM_HEAD_STREAM,
                                   make_final_norm, make_kv_prefix, make_layer_weights, make_lm_head, make_tree)
        s = cfg.shape
        self.cfg, self.n_layers = cfg, n_layers
        seed = cfg.seeds()["weights"]
        shape = (n_layers, s.Hkv, cfg.S_max, s.D)
        self.kc = torch.zeros(shape, dtype=torch.int16, device=dev())
        self.vc = torch.zeros(shape, dtype=torch.int16, device=dev())
        self.keep, descs = [], []
        for l in range(n_layers):
            if source == "host":
                w = make_layer_weights(cfg, l)
                kc, vc = make_kv_prefix(cfg, l)
                self.kc[l].copy_(up(kc))
                self.vc[l].copy_(up(vc))
                w4 = {}
                for name in ("wqkv", "wo", "wgate", "wup", "wdown"):
                    t, d = upload_w4(w[name])
                    self.keep.append(t)
                    w4[name] = d
                an, mn = up(w["attn_norm"]), up(w["mlp_norm"])
            else:
                base = l * LAYER_STREAM_STRIDE
                w4 = {}
                for name, K, N in s.gemms():
                    q, sc, z = gdev.w4_random_device(seed, base + W_STREAMS[name], N, K, device=dev())
                    d = ss.make_w4(q, sc, z)
                    packed = ss.prepack_w4(d)
                    self.keep.append((q, sc, z, packed))
                    w4[name] = d
                an = gdev.normal_f16_device(seed, base + W_STREAMS["attn_norm"], (s.H,), 1.0, 0.02, dev())
                mn = gdev.normal_f16_device(seed, base + W_STREAMS["mlp_norm"], (s.H,), 1.0, 0.02, dev())
                kv_seed = cfg.seeds()["kv"]
                if cfg.P > 0:
                    self.kc[l, :, :cfg.P] = gdev.normal_f16_device(kv_seed, 2 * l, (s.Hkv, cfg.P, s.D), device=dev())
                    self.vc[l, :, :cfg.P] = gdev.normal_f16_device(kv_seed, 2 * l + 1, (s.Hkv, cfg.P, s.D),
                                                                   device=dev())
            self.keep.append((an, mn))
            descs.append(ss.make_layer(an, mn, w4["wqkv"], w4["wo"], w4["wgate"], w4["wup"], w4["wdown"],
                                       self.kc[l], self.vc[l]))
        self.layers = ss.make_layers(descs)
        self.layer_descs = descs
        self.V = cfg.vocab if with_head else 0
        self.final_norm = self.lm_w = None
        if self.V:
            if source == "host":
                self.final_norm = up(make_final_norm(cfg))
                self.lm_w = up(make_lm_head(cfg))
            else:
                self.final_norm = gdev.normal_f16_device(seed, FINAL_NORM_STREAM, (s.H,), 1.0, 0.02, dev())
                self.lm_w = gdev.normal_f16_device(seed, LM_HEAD_STREAM, (self.V, s.H), 0.0, 0.02, dev())
        self.parent_h, self.acc = make_tree(cfg)
        self.parent = up(np.asarray(self.parent_h, np.int32))
        self.P = up(np.array([cfg.P], np.int32))
        self.rope = up(ss.rope_table(rope_theta, cfg.S_max, s.D))
        self.dims = ss.make_dims(s.H, s.Hq, s.Hkv, s.D, s.F, cfg.S_max)
        self.ws = ss.workspace(ss.verify_step_workspace_bytes(self.dims, cfg.T, self.V), dev())
        self.logits = torch.zeros((cfg.T, max(self.V, 1)), dtype=torch.int16, device=dev())

    def enqueue(self, hidden, stream=None):
        ss.verify_step(self.layers, self.dims, hidden, self.P, self.parent, self.rope, self.ws,
                       self.final_norm, self.lm_w, self.logits if self.V else None, stream=stream)
