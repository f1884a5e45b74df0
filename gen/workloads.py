"""Workload presets: Llama-3-shaped decoder layers verifying a seeded draft tree.

Each preset fixes the layer shape, the prefix length P already in the KV
cache, the tree size T (= GEMM M), the number of tree levels and the maximum
branching factor.  Seeds follow ``1000 * index + {1: weights, 2: activations,
3: KV prefix, 4: tree, 5: accepted path}``.

Recipes (all seeded, all synthetic; no dataset or checkpoint is involved):
  * weights ~ N(0, 0.02) fp16, quantised to int4 with per-(row, 128-group)
    min/max scale and zero point;
  * RMSNorm gains gamma = fp16(1 + 0.02 * N(0, 1));
  * activations ~ N(0, 1) fp16, shape [T][H];
  * KV prefix rows [0, P) ~ N(0, 1) fp16 (taken as already rotated); rows
    [P, S_max) start at zero and receive the tree's keys and values;
  * tree: spine of `levels` nodes, remaining nodes hung on random eligible
    parents, random topological relabelling;
  * accepted node: a uniformly random leaf (the long-context preset takes a
    leaf of maximal depth, so its accepted path has `levels` tokens).
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class LayerShape:
    H: int      # hidden size
    Hq: int     # query heads
    Hkv: int    # key/value heads
    D: int      # head dim
    F: int      # FFN (SwiGLU) width

    @property
    def n_qkv(self) -> int:
        return (self.Hq + 2 * self.Hkv) * self.D

    def gemms(self):
        """(name, K, N) of the four int4 weight matrices of one layer (gate/up counted once each)."""
        return [("wqkv", self.H, self.n_qkv), ("wo", self.Hq * self.D, self.H),
                ("wgate", self.H, self.F), ("wup", self.H, self.F), ("wdown", self.F, self.H)]

    def w4_bytes(self) -> int:
        """Algorithmic bytes of the layer's int4 weights: K*N/2 + (K/128)*N*(2 + 1)."""
        return sum(K * N // 2 + (K // 128) * N * 3 for _, K, N in self.gemms())


@dataclass(frozen=True)
class WorkloadConfig:
    index: int
    name: str
    shape: LayerShape
    P: int            # prefix tokens already in the KV cache
    T: int            # draft-tree tokens verified in one step
    levels: int       # tree levels (longest root-to-leaf path, in nodes)
    branching: int    # maximum children per node
    n_layers: int = 1
    vocab: int = 0    # LM head rows (0: no LM head)
    deepest_leaf: bool = False

    @property
    def S_max(self) -> int:
        return self.P + self.T

    def seeds(self) -> dict:
        return seeds_for(self.index)

    def kv_bytes_per_layer(self) -> int:
        s = self.shape
        return 2 * s.Hkv * (self.P + self.T) * s.D * 2


def seeds_for(index: int) -> dict:
    base = 1000 * index
    return {"weights": base + 1, "activations": base + 2, "kv": base + 3, "tree": base + 4,
            "path": base + 5}


LLAMA_1B = LayerShape(H=2048, Hq=32, Hkv=8, D=64, F=8192)
LLAMA_8B = LayerShape(H=4096, Hq=32, Hkv=8, D=128, F=14336)
LLAMA_70B = LayerShape(H=8192, Hq=64, Hkv=8, D=128, F=28672)

CONFIGS = {
    "c1": WorkloadConfig(1, "llama3-1b-layer", LLAMA_1B, P=512, T=8, levels=4, branching=2),
    "c2": WorkloadConfig(2, "llama3-8b-layer", LLAMA_8B, P=2048, T=16, levels=6, branching=3),
    "c3": WorkloadConfig(3, "llama3-70b-layer", LLAMA_70B, P=4096, T=32, levels=8, branching=4),
    "c4": WorkloadConfig(4, "llama3-8b-long-context", LLAMA_8B, P=32768, T=64, levels=10,
                         branching=4, deepest_leaf=True),
    "c5": WorkloadConfig(5, "llama3-70b-80-layers", LLAMA_70B, P=8192, T=64, levels=8,
                         branching=4, n_layers=80, vocab=128256),
}

# stream ids within the weight seed, per layer
W_STREAMS = {"wqkv": 0, "wo": 1, "wgate": 2, "wup": 3, "wdown": 4, "attn_norm": 5,
             "mlp_norm": 6}
LAYER_STREAM_STRIDE = 16
FINAL_NORM_STREAM = 1 << 40
LM_HEAD_STREAM = (1 << 40) + 1


def make_layer_weights(cfg: WorkloadConfig, layer: int = 0) -> dict:
    """int4 weights and RMSNorm gains of one layer, as numpy arrays."""
    from . import normal_f16, w4_random
    s = cfg.shape
    seed = cfg.seeds()["weights"]
    base = layer * LAYER_STREAM_STRIDE
    out = {}
    for name, K, N in s.gemms():
        q, sc, z = w4_random(seed, base + W_STREAMS[name], N, K, std=0.02)
        out[name] = {"qweight": q, "scales": sc, "zeros": z, "K": K, "N": N}
    out["attn_norm"] = normal_f16(seed, base + W_STREAMS["attn_norm"], (s.H,), 1.0, 0.02)
    out["mlp_norm"] = normal_f16(seed, base + W_STREAMS["mlp_norm"], (s.H,), 1.0, 0.02)
    return out


def make_kv_prefix(cfg: WorkloadConfig, layer: int = 0):
    """K and V caches [Hkv][S_max][D] fp16 bits; rows [0, P) drawn, the rest zero."""
    import numpy as np
    from . import normal_f16
    s = cfg.shape
    seed = cfg.seeds()["kv"]
    caches = []
    for which in range(2):
        c = np.zeros((s.Hkv, cfg.S_max, s.D), np.uint16)
        if cfg.P > 0:
            c[:, :cfg.P, :] = normal_f16(seed, layer * 2 + which, (s.Hkv, cfg.P, s.D))
        caches.append(c)
    return caches[0], caches[1]


def make_activations(cfg: WorkloadConfig):
    from . import normal_f16
    return normal_f16(cfg.seeds()["activations"], 0, (cfg.T, cfg.shape.H))


def make_tree(cfg: WorkloadConfig):
    """(parent int32[T], accepted node)."""
    from . import accept_leaf, tree
    seeds = cfg.seeds()
    parent = tree(cfg.T, cfg.levels, cfg.branching, seeds["tree"])
    acc = accept_leaf(parent, seeds["path"], cfg.deepest_leaf)
    return parent, acc


def make_final_norm(cfg: WorkloadConfig):
    """Final RMSNorm gain [H] fp16 bits (80-layer configuration)."""
    from . import normal_f16
    return normal_f16(cfg.seeds()["weights"], FINAL_NORM_STREAM, (cfg.shape.H,), 1.0, 0.02)


def make_lm_head(cfg: WorkloadConfig, rows=None):
    """LM head W [V][H] fp16 bits, N(0, 0.02); `rows` (a sequence of vocabulary
    indices) returns just those rows, drawn from the same counter positions."""
    import numpy as np
    from . import normal_f16
    H = cfg.shape.H
    seed = cfg.seeds()["weights"]
    if rows is None:
        return normal_f16(seed, LM_HEAD_STREAM, (cfg.vocab, H), 0.0, 0.02)
    out = np.empty((len(rows), H), np.uint16)
    for i, r in enumerate(rows):
        out[i] = normal_f16(seed, LM_HEAD_STREAM, (H,), 0.0, 0.02, offset=int(r) * H)
    return out
