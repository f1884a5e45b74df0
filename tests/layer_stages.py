"""The reference decoder layer written as its stages, for stage-by-stage
parity checks (host only)."""
import numpy as np

import oracle


def split_qkv(s, qkv):
    Hd = s.Hq * s.D
    return tuple(qkv[:, a:b] for a, b in ((0, Hd), (Hd, Hd + s.Hkv * s.D), (Hd + s.Hkv * s.D, s.n_qkv)))


def oracle_stages(cfg, w, kc, vc, x, parent):
    """The reference layer stage by stage (each stage applied to the previous
    reference stage's output; equal to oracle.verify_layer, which the CPU
    tests pin).  The caches kc, vc (host) are updated in place."""
    s = cfg.shape
    r = {"x": x}
    r["xn"] = oracle.rmsnorm(x, w["attn_norm"])
    r["qkv"] = oracle.w4a16_gemm(w["wqkv"], r["xn"])
    q, k, v = (np.ascontiguousarray(a) for a in split_qkv(s, r["qkv"]))
    r["o"] = oracle.tree_attention(q, k, v, kc, vc, cfg.P, parent, s.Hq, s.Hkv, s.D)
    r["h"] = oracle.w4a16_gemm(w["wo"], r["o"], residual=x)
    r["hn"] = oracle.rmsnorm(r["h"], w["mlp_norm"])
    r["m"] = oracle.w4a16_swiglu(w["wgate"], w["wup"], r["hn"])
    r["out"] = oracle.w4a16_gemm(w["wdown"], r["m"], residual=r["h"])
    return r
