"""The algorithmic-byte model used for every roofline figure in this repo
(int4 weights K*N/2 bytes plus fp16 scale and uint8 zero per 128-group) and
the flop model 2*M*K*N reproduce the utilisation percentages the paper prints
for int4 AWQ Llama-3-70B at tensor-parallel degree 4, batch 8."""
import os

import pytest

from gen.workloads import LLAMA_70B

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tab_utilization.txt")
HBM_H800 = 3.35e12
MFMA_H800 = 989.4e12


def _load():
    rows = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        name, t, comp, band = line.split()
        rows[name] = (float(t) * 1e-6, float(comp), float(band))
    return rows


def _w4_bytes(K, N):
    return K * N // 2 + (K // 128) * N * (2 + 1)


def _shards(tp=4):
    s = LLAMA_70B
    return {  # column-parallel projections split N, row-parallel split K
        "qkv_projection": [(s.H, s.n_qkv // tp)],
        "o_projection": [(s.Hq * s.D // tp, s.H)],
        "swiglu": [(s.H, s.F // tp), (s.H, s.F // tp)],
        "down_projection": [(s.F // tp, s.H)],
    }


@pytest.mark.parametrize("op", ["qkv_projection", "o_projection", "swiglu", "down_projection"])
def test_byte_and_flop_models_reproduce_printed_utilisation(op):
    t, comp, band = _load()[op]
    mats = _shards()[op]
    nbytes = sum(_w4_bytes(K, N) for K, N in mats)
    flops = sum(2 * 8 * K * N for K, N in mats)
    band_pred = 100 * nbytes / t / HBM_H800
    comp_pred = 100 * flops / t / MFMA_H800
    assert band_pred == pytest.approx(band, rel=0.06)
    assert comp_pred == pytest.approx(comp, rel=0.03)


def test_layer_byte_model_is_the_sum_of_its_matrices():
    s = LLAMA_70B
    assert s.w4_bytes() == sum(_w4_bytes(K, N) for _, K, N in s.gemms())
    assert s.w4_bytes() == 447_873_024
