"""The benchmark's work accounting (CPU): the algorithmic flops and bytes that
turn measured kernel times into the reported rates.  Each formula is checked
against numbers worked out by hand from the workload's shapes, or against a
brute-force count on small inputs, so that a dropped term or a wrong factor in
the reported roofline fractions fails here."""
import importlib.util
import json
import os
import types

import numpy as np
import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_gemm_flops_per_token_2b_shapes(bench):
    """18-layer d2048 backbone, 8 heads of 256, GeGLU MLP 16384: per token
    the QKV projection is 2*(3*2048)*2048 flops, O 2*2048*2048, the fused
    gate+up projection 2*(2*16384)*2048 and down 2*16384*2048."""
    bb = W.BackboneSpec(18, 2048, 8, 16384, True)
    f = bench.gemm_flops_per_token(bb)
    assert f == {"gemm_qkv": 25_165_824, "gemm_o": 8_388_608, "gemm_up": 134_217_728, "gemm_down": 67_108_864}
    # one launch of the GeGLU projection over config 3's 75,529 valid tokens
    assert f["gemm_up"] * 75_529 == 10_137_330_778_112


def test_gemm_flops_per_token_grouped_kv_and_gelu(bench):
    """One key/value head of 256 next to 8 query heads: QKV has (8 + 2) * 256
    rows; a plain GELU MLP of 3072 on d 768 counts its up projection once."""
    assert bench.gemm_flops_per_token(W.BackboneSpec(18, 2048, 8, 16384, True, kv_heads=1))["gemm_qkv"] \
        == 2 * 2560 * 2048
    f = bench.gemm_flops_per_token(W.BackboneSpec(12, 768, 12, 3072, False))
    assert f["gemm_up"] == 2 * 3072 * 768 and f["gemm_down"] == 2 * 3072 * 768


def _brute_attention_flops(lens, d, causal):
    # 2*d flops per (query, key) pair for QK^T and 2*d for PV, over the pairs
    # the mask keeps
    total = 0
    for L in lens:
        for q in range(L):
            for k in range(L):
                if causal and k > q:
                    continue
                total += 4 * d
    return total


@pytest.mark.parametrize("causal", [False, True])
def test_attention_flops_match_a_pair_count(bench, causal):
    bb = W.BackboneSpec(3, 128, 4, 256, False, causal=causal)
    spec = types.SimpleNamespace(backbone=bb)
    lens = [1, 7, 16, 33]
    reqs = [types.SimpleNamespace(lengths=np.array(lens[:2])), types.SimpleNamespace(lengths=np.array(lens[2:]))]
    out = bench.kernel_rates({"attention": {"ms": 2.0}}, 2, spec, reqs, T=sum(lens), valid=sum(lens), N=len(lens))
    flops = 3 * _brute_attention_flops(lens, 128, causal)
    assert out["attention"]["tflops"] == pytest.approx(flops / 1e-3 / 1e12, rel=1e-12)


def test_hbm_kernel_bytes(bench):
    """Two layers, d 256, T 40 packed rows of which 36 valid, N 3 samples,
    1 ms per kernel per step:
      pack / unpack: every valid row read and written once in bf16: 36*256*4 B;
      RMSNorm: the first reads bf16 tokens and writes the fp32 residual and the
      bf16 output (8 B/element), the other 2*2 read fp32 and write bf16 (6 B),
      over all T rows: (8 + 24) * 40 * 256 B;
      pool: the valid rows read once in bf16 plus N fp32 rows written:
      36*256*2 + 3*256*4 B;
      rotation (H 4 query heads of 64, 2 KV heads): q and k read and written in
      bf16 per layer: 2 * 4 * 40 * (4 + 2) * 64 B."""
    bb = W.BackboneSpec(2, 256, 4, 512, False, kv_heads=2)
    spec = types.SimpleNamespace(backbone=bb)
    reqs = [types.SimpleNamespace(lengths=np.array([10, 12, 14]))]
    ops = {k: {"ms": 1.0} for k in ("pack", "unpack", "rmsnorm", "pool", "rope")}
    out = bench.kernel_rates(ops, 1, spec, reqs, T=40, valid=36, N=3)
    expect = {"pack": 36 * 256 * 4, "unpack": 36 * 256 * 4, "rmsnorm": 32 * 40 * 256,
              "pool": 36 * 256 * 2 + 3 * 256 * 4, "rope": 2 * 4 * 40 * 6 * 64}
    for op, nbytes in expect.items():
        assert out[op]["GB_per_s"] == pytest.approx(nbytes / 1e-3 / 1e9, rel=1e-12), op
        assert out[op]["frac_of_hbm"] == pytest.approx(out[op]["GB_per_s"] / 8000.0, rel=1e-12), op


def test_measured_traffic_follows_the_kernel_source(bench, tmp_path, monkeypatch):
    """The bench reports the counter-derived traffic only for the workload it
    was taken on and only while the GEMM source has the recorded hash."""
    good = {"config": 3, "kernel_source_sha256_16": bench.source_hash(bench.GEMM_SRC), "bytes_per_launch": 123.0}
    path = tmp_path / "traffic.json"
    path.write_text(json.dumps(good))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(path))
    assert bench.measured_traffic(3) == 123.0
    assert bench.measured_traffic(5) is None
    path.write_text(json.dumps(dict(good, kernel_source_sha256_16="0" * 16)))
    assert bench.measured_traffic(3) is None
    path.write_text("not json")
    assert bench.measured_traffic(3) is None
