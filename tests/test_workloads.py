"""Byte accounting of the decode sweep, pinned to the figures the paper prints."""
import json
import os

from synth import workloads as wl

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_byte_accounting.json")))


def test_qwen72b_bytes_per_token_matches_paper():
    g = GOLD["qwen25_72b_int8_rowscale_gb_per_token"]
    m = wl.QWEN25_72B
    # the model also reads per-layer vectors: q/k/v biases and two norms per layer, one final norm
    vectors = (m.layers * (m.n_q * m.head_dim + 2 * m.n_kv * m.head_dim) + m.layers * 2 * m.d + m.d)
    b = wl.bytes_per_token(m, wl.I8) + vectors * 2
    assert round(b / 1e9, g["decimals"]) == g["value"]
    # the matrices and scales alone are within 0.01 GB of it; the embedding table is excluded
    assert abs(wl.bytes_per_token(m, wl.I8) / 1e9 - g["value"]) < 0.01
    assert (b + wl.embedding_bytes(m, wl.I8)) / 1e9 > g["value"] + 1.0
    for tok_s, gbps in GOLD["qwen25_72b_logical_rates"]["pairs_tok_s_to_gbps"]:
        assert round(tok_s * g["value"]) == gbps


def test_protocol_matrix_bytes():
    g = GOLD["protocol_matrix_mb"]
    assert round(g["rows"] * g["cols"] / 1e6, g["decimals"]) == g["value"]


def test_sweep_bytes_closed_forms():
    # Llama-3-8B shape in q4 (16 + 2 bytes per 32 weights) and Llama-70B shape in bf16
    assert wl.bytes_per_token(wl.LLAMA3_8B, wl.Q4) == 4_221_370_368
    assert wl.bytes_per_token(wl.LLAMA_70B, wl.BF16) == 139_003_428_864
    assert wl.footprint_bytes(wl.LLAMA_70B, wl.BF16) == 141_104_775_168
    mats = wl.decode_matrices(wl.LLAMA3_8B)
    assert len(mats) == 32 * 7 + 1 and mats[-1].name == "lm_head"
    assert [m.name for m in mats[:7]] == ["q", "k", "v", "o", "gate", "up", "down"]
    weights = sum(m.M * m.K for m in mats)
    assert weights * 9 // 16 == wl.bytes_per_token(wl.LLAMA3_8B, wl.Q4)
