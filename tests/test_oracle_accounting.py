"""Pins for the oracle's byte and parameter accounting against the paper's printed numbers."""

import json
import os

import numpy as np

from oracle import accounting as acc

with open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")) as f:
    PAPER = json.load(f)


def test_bf16_bytes():
    assert acc.bf16_kv_bytes_per_token(1, 1, 128) == PAPER["bf16_bytes_per_kv_head_token"]["value"]
    for model in ("llama31_8b", "qwen3_8b", "gpt_oss_20b"):
        layers, kv, d = PAPER["arch"][model]
        assert acc.bf16_kv_bytes_per_token(layers, kv, d) == PAPER["kv_bytes_per_token"][model]


def test_per_gpu_cache_footprint():
    p = PAPER["per_gpu_cache_gb"]
    layers, kv, d = PAPER["arch"]["qwen3_8b"]
    per_gpu_heads = kv // p["tp"]
    b1 = acc.bf16_kv_bytes_per_token(layers, per_gpu_heads, d) * p["context"]
    assert round(b1 / 1e9, 2) == p["batch1"]
    assert round(64 * b1 / 1e9, 2) == p["batch64"]


def test_parameter_storage():
    p = PAPER["params_scalars_per_head"]
    assert acc.params_scalars(128) == sum(p["parts"])
    assert abs(acc.params_scalars(128) - p["approx"]) / p["approx"] < 0.01
    t = PAPER["params_total_gbit"]
    total = acc.params_bits(128) * t["layers"] * t["kv_heads"] / 1e9
    assert round(total, 2) == t["approx"]


def test_bits_per_element():
    p = PAPER["bpe"]
    key = acc.vq_bits_per_element(128, per_token_bits=16)
    val = acc.sq_bits_per_element(128, bits=2, per_token_bits=32)
    assert np.isclose(key, p["key"]) and np.isclose(val, p["value"])
    avg = 0.5 * (key + val)
    assert np.isclose(avg, p["average"])
    band = acc.band_overhead_bpe(p["context"], p["band_tokens"], avg)
    assert round(band, 3) == p["band"]
    assert round(avg + band, 2) == p["total"]
    # this build's format: exactly 2 bits per element for keys and values
    assert acc.vq_bits_per_element(128) == 2.0 and acc.vq_bits_per_element(64) == 2.0
    assert acc.code_bytes_per_token_head(128) == 64 and acc.code_bytes_per_token_head(64) == 32


def test_decode_code_bytes():
    assert acc.decode_code_bytes(8, 8, 16384, 128) == 67_108_864
    assert acc.decode_code_bytes(64, 8, 32768, 128) == 1_073_741_824
    assert acc.decode_code_bytes(16, 8, 65536, 64) == 268_435_456
