"""Oracle byte and parameter accounting.

Test infrastructure only (see ``oracle/__init__.py``).
"""

from __future__ import annotations


def bf16_kv_bytes_per_token(layers: int, kv_heads: int, head_dim: int) -> int:
    """BF16 cache bytes per token: key and value, 2 bytes each, per layer and KV head.

    Paper, Decode-time breakdown appendix (512 bytes per KV head per token at
    head_dim 128) and the GPT-OSS architecture table (KV bytes/token row).
    """
    return 2 * layers * kv_heads * head_dim * 2


def code_bytes_per_token_head(head_dim: int, group_dim: int = 4, bits: int = 8) -> int:
    """K + V code bytes of one token of one KV head: one b-bit index per group, per side."""
    return 2 * (head_dim // group_dim) * bits // 8


def decode_code_bytes(batch: int, kv_heads: int, attended: int, head_dim: int,
                      group_dim: int = 4) -> int:
    """Code bytes one decode step reads (K and V codes of every attended token-head)."""
    return batch * kv_heads * attended * code_bytes_per_token_head(head_dim, group_dim)


def params_scalars(head_dim: int, group_dim: int = 4, codebook_size: int = 256,
                   value_codebooks: bool = False) -> int:
    """Stored scalars per (layer, KV head): 3 d^2 + d + L * 2^{gb} * g.

    Paper, Sec. "Reported quantities" (three d x d transforms, the mean and the
    key codebooks).  ``value_codebooks`` adds the value-side codebooks of the VQ
    value arm.
    """
    L = head_dim // group_dim
    n = 3 * head_dim * head_dim + head_dim + L * codebook_size * group_dim
    if value_codebooks:
        n += L * codebook_size * group_dim
    return n


def params_bits(head_dim: int, group_dim: int = 4, codebook_size: int = 256,
                transform_bits: int = 16, codebook_bits: int = 8) -> int:
    """Bits per (layer, KV head) at the given transform and codebook precisions."""
    L = head_dim // group_dim
    return (3 * head_dim * head_dim + head_dim) * transform_bits + \
        L * codebook_size * group_dim * codebook_bits


def vq_bits_per_element(head_dim: int, group_dim: int = 4, codebook_size: int = 256,
                       per_token_bits: int = 0) -> float:
    """Stored bits per element of a VQ'd cache side: log2(k)/g index bits plus per-token metadata.

    Paper, Sec. "Bit rate": one 8-bit index per group of 4 entries is 2 bits per
    element; a per-token BF16 scale adds 16/head_dim.
    """
    import math
    return math.log2(codebook_size) / group_dim + per_token_bits / head_dim


def sq_bits_per_element(head_dim: int, bits: int = 2, per_token_bits: int = 32) -> float:
    """Scalar-quantized side: ``bits`` per element plus per-token scale/offset bits."""
    return bits + per_token_bits / head_dim


def band_overhead_bpe(context: int, band_tokens: int, base_bpe: float, band_bits: int = 16) -> float:
    """Extra bits per element of a full-precision sink+recent band of band_tokens tokens."""
    return band_tokens * (band_bits - base_bpe) / context
