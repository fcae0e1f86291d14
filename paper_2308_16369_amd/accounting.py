"""Throughput accounting of the hybrid batch (host arithmetic only).

Decode cost follows Sec. 5.1.1: for a decode-only batch the time per decode
token is the iteration time divided by the batch size; for a decode-maximal
batch of p prefill and d decode tokens it is the difference between the
hybrid iteration and a prefill-only iteration of the same p tokens, divided
by d (the marginal decode time).  The maximum decode batch follows the
equation of Sec. 4.3.1: B = floor((M_G - M_S) / (L * m_kv)).
"""
from __future__ import annotations

import math


def decode_time_per_token_baseline(t_decode_only: float, batch: int) -> float:
    """Decode-only iteration time / its batch size (Sec. 5.1.1)."""
    if batch <= 0:
        raise ValueError("batch must be positive")
    return t_decode_only / batch


def decode_time_per_token_hybrid(t_hybrid: float, t_prefill_only: float, n_decodes: int) -> float:
    """(decode-maximal time - prefill-only time) / decodes (Sec. 5.1.1)."""
    if n_decodes <= 0:
        raise ValueError("n_decodes must be positive")
    return (t_hybrid - t_prefill_only) / n_decodes


def max_decode_batch(mem_gpu: float, mem_params: float, max_seq_len: int, kv_bytes_per_token: float) -> int:
    """B = floor((M_G - M_S) / (L * m_kv)) (Sec. 4.3.1); piggybacked decodes
    are then at most B - 1."""
    return int(math.floor((mem_gpu - mem_params) / (max_seq_len * kv_bytes_per_token)))


def tokens_per_second(n_tokens: int, seconds: float) -> float:
    return n_tokens / seconds
