"""Seeded synthetic inputs for the sparse-selection hot path of append prefill.

This package only draws random numbers and lays them out; it holds none of the
method's arithmetic (no scoring, selection, page mapping or attention).  Both
the CPU oracle (through the tests) and the HIP library consume the bytes it
produces.
"""
from .gen import (  # noqa: F401
    Workload,
    AttnInputs,
    make_workload,
    config,
    CONFIG_NAMES,
    attention_inputs,
    attention_kv_fp8,
    KV8_ROW_BYTES,
    attention_q_rows,
    to_fp8_bytes,
    to_bf16_bits,
    quantize_fp8_per_row,
    quantize_mxfp4,
    E2M1_MAGNITUDES,
    synth_topk,
    decode_lengths,
    resident_pages,
)
