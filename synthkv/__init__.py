"""Seeded synthetic inputs for KV-cache migration and the weight-shard rebuild
(shared by the oracle's tests, the GPU tests and the benchmark; holds no
migration or slicing arithmetic)."""
from .configs import KVWorkload, WORKLOADS, TINY, MHA_7B, MHA_13B, GQA_70B, GQA_70B_LONG, QWEN3_30B, DS_32B, reduced
from .gen import (BlockTables, Inputs, make_inputs, make_tables, seq_lens, tables_from_rows,
                  fill_words_, fill_pool_layer_, fill_sentinel_, words_at, bytes_at, stream_key,
                  torch_dtype_for, numpy_dtype_for, SOURCE, SENTINEL)
from . import models
from .models import (DecoderSpec, DECODERS, TINY_DECODER, ODD_DECODER, TINY_BIAS, TINY_MOE, LLAMA2_7B,
                     LLAMA3_70B, QWEN2_32B, QWEN3_30B_A3B)

__all__ = [
    "models", "DecoderSpec", "DECODERS", "TINY_DECODER", "ODD_DECODER", "TINY_BIAS", "TINY_MOE", "LLAMA2_7B",
    "LLAMA3_70B", "QWEN2_32B", "QWEN3_30B_A3B",
    "KVWorkload", "WORKLOADS", "TINY", "MHA_7B", "MHA_13B", "GQA_70B", "GQA_70B_LONG", "QWEN3_30B", "DS_32B",
    "reduced",
    "BlockTables", "Inputs", "make_inputs", "make_tables", "seq_lens", "tables_from_rows",
    "fill_words_", "fill_pool_layer_", "fill_sentinel_", "words_at", "bytes_at", "stream_key",
    "torch_dtype_for", "numpy_dtype_for", "SOURCE", "SENTINEL",
]
