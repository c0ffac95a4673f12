"""fp64 CPU oracle of the CompressKV eviction path (test infrastructure only).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark
may import this package; the product path never does.
"""
from .compresskv_oracle import (  # noqa: F401
    POOL_MAX, POOL_AVG, POOL_THEN_MEAN, MEAN_THEN_POOL, PER_GROUP, LAYER_SHARED,
    window_logits, row_softmax, window_column_sums, pool1d, group_scores, layer_scores,
    select_tokens, compress_layer, compress_layer_heads, LayerResult,
)
