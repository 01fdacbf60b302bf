"""CPU oracle (test infrastructure only; see litetopk_oracle)."""
from .litetopk_oracle import (  # noqa: F401
    PAD_INDEX, PAD_SCORE, bf16_to_f64, dequantize, e4m3fn_to_f64, index_scores, indexer_topk,
    order, row_scores, select_row, topk_select, visible_counts,
)
