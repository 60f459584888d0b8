"""Per-step compute accounting (Tables I and II report TFLOPs per step).

The tables' figures match one multiply-add per backbone parameter per prompt
token (Llama-2-7B has about 6.74e9 parameters; 276 prompt tokens give
1.86e12, inside Table I's full-inference range, and the 589 tokens of the
parallel-decoded action chunk give 3.97e12, Table II's full-inference
average).  `paper_step_tflops` reproduces that convention; `step_flops` is
the 2*MAC count of the rows a step actually recomputes.
"""


def backbone_params(cfg) -> int:
    """Decoder layers plus the token embedding and the LM head."""
    d, F, L, V = cfg.d_model, cfg.ffn, cfg.n_layers, cfg.vocab
    return L * (4 * d * d + 3 * d * F) + 2 * V * d


def paper_step_tflops(cfg, tokens: int) -> float:
    return backbone_params(cfg) * tokens / 1e12


def layer_macs(cfg, rows: int) -> int:
    d, F = cfg.d_model, cfg.ffn
    return rows * (4 * d * d + 3 * d * F)


def attention_macs(cfg, query_pos, ) -> int:
    """QK^T and PV multiply-adds of queries at the given positions (causal)."""
    d = cfg.d_model
    return sum(2 * (p + 1) * d for p in query_pos)


def step_flops(cfg, rows_per_layer, query_pos_per_layer, head_rows: int, decode_passes: int,
               prompt_len: int) -> int:
    """2*MAC of one control step: the prompt pass over the recomputed rows of
    each layer, the head rows, and the single-token decode passes."""
    d, V = cfg.d_model, cfg.vocab
    macs = 0
    for rows, qp in zip(rows_per_layer, query_pos_per_layer):
        macs += layer_macs(cfg, rows) + attention_macs(cfg, qp)
    macs += head_rows * V * d
    for j in range(decode_passes):
        pos = prompt_len + j
        macs += cfg.n_layers * (layer_macs(cfg, 1) + attention_macs(cfg, [pos])) + V * d
    return 2 * macs
