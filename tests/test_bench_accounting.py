"""The benchmark's algorithmic byte and flop counts (the numerators of every
roofline fraction it reports) against independent counts: the model's own
tensor inventory, parameter totals from the configuration dimensions, and
the per-step figures they imply at each configuration's expected context."""
import pytest

import bench
from paper_2410_02425_amd import synth

# parameters of each configuration (untied embedding and LM head, RMSNorm
# gains, no biases), from its dimensions
PARAMS = {"tiny": 2_106_624, "7b": 6_738_415_616, "13b": 13_015_864_320, "8b": 8_030_261_248,
          "70b": 70_553_706_496}


@pytest.mark.parametrize("name", sorted(PARAMS))
def test_tensor_inventory_matches_the_parameter_count(name):
    shape = synth.SHAPES[name]
    assert sum(r * c for _, _, (r, c) in synth.tensor_shapes(shape)) == PARAMS[name]


@pytest.mark.parametrize("name", ["7b", "13b", "8b", "70b"])
def test_decode_step_weight_bytes_are_the_model_tensors(name):
    """With no rows the step's bytes are its weights: every matrix once in
    bf16 (the embedding table excluded: a step reads only its rows), the
    fp32 norm gains once."""
    shape = synth.SHAPES[name]
    want = 0
    for tname, _, (r, c) in synth.tensor_shapes(shape):
        if tname == "embed":
            continue
        want += r * c * (4 if synth.is_gain(tname) else 2)
    assert bench.decode_step_bytes(shape, 0, 0) == want


@pytest.mark.parametrize("name,rows,ctx,gb", [("8b", 64, 703, 20.92), ("7b", 16, 670, 18.84), ("13b", 32, 670, 43.29),
                                              ("70b", 32, 685, 146.20)])
def test_decode_step_bytes_at_the_expected_context(name, rows, ctx, gb):
    """The full-batch step at the workload's step-weighted mean context: the
    weights, every row's KV cache, the appended K/V and the embedding rows."""
    shape = synth.SHAPES[name]
    got = bench.decode_step_bytes(shape, rows, rows * ctx)
    assert abs(got / 1e9 - gb) < 0.015
    kv_token = 2 * shape.n_layers * shape.n_kv_heads * shape.head_dim * 2
    assert bench.decode_step_bytes(shape, rows, rows * ctx + 1) - got == kv_token


@pytest.mark.parametrize("name,gflop", [("8b", 13.96), ("7b", 12.95), ("13b", 25.38), ("70b", 136.9)])
def test_prefill_flops_per_prompt_token(name, gflop):
    """Linear-layer flops per prompt token (2 per weight of every layer
    matrix), then the causal attention and LM-head terms on top."""
    shape = synth.SHAPES[name]
    d, hd, L, V = shape.d_model, shape.head_dim, shape.n_layers, shape.vocab
    one = bench.prefill_flops(shape, [1])
    attn_1, head = 2 * 1 * 2 * shape.n_heads * hd * L, 2 * d * V
    lin = one - attn_1 - head
    layer_weights = sum(r * c for t, _, (r, c) in synth.tensor_shapes(shape)
                        if t.startswith("layers.") and not synth.is_gain(t))
    assert lin == 2 * layer_weights
    assert abs(lin / 1e9 - gflop) < 0.01 * gflop
    n = 553  # causal pairs n(n+1)/2 per head, QK^T and PV, 2 flops each
    assert bench.prefill_flops(shape, [n]) == n * lin + 2 * n * (n + 1) * shape.n_heads * hd * L + head


def test_gate_up_bytes_per_launch():
    shape = synth.SHAPES["8b"]
    d, F = shape.d_model, shape.ffn_dim
    assert bench.gate_up_bytes(shape, 1, 64) == 2 * F * d * 2 + 64 * (d + F) * 2
    assert bench.gate_up_bytes(shape, 3, 100) == 3 * 2 * F * d * 2 + 100 * (d + F) * 2
