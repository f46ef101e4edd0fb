"""The synthetic workload shapes: parameter totals of the models the paper trains."""

import numpy as np
import pytest

import workloads


@pytest.mark.parametrize("name,n", [("opt125m", 125_239_296), ("opt1.3b", 1_315_758_080),
                                    ("opt13b", 12_853_473_280), ("opt30b", 29_974_540_288)])
def test_opt_totals(name, n):
    """OPT decoders with learned positions (2050 rows), biases and two LayerNorms per layer."""
    assert workloads.WORKLOADS[name].n == n


@pytest.mark.parametrize("name,total,non_embedding", [("qwen3-1.7b", 1.7e9, 1.4e9), ("qwen3-8b", 8.2e9, 6.95e9)])
def test_qwen3_totals_match_the_published_sizes(name, total, non_embedding):
    """Qwen3 model sizes as published (total and non-embedding parameters, rounded)."""
    w = workloads.WORKLOADS[name]
    emb = sum(sz for nm, sz, _ in workloads.model_tensors(w) if nm in ("embed_tokens", "lm_head.weight"))
    assert abs(w.n / total - 1) < 0.015
    assert abs((w.n - emb) / non_embedding - 1) < 0.01


def test_tensor_offsets_tile_the_buffer():
    for w in workloads.WORKLOADS.values():
        if not w.hidden:
            continue
        spans = workloads.tensor_offsets(w)
        assert spans[0][1] == 0
        for (_, o, sz), (_, o2, _) in zip(spans, spans[1:]):
            assert o + sz == o2
        assert spans[-1][1] + spans[-1][2] == w.n
        kinds = {k for _, _, k in workloads.model_tensors(w)}
        assert kinds <= {"normal", "zero", "one"}


def test_losses_are_seeded():
    a = workloads.synthetic_losses(8, 3)
    b = workloads.synthetic_losses(8, 3)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
