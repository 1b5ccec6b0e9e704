"""The seeded input recipe is deterministic and has the stated shapes."""

import torch

import workloads as W


def test_same_seed_same_bytes():
    a = W.attention_inputs(300, 2, 1, 128, 7)
    b = W.attention_inputs(300, 2, 1, 128, 7)
    for x, y in zip(a, b):
        assert x.dtype == torch.bfloat16
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))
    c = W.attention_inputs(300, 2, 1, 128, 8)
    assert not torch.equal(a[0], c[0])


def test_layer_shapes_and_scale():
    x, wqkv, wo, dy = W.layer_inputs(64, 256, 4, 1, 128, 3)
    assert x.shape == (64, 256) and dy.shape == (64, 256)
    assert wqkv.shape == (256, 6 * 128) and wo.shape == (512, 256)
    assert 0.015 < wqkv.float().std().item() < 0.025
    assert 0.9 < x.float().std().item() < 1.1


def test_flop_convention():
    fwd, bwd = W.attention_flops(131072, 4, 128)
    assert abs((fwd + bwd) - 6.157e13) / 6.157e13 < 1e-3
    assert W.causal_pairs(4) == 10
