"""CPU checks of the torch.optim adapter: parameter routing and argument
validation (no plan is built before the first step)."""
import pytest


def test_routing_and_validation():
    import torch
    from paper_2608_05088_amd.optim import MALT, is_matrix
    w = torch.zeros(8, 16, requires_grad=True)
    b = torch.zeros(16, requires_grad=True)
    c = torch.zeros(4, 3, 3, requires_grad=True)
    opt = MALT([w, b, c], lr=1e-3)
    assert [p is w for p in opt._mats[0]] == [True]
    assert opt._adam is not None and len(opt._adam.param_groups[0]["params"]) == 2
    assert is_matrix(w) and not is_matrix(b) and not is_matrix(c)
    with pytest.raises(ValueError):
        MALT([w], variant="adam")
    with pytest.raises(ValueError):
        MALT([c], matrix_filter=lambda p: True)   # selects a non-2-D tensor


def test_gpt2_block_matrices_are_the_paper_shapes():
    from transformers import GPT2Config, GPT2LMHeadModel
    from paper_2608_05088_amd.train import block_matrix
    m = GPT2LMHeadModel(GPT2Config(n_layer=2, n_embd=64, n_head=4, vocab_size=100, n_positions=32,
                                   bos_token_id=0, eos_token_id=0))
    shapes = [tuple(p.shape) for n, p in m.named_parameters() if block_matrix(n, p)]
    d = 64
    assert shapes == [(d, 3 * d), (d, d), (d, 4 * d), (4 * d, d)] * 2
