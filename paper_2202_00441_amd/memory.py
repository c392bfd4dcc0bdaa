"""Activation memory held for the backward pass, vanilla vs few-bit (Sec. 2;
the memory tables of Sec. 4 and Appendix B).

A pointwise activation normally keeps its input (s bytes per element) for
the backward pass; the few-bit one keeps ceil(n b / 32) words of packed
codes.  On a stack of transformer feed-forward blocks, x -> x + W2 f(W1 x),
every other tensor autograd keeps is the same in both variants (each Linear
keeps its input), so the difference is exactly
    layers * (n s - 4 ceil(n b / 32))   bytes, n = tokens * d_ff,
and the saved fraction equals the paper's formula
    Nonlin * (1 - b / (8 s)) / All
up to the word rounding, Nonlin being the activation inputs and All every
saved tensor.
"""
from __future__ import annotations

import torch

from .autograd import FewBitAct


class FFNBlock(torch.nn.Module):
    def __init__(self, d: int, d_ff: int, act: torch.nn.Module):
        super().__init__()
        self.up = torch.nn.Linear(d, d_ff)
        self.act = act
        self.down = torch.nn.Linear(d_ff, d)

    def forward(self, x):
        return x + self.down(self.act(self.up(x)))


def ffn_stack(d: int, d_ff: int, layers: int, act_factory, dtype, device) -> torch.nn.Module:
    """`layers` feed-forward blocks with random weights (seeded by caller)."""
    blocks = [FFNBlock(d, d_ff, act_factory()) for _ in range(layers)]
    return torch.nn.Sequential(*blocks).to(device=device, dtype=dtype)


def held_for_backward(model: torch.nn.Module, x: torch.Tensor) -> tuple:
    """What autograd keeps for the backward pass, two ways:
      * tensor bytes: the storages handed to autograd (saved-tensor hook),
        parameters excluded, each storage once;
      * allocator bytes: device memory still allocated after the forward
        beyond its input and output (the caching allocator's block sizes,
        so allocations above 1 MiB are rounded up).
    One forward and backward run first, so that one-time allocations
    (library workspaces) are not counted."""
    model(x).sum().backward()
    model.zero_grad(set_to_none=True)
    params = {p.untyped_storage().data_ptr() for p in model.parameters()}
    storages = {}

    def pack(t):
        st = t.untyped_storage()
        if st.data_ptr() not in params:
            storages[st.data_ptr()] = st.nbytes()
        return t

    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    with torch.autograd.graph.saved_tensors_hooks(pack, lambda t: t):
        out = model(x)
    torch.cuda.synchronize()
    allocator = torch.cuda.memory_allocated() - base - out.numel() * out.element_size()
    out.sum().backward()               # run the backward once, then free everything
    del out
    model.zero_grad(set_to_none=True)
    return sum(storages.values()), allocator


def compare(d: int, d_ff: int, layers: int, tokens: int, bits: int, dtype=torch.bfloat16,
            act: str = "gelu", device: str = "cuda", seed: int = 0) -> dict:
    """Held-for-backward bytes of the vanilla and the few-bit stack, with the
    expected difference and the paper's saving formula."""
    s = torch.empty((), dtype=dtype).element_size()
    vanilla_act = {"gelu": lambda: torch.nn.GELU(), "silu": lambda: torch.nn.SiLU(),
                   "sigmoid": lambda: torch.nn.Sigmoid(), "tanh": lambda: torch.nn.Tanh()}[act]
    fewbit = FewBitAct(act, bits)               # one fitted table, shared by all layers
    res = {}
    for name, factory in (("vanilla", vanilla_act), ("fewbit", lambda: fewbit)):
        torch.manual_seed(seed)
        model = ffn_stack(d, d_ff, layers, factory, dtype, device)
        x = torch.randn(tokens, d, device=device, dtype=dtype)
        res[name] = held_for_backward(model, x)
        del model, x
        torch.cuda.empty_cache()
    n = tokens * d_ff
    words = (n * bits + 31) // 32
    nonlin = layers * n * s                      # activation inputs (vanilla)
    (tv, av), (tf, af) = res["vanilla"], res["fewbit"]
    return {
        "d": d, "d_ff": d_ff, "layers": layers, "tokens": tokens, "bits": bits,
        "dtype": str(dtype).replace("torch.", ""), "act": act,
        "saved_tensor_bytes_vanilla": tv, "saved_tensor_bytes_fewbit": tf,
        "allocator_bytes_vanilla": av, "allocator_bytes_fewbit": af,
        "saved_bytes": tv - tf,
        "expected_saved_bytes": layers * (n * s - 4 * words),
        "allocator_saved_bytes": av - af,
        "saved_fraction": (tv - tf) / tv,
        "paper_formula_fraction": nonlin * (1 - bits / (8 * s)) / tv,
    }
