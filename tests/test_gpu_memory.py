"""Activation memory held for the backward pass (Sec. 2; memory tables of
Sec. 4): on a stack of feed-forward blocks the few-bit activation keeps
ceil(n b / 32) words instead of its n-element input, and nothing else
changes, so the saving is exact and the saved fraction equals the paper's
formula Nonlin * (1 - b / bits_per_element) / All."""
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2202_00441_amd.memory import compare  # noqa: E402


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16, torch.float32])
@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_saving_is_exact_and_matches_the_papers_formula(dtype, bits):
    # sizes chosen so every tensor is a multiple of the allocator's 512 bytes
    r = compare(d=64, d_ff=256, layers=3, tokens=512, bits=bits, dtype=dtype)
    print(r, flush=True)
    assert r["saved_bytes"] == r["expected_saved_bytes"]
    assert r["allocator_saved_bytes"] == r["expected_saved_bytes"]
    assert r["saved_fraction"] == pytest.approx(r["paper_formula_fraction"], rel=1e-12)


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_saving_is_exact_at_ragged_sizes(bits):
    # odd token count: code buffers end in a partial word; the saved tensors
    # still account exactly (the allocator rounds its blocks, so only the
    # tensor bytes are compared)
    r = compare(d=48, d_ff=200, layers=2, tokens=333, bits=bits, dtype=torch.bfloat16)
    assert r["saved_bytes"] == r["expected_saved_bytes"]


def test_fewbit_stack_trains():
    # the backward through the few-bit stack runs and gives finite gradients
    from paper_2202_00441_amd.autograd import FewBitAct
    from paper_2202_00441_amd.memory import ffn_stack
    torch.manual_seed(0)
    act = FewBitAct("gelu", 3)
    model = ffn_stack(64, 256, 2, lambda: act, torch.bfloat16, "cuda")
    x = torch.randn(300, 64, device="cuda", dtype=torch.bfloat16)
    model(x).float().square().mean().backward()
    for p in model.parameters():
        assert p.grad is not None and bool(torch.isfinite(p.grad.float()).all())
