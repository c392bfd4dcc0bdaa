"""The committed output-table rules of the 16-bit forward
(paper_2202_00441_amd/csrc/fwd16_rules.h) are what their generator writes,
and are well formed: per activation and type at most 16 runs, the first at
block 0, strictly increasing starts, known rules.  The rules themselves are
checked on the GPU against the oracle over every 16-bit input pattern
(tests/test_gpu_parity.py, test_every_input_pattern)."""
import importlib.util
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2202_00441_amd", "csrc")


def _gen():
    spec = importlib.util.spec_from_file_location("gen_fwd16_rules",
                                                  os.path.join(CSRC, "gen_fwd16_rules.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_header_is_the_generators_output():
    text, _ = _gen().generate()
    with open(os.path.join(CSRC, "fwd16_rules.h")) as fh:
        assert fh.read() == text


def test_runs_are_well_formed():
    g = _gen()
    with open(os.path.join(CSRC, "fwd16_rules.h")) as fh:
        src = fh.read()
    tables = re.findall(r"\{(\d+), \{(.*?)\}\},", src)
    assert len(tables) == len(g.ACTS) * len(g.DTYPES)
    for i, (count, body) in enumerate(tables):
        # the kernel tests for SCALE only in SELU's table
        assert ("SCALE" in body) == (g.ACTS[i // len(g.DTYPES)] == "selu")
        runs = re.findall(r"run\((\d+), (\w+), 0x([0-9a-f]{4})\)", body)
        assert int(count) == len(runs) <= g.MAX_RUNS
        starts = [int(r[0]) for r in runs]
        assert starts[0] == 0 and all(a < b for a, b in zip(starts, starts[1:]))
        assert starts[-1] < 512
        assert {r[1] for r in runs} <= set(g.RULE_NAMES.values())


def test_rounding_to_bf16_matches_torch():
    import numpy as np
    import torch
    g = _gen()
    rng = np.random.default_rng(3)
    v = np.concatenate([rng.normal(0, 1, 20000), rng.normal(0, 1e-38, 5000),
                        rng.normal(0, 1e38, 2000), [0.0, -0.0, np.inf, -np.inf, 3.4e38, -1e-45]])
    mine = g.round_to("bf16", v)
    # torch rounds fp32 -> bf16 to nearest even; these doubles are first made fp32-exact
    v32 = v.astype(np.float32)
    ref = torch.from_numpy(v32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(g.round_to("bf16", v32.astype(np.float64)), ref.astype(np.uint32))
    assert mine.shape == v.shape
