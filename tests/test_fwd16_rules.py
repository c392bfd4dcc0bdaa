"""The committed output-table rules of the 16-bit forward
(paper_2202_00441_amd/csrc/fwd16_rules.h) are what their generator writes,
and are well formed: per activation and type at most 16 runs, the first at
block 0, strictly increasing starts, known rules; every block a rule covers
agrees with the oracle's forward (its own double-precision f) on all of its
patterns, within the parity tests' 1 ulp.  The kernels that use the rules are
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


def test_rules_agree_with_the_oracle():
    # Every block the rules cover (all but EVAL) reproduces the oracle's
    # forward output (its own double-precision f, one rounding) for each of
    # its 128 patterns, within the 1-ulp bound of the parity tests: the
    # rules are checked on the CPU against the independent implementation,
    # not only against their generator.
    import numpy as np
    import oracle as O
    from parity import ODT, check_y
    g = _gen()
    with open(os.path.join(CSRC, "fwd16_rules.h")) as fh:
        src = fh.read()
    tables = re.findall(r"\{(\d+), \{(.*?)\}\},", src)
    oact = {"gelu": O.GELU, "silu": O.SILU, "sigmoid": O.SIGMOID, "tanh": O.TANH,
            "relu": O.RELU, "selu": O.SELU, "softplus": O.SOFTPLUS}
    pats = np.arange(65536, dtype=np.uint16)
    lam32 = np.float32(g.SELU_LAMBDA)
    for i, (_, body) in enumerate(tables):
        act, dt = g.ACTS[i // len(g.DTYPES)], g.DTYPES[i % len(g.DTYPES)]
        y_ref, _ = O.fwd(oact[act], ODT[dt], 1, np.float32([0.0]), pats)
        x32 = O.widen_array(ODT[dt], pats).astype(np.float32)
        runs = [(int(s), r, int(p, 16)) for s, r, p in re.findall(r"run\((\d+), (\w+), 0x([0-9a-f]{4})\)", body)]
        covered = 0
        for k, (start, rule, payload) in enumerate(runs):
            end = runs[k + 1][0] if k + 1 < len(runs) else 512
            if rule == "EVAL":
                continue
            p = pats[start * 128:end * 128]
            if rule == "IDENTITY":
                y = p.copy()
            elif rule == "CONST":
                y = np.full_like(p, payload)
            elif rule == "HALF":
                y = p - np.uint16(0x80 if dt == "bf16" else 0x400)
            else:   # SCALE: the fp32 product with lambda, one rounding
                y = O.round_array(ODT[dt], (x32[start * 128:end * 128] * lam32).astype(np.float64))
            check_y(y.astype(np.uint16), y_ref[start * 128:end * 128], dt, f"{act} {dt} {rule} run at block {start}")
            covered += end - start
        assert covered >= 200, (act, dt, covered)     # much of every table follows a rule
