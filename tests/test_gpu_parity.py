"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bit-exact on packed codes and grad_in; y within 2e-6 abs + 1e-5 rel (fp32)
or 1 ulp (fp16 / bf16).  Cases: all five workloads at full size (the sizes
the benchmark runs, in its launch configuration), the same workloads cut to
ragged lengths, an edge-size sweep over every dtype x bits x activation,
special values, boundaries, ReLU / SELU / Softplus (Table 1's other rows),
both fp16 / bf16 forward kernels (per-element evaluation, and table lookups
in tables each workgroup builds; chosen by size, or by the table's kernel
flag), the symmetric (|x|) tables of Sigmoid and Tanh, in-place aliasing, a
second stream, three streams running at once, canaries past every output,
and the autograd wrapper.
"""
import numpy as np
import pytest

import oracle as O
import workloads as WL
from parity import (OACT, ODT, TABLES, THREADS, check_exact, check_y, download,
                    download_codes, golden_table, run_case, upload)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2202_00441_amd as P  # noqa: E402

_INPUTS = {}


def inputs(name, limit=None):
    key = (name, limit)
    if key not in _INPUTS:
        _INPUTS.clear()
        _INPUTS[key] = WL.inputs(WL.WORKLOADS[name], limit)
    return _INPUTS[key]


FULL = [(name, b) for name, w in WL.WORKLOADS.items() for b in w.bits]


@pytest.mark.parametrize("name,bits", FULL, ids=[f"{n}-b{b}" for n, b in FULL])
def test_workload_full_size(name, bits):
    w = WL.WORKLOADS[name]
    x, g = inputs(name)
    stats = run_case(f"{name}/b{bits}", w.dtype, x, g, label=f"{name} b{bits} full")
    print(stats, flush=True)


RAGGED = [1, 7, 511, 512, 513, 4097, 100003]


@pytest.mark.parametrize("name,bits", FULL, ids=[f"{n}-b{b}" for n, b in FULL])
def test_workload_ragged_prefixes(name, bits):
    w = WL.WORKLOADS[name]
    x, g = inputs(name, limit=200000)
    for n in RAGGED:
        run_case(f"{name}/b{bits}", w.dtype, x[:n].copy(), g[:n].copy(),
                 label=f"{name} b{bits} n={n}")


EDGE_N = [1, 2, 31, 32, 33, 63, 64, 65, 511, 512, 513, 1023, 1024, 1025, 4095, (1 << 20) + 7]


def _synthetic_table(act, bits):
    import oracle as O
    key = {"gelu": "gelu3_f32_1m/b3", "silu": "silu2_f16_resnet_64x256x56x56/b2",
           "sigmoid": "sigmoid4_f32_odd_67108863/b4", "tanh": "tanh3_f32_odd_67108863/b3"}.get(act)
    spec = golden_table(key)[0] if key else None
    if spec is not None and spec["bits"] == bits:
        s = np.float32([float.fromhex(h) for h in spec["s"]])
        v = np.float32([float.fromhex(h) for h in spec["v"]])
    else:
        F = O.fit(OACT[act], bits, O.uniform(-8.0, 8.0), 400)
        s, v = F.s, F.v
    return s, v, P.Table.from_values(P.ACTS[act], bits, s, v)


def _run_synthetic(act, bits, dt, x_bits, g_bits, label, flags=0):
    s, v, table = _synthetic_table(act, bits)
    table = table.with_flags(flags)
    n = x_bits.size
    print(f"[edge] {label} act={act} dt={dt} bits={bits} n={n}", flush=True)
    y_ref, c_ref = O.fwd(OACT[act], ODT[dt], bits, s, x_bits, threads=THREADS)
    gin_ref = O.bwd(ODT[dt], bits, v, g_bits, c_ref, threads=THREADS)
    x = upload(x_bits, dt)
    y, codes = P.fwd(table, x)
    gin = P.bwd(table, upload(g_bits, dt), codes)
    torch.cuda.synchronize()
    check_exact(download_codes(codes)[:P.packed_words(n, bits)], c_ref, f"{label} codes")
    check_y(download(y, dt), y_ref, dt, f"{label} y")
    check_exact(download(gin, dt), gin_ref, f"{label} grad_in")


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_edge_sizes_gelu(dt, bits):
    rng = np.random.default_rng(100 + bits)
    for n in EDGE_N:
        x = O.round_array(ODT[dt], rng.normal(0, 2, n))
        g = O.round_array(ODT[dt], rng.normal(0, 1, n))
        _run_synthetic("gelu", bits, dt, x, g, f"edge n={n}")


MORE_ACTS = ["relu", "selu", "softplus"]


@pytest.mark.parametrize("act", ["silu", "sigmoid", "tanh"] + MORE_ACTS)
@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_edge_sizes_other_acts(act, dt):
    rng = np.random.default_rng(7)
    for bits in (1, 3, 4):
        for n in (1, 33, 513, 4097):
            x = O.round_array(ODT[dt], rng.uniform(-9, 9, n))
            g = O.round_array(ODT[dt], rng.normal(0, 1, n))
            _run_synthetic(act, bits, dt, x, g, f"{act} n={n}")


@pytest.mark.parametrize("act", MORE_ACTS)
@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_more_activations_several_waves(act, dt):
    # enough tiles for every wave of the grid to walk several, plus a ragged end
    rng = np.random.default_rng(21)
    n = (1 << 22) + 13
    x = O.round_array(ODT[dt], rng.uniform(-9, 9, n))
    g = O.round_array(ODT[dt], rng.normal(0, 1, n))
    _run_synthetic(act, 2, dt, x, g, f"{act} n={n}")


def _special_values(dt, s):
    big = {"f32": 3.0e38, "f16": 65000.0, "bf16": 3.0e38}[dt]
    tiny = {"f32": [1e-45, 1e-40, 1.17e-38], "f16": [6e-8, 3e-6, 6.1e-5],
            "bf16": [1e-40, 9.2e-41, 1.2e-38]}[dt]
    vals = [0.0, -0.0, np.inf, -np.inf, np.nan, -np.nan, big, -big]
    vals += tiny + [-t for t in tiny]
    # every boundary, and its neighbours in the storage type
    for b in s:
        bb = float(b)
        vals.append(bb)
        vals.append(bb * (1 + 2 ** -20) if bb else 1e-30)
        vals.append(bb * (1 - 2 ** -20) if bb else -1e-30)
    # the GELU / SiLU tail where outputs pass through the subnormals
    vals += list(np.linspace(-16.0, -12.0, 257)) + list(np.linspace(-110.0, -80.0, 97))
    vals += list(np.linspace(-20.0, 20.0, 401))
    return np.array(vals, np.float64)


@pytest.mark.parametrize("act", ["gelu", "silu", "sigmoid", "tanh"] + MORE_ACTS)
@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_special_values_and_boundaries(act, dt):
    bits = 3
    s, v, table = _synthetic_table(act, bits)
    xd = _special_values(dt, s)
    x = O.round_array(ODT[dt], xd)
    # boundary neighbours in the storage type itself
    if dt == "f32":
        sb = s.view(np.uint32)
        extra = np.concatenate([sb, sb + 1, sb - 1])
        extra = extra[(extra & 0x7F800000) != 0x7F800000]
        x = np.concatenate([x, extra.astype(np.uint32)])
    else:
        hb = O.round_array(ODT[dt], s.astype(np.float64))
        x = np.concatenate([x, hb, (hb + 1).astype(np.uint16), (hb - 1).astype(np.uint16)])
    x = np.tile(x, 3)            # several tiles' worth, with a ragged end
    rng = np.random.default_rng(11)
    g = O.round_array(ODT[dt], rng.normal(0, 1, x.size))
    _run_synthetic(act, bits, dt, x, g, f"special {act}")


# fp16 / bf16 forwards run the table kernel (LDS lookups per input bit
# pattern) from a size that depends on the activation, type and bit width, or
# whenever the table carries FLAG_TABLE_FWD; otherwise they evaluate f and the
# compares per element.  The cases above are mostly small; this one takes
# every activation, half type and bit width through the table kernel, over
# enough tiles for every wave of its persistent grid to walk several, with
# the special values and boundary neighbours in the mix.
@pytest.mark.parametrize("act", ["gelu", "silu", "sigmoid", "tanh"] + MORE_ACTS)
@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_table_kernel_every_activation(act, dt):
    rng = np.random.default_rng(17)
    for bits in (1, 2, 3, 4):
        n = (1 << 23) + 1234
        s, v, table = _synthetic_table(act, bits)
        special = O.round_array(ODT[dt], _special_values(dt, s))
        hb = O.round_array(ODT[dt], s.astype(np.float64))
        special = np.concatenate([special, hb, (hb + 1).astype(np.uint16), (hb - 1).astype(np.uint16)])
        x = O.round_array(ODT[dt], rng.uniform(-20, 20, n))
        pos = rng.choice(n, special.size * 64, replace=False)
        x[pos] = np.tile(special, 64)
        g = O.round_array(ODT[dt], rng.normal(0, 1, n))
        _run_synthetic(act, bits, dt, x, g, f"table kernel {act}", flags=P.FLAG_TABLE_FWD)


# Every one of the 65536 fp16 / bf16 input patterns (NaNs, infinities,
# subnormals and both zeros included) through both forward kernels, each on
# two shuffled copies of the pattern set plus a ragged end, so that every
# entry of the LDS output and code tables is read and checked.  All bit
# widths, and for the even f' of Sigmoid and Tanh also the |x| tables.
# Beyond the oracle's tolerance: the table kernel's output for a pattern is
# either the per-element kernel's (the blocks where it evaluates the same f)
# or the correctly rounded one (the blocks it fills by rule).
@pytest.mark.parametrize("act", ["gelu", "silu", "sigmoid", "tanh"] + MORE_ACTS)
@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_every_input_pattern(act, dt):
    rng = np.random.default_rng(41)
    pats = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    cases = [(b, False) for b in (1, 2, 3, 4)]
    if act in ("sigmoid", "tanh"):
        cases += [(b, True) for b in (1, 2, 3, 4)]
    for bits, sym in cases:
        if sym:
            F = O.fit(OACT[act], bits, O.uniform(-8.0, 8.0), 400, symmetric=True)
            s, v = F.s, F.v
            table = P.Table.from_values(P.ACTS[act], bits, s, v, flags=P.FLAG_SYMMETRIC)
        else:
            s, v, table = _synthetic_table(act, bits)
        kernels = {"per-element": P.FLAG_ELEMENT_FWD, "table": P.FLAG_TABLE_FWD}
        y_of_pattern, ref_of_pattern = {}, np.zeros(pats.size, np.uint16)
        for kernel, kflag in kernels.items():
            n = 2 * pats.size + 77
            reps = -(-n // pats.size)
            x_bits = np.concatenate([rng.permutation(pats) for _ in range(reps)])[:n]
            g_bits = O.round_array(ODT[dt], rng.normal(0, 1, n))
            label = f"every pattern {act} {dt} b{bits}{' sym' if sym else ''} {kernel} n={n}"
            print(f"[patterns] {label}", flush=True)
            y_ref, c_ref = O.fwd(OACT[act], ODT[dt], bits, s, x_bits, symmetric=sym,
                                 threads=THREADS)
            gin_ref = O.bwd(ODT[dt], bits, v, g_bits, c_ref, threads=THREADS)
            y, codes = P.fwd(table.with_flags(kflag), upload(x_bits, dt))
            gin = P.bwd(table, upload(g_bits, dt), codes)
            torch.cuda.synchronize()
            check_exact(download_codes(codes)[:P.packed_words(n, bits)], c_ref, f"{label} codes")
            check_y(download(y, dt), y_ref, dt, f"{label} y")
            check_exact(download(gin, dt), gin_ref, f"{label} grad_in")
            y_bits = download(y, dt)
            by_pattern = np.zeros(pats.size, np.uint16)
            by_pattern[x_bits] = y_bits
            check_exact(by_pattern[x_bits], y_bits, f"{label}: one y per pattern")
            y_of_pattern[kernel] = by_pattern
            ref_of_pattern[x_bits] = y_ref
        if "table" in y_of_pattern:
            # the table kernel fills most blocks of its output table by rule
            # (the correctly rounded value) and evaluates the kernel's f in
            # the rest (the per-element kernel's value)
            t, e = y_of_pattern["table"], y_of_pattern["per-element"]
            from parity import _isnan
            both_nan = _isnan(t, dt) & _isnan(ref_of_pattern, dt)
            odd = np.flatnonzero((t != e) & (t != ref_of_pattern) & ~both_nan)
            assert odd.size == 0, (f"every pattern {act} {dt} b{bits}: table y neither the "
                                   f"per-element y nor the oracle's at patterns {odd[:8]}")


# Symmetric tables (Fig. 3 caption: an even f' is fitted on [0, B] and the
# bins apply to |x|), fitted by the oracle for the Sigmoid and Tanh inputs.
SYM = sorted((k.split("/")[0], int(k.split("/")[1][1:])) for k in TABLES if k.endswith("/sym"))


@pytest.mark.parametrize("name,bits", SYM, ids=[f"{n}-b{b}" for n, b in SYM])
def test_symmetric_full_size(name, bits):
    w = WL.WORKLOADS[name]
    x, g = inputs(name)
    print(run_case(f"{name}/b{bits}/sym", w.dtype, x, g, label=f"{name} b{bits} sym full"),
          flush=True)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("name,bits", SYM, ids=[f"{n}-b{b}" for n, b in SYM])
def test_symmetric_half_types(name, bits, dt):
    w = WL.WORKLOADS[name]
    for n, flags in ((1, 0), (513, 0), (4097, 0), ((1 << 20) + 3, 0),
                     (4097, P.FLAG_TABLE_FWD), ((1 << 23) + 3, P.FLAG_TABLE_FWD)):
        x = WL.draw(w.x_dist, w.x_scale, n, dt, w.seed)
        g = WL.draw("normal", w.g_sigma, n, dt, w.seed + 1000)
        run_case(f"{name}/b{bits}/sym", dt, x, g, label=f"{name} b{bits} sym {dt} n={n} flags={flags}",
                 flags=flags)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("name,bits", SYM, ids=[f"{n}-b{b}" for n, b in SYM])
def test_symmetric_special_values(name, bits, dt):
    key = f"{name}/b{bits}/sym"
    spec, _ = golden_table(key)
    s = np.float32([float.fromhex(h) for h in spec["s"]])
    xd = _special_values(dt, s)
    x = O.round_array(ODT[dt], np.concatenate([xd, -xd]))
    # +-boundary and its storage neighbours: |x| lands on, just below and
    # just above every boundary from both sides of zero
    if dt == "f32":
        sb = s.view(np.uint32)
        nb = np.concatenate([sb, sb + 1, sb - 1])
        x = np.concatenate([x, nb, nb | np.uint32(0x80000000)])
    else:
        hb = O.round_array(ODT[dt], s.astype(np.float64))
        nb = np.concatenate([hb, (hb + 1).astype(np.uint16), (hb - 1).astype(np.uint16)])
        x = np.concatenate([x, nb, nb | np.uint16(0x8000)])
    x = np.tile(x, 3)
    rng = np.random.default_rng(13)
    g = O.round_array(ODT[dt], rng.normal(0, 1, x.size))
    run_case(key, dt, x, g, label=f"{key} special {dt}")


def _canary_buffers(n, dt, bits):
    pad_e, pad_w = 256, 64
    y_full = torch.empty(n + pad_e, dtype=torch.int32 if dt == "f32" else torch.int16,
                         device="cuda")
    y_full.fill_(0x5A5A)
    c_full = torch.empty(P.packed_words(n, bits) + pad_w, dtype=torch.int32, device="cuda")
    c_full.fill_(0x3C3C3C3C)
    return y_full, c_full


@pytest.mark.parametrize("dt,bits", [("bf16", 3), ("f32", 3), ("f16", 1), ("bf16", 4), ("f32", 2)])
def test_no_write_past_the_end(dt, bits):
    rng = np.random.default_rng(12)
    s, v, table = _synthetic_table("gelu", bits)
    for n in (1, 37, 511, 1025, 67109 * 3 + 1):
        x = upload(O.round_array(ODT[dt], rng.normal(0, 2, n)), dt)
        y_full, c_full = _canary_buffers(n, dt, bits)
        nw = P.packed_words(n, bits)
        from parity import torch_dtype
        y = y_full[:n].view(torch_dtype(dt))
        P.fwd(table, x, y=y, codes=c_full[:nw])
        gin_full, _ = _canary_buffers(n, dt, bits)
        P.bwd(table, x, c_full[:nw], grad_in=gin_full[:n].view(torch_dtype(dt)))
        torch.cuda.synchronize()
        assert bool((y_full[n:] == 0x5A5A).all()), f"y written past the end n={n}"
        assert bool((gin_full[n:] == 0x5A5A).all()), f"grad_in written past the end n={n}"
        assert bool((c_full[nw:] == 0x3C3C3C3C).all()), f"codes written past the end n={n}"


@pytest.mark.parametrize("dt,bits", [("bf16", 3), ("bf16", 4), ("f16", 3), ("f16", 4)])
def test_no_write_past_the_end_table_kernel(dt, bits):
    # the table forward (chosen by flag) with a partial last tile, against
    # the oracle and with canaries after every output
    rng = np.random.default_rng(14)
    s, v, table = _synthetic_table("gelu", bits)
    table = table.with_flags(P.FLAG_TABLE_FWD)
    from parity import torch_dtype
    base = (1 << 22)            # several rounds of the persistent grid
    for n in (1, 37, 511, base + 1, base + 37, base + 511):
        print(f"[canary-table] {dt} b{bits} n={n}", flush=True)
        xb = O.round_array(ODT[dt], rng.normal(0, 2, n))
        gb = O.round_array(ODT[dt], rng.normal(0, 1, n))
        y_ref, c_ref = O.fwd(O.GELU, ODT[dt], bits, s, xb, threads=THREADS)
        gin_ref = O.bwd(ODT[dt], bits, v, gb, c_ref, threads=THREADS)
        y_full, c_full = _canary_buffers(n, dt, bits)
        gin_full, _ = _canary_buffers(n, dt, bits)
        nw = P.packed_words(n, bits)
        P.fwd(table, upload(xb, dt), y=y_full[:n].view(torch_dtype(dt)), codes=c_full[:nw])
        P.bwd(table, upload(gb, dt), c_full[:nw], grad_in=gin_full[:n].view(torch_dtype(dt)))
        torch.cuda.synchronize()
        assert bool((y_full[n:] == 0x5A5A).all()), f"y written past the end n={n}"
        assert bool((gin_full[n:] == 0x5A5A).all()), f"grad_in written past the end n={n}"
        assert bool((c_full[nw:] == 0x3C3C3C3C).all()), f"codes written past the end n={n}"
        codes = c_full[:nw].cpu().numpy().view(np.uint32)
        assert np.array_equal(codes, c_ref), f"codes n={n}"
        gin = gin_full[:n].cpu().numpy().view(np.uint16)
        assert np.array_equal(gin, gin_ref), f"grad_in n={n}"
        check_y(y_full[:n].cpu().numpy().view(np.uint16), y_ref, dt, f"y n={n}")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_in_place(dt):
    rng = np.random.default_rng(13)
    n = 100000 + 3
    s, v, table = _synthetic_table("gelu", 3)
    xb = O.round_array(ODT[dt], rng.normal(0, 2, n))
    gb = O.round_array(ODT[dt], rng.normal(0, 1, n))
    y_ref, c_ref = O.fwd(O.GELU, ODT[dt], 3, s, xb, threads=THREADS)
    gin_ref = O.bwd(ODT[dt], 3, v, gb, c_ref, threads=THREADS)
    x = upload(xb, dt)
    _, codes = P.fwd(table, x, y=x)                 # y == x
    g = upload(gb, dt)
    P.bwd(table, g, codes, grad_in=g)               # grad_in == grad_out
    torch.cuda.synchronize()
    check_y(download(x, dt), y_ref, dt, "in-place y")
    check_exact(download_codes(codes)[:c_ref.size], c_ref, "in-place codes")
    check_exact(download(g, dt), gin_ref, "in-place grad_in")


def test_side_stream():
    rng = np.random.default_rng(14)
    n = 300001
    s, v, table = _synthetic_table("gelu", 3)
    xb = O.round_array(O.BF16, rng.normal(0, 2, n))
    y_ref, c_ref = O.fwd(O.GELU, O.BF16, 3, s, xb, threads=THREADS)
    x = upload(xb, "bf16")
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        y, codes = P.fwd(table, x)
    torch.cuda.current_stream().wait_stream(st)
    torch.cuda.synchronize()
    check_exact(download_codes(codes)[:c_ref.size], c_ref, "stream codes")
    check_y(download(y, "bf16"), y_ref, "bf16", "stream y")


def test_concurrent_streams():
    # The library keeps no device state: calls on three streams that run at
    # the same time (the table forward, the per-element forward and the fp32
    # path, with different tables, activations and bit widths, each followed
    # by its backward, three rounds) give what each gives alone.
    rng = np.random.default_rng(15)
    cases = [("gelu", 3, "bf16", (1 << 22) + 1234, P.FLAG_TABLE_FWD),
             ("silu", 2, "f16", 300001, P.FLAG_ELEMENT_FWD),
             ("tanh", 3, "f32", 500003, 0)]
    runs = []
    for act, bits, dt, n, flags in cases:
        s, v, table = _synthetic_table(act, bits)
        table = table.with_flags(flags)
        xb = O.round_array(ODT[dt], rng.normal(0, 2, n))
        gb = O.round_array(ODT[dt], rng.normal(0, 1, n))
        y_ref, c_ref = O.fwd(OACT[act], ODT[dt], bits, s, xb, threads=THREADS)
        gin_ref = O.bwd(ODT[dt], bits, v, gb, c_ref, threads=THREADS)
        runs.append(dict(table=table, dt=dt, x=upload(xb, dt), g=upload(gb, dt), y_ref=y_ref,
                         c_ref=c_ref, gin_ref=gin_ref, stream=torch.cuda.Stream(), out=[]))
    print(f"[streams] {[(c[0], c[2], c[3]) for c in cases]}", flush=True)
    main = torch.cuda.current_stream()
    for r in runs:
        r["stream"].wait_stream(main)
    for _ in range(3):
        for r in runs:                     # interleaved launches on the three streams
            with torch.cuda.stream(r["stream"]):
                y, codes = P.fwd(r["table"], r["x"])
                gin = P.bwd(r["table"], r["g"], codes)
                r["out"].append((y, codes, gin))
    for r in runs:
        main.wait_stream(r["stream"])
    torch.cuda.synchronize()
    for r in runs:
        for k, (y, codes, gin) in enumerate(r["out"]):
            what = f"{r['dt']} round {k}"
            check_exact(download_codes(codes)[:r["c_ref"].size], r["c_ref"], f"{what} codes")
            check_y(download(y, r["dt"]), r["y_ref"], r["dt"], f"{what} y")
            check_exact(download(gin, r["dt"]), r["gin_ref"], f"{what} grad_in")


def _codes_at(codes_dev, idx, bits):
    """Codes of elements idx from the packed device buffer (fetching only
    the words they touch), by the stream layout: bit t of code i is stream
    bit bits*i + t, in word p / 32 at bit p % 32."""
    first = (idx * bits) // 32
    words = torch.stack([codes_dev[torch.from_numpy(first).cuda()],
                         codes_dev[torch.from_numpy(np.minimum(first + 1, codes_dev.numel() - 1)).cuda()]])
    w = words.cpu().numpy().view(np.uint32).astype(np.uint64)
    both = w[0] | (w[1] << np.uint64(32))
    return ((both >> ((idx * bits) % 32).astype(np.uint64)) & np.uint64((1 << bits) - 1)).astype(np.int64)


@pytest.mark.slow
def test_beyond_two_to_the_31_elements():
    # 64-bit element, tile and word indexing: a bf16 tensor of 2^31 + 12345
    # elements (about 18 GB resident with outputs and gradients), checked at
    # sampled positions around 2^31, at the end and at random, against the
    # oracle evaluated on those elements alone
    n = (1 << 31) + 12345
    key = "gelu_bf16_lm_ffn_16x2048x8192/b3"
    spec, table = golden_table(key)
    bits = spec["bits"]
    s = np.float32([float.fromhex(h) for h in spec["s"]])
    v = np.float32([float.fromhex(h) for h in spec["v"]])
    print(f"[big] n={n}", flush=True)
    gen = torch.Generator(device="cuda").manual_seed(41)
    x = (torch.randn(n, device="cuda", generator=gen) * 3).to(torch.bfloat16)
    g = torch.randn(n, device="cuda", generator=gen).to(torch.bfloat16)
    y, codes = P.fwd(table, x)
    gin = P.bwd(table, g, codes)
    torch.cuda.synchronize()
    rng = np.random.default_rng(42)
    idx = np.unique(np.concatenate([
        np.arange((1 << 31) - 3000, (1 << 31) + 3000), np.arange(n - 5000, n),
        rng.integers(0, n, 200000)]))
    it = torch.from_numpy(idx).cuda()
    xs = x[it].view(torch.int16).cpu().numpy().view(np.uint16)
    gs = g[it].view(torch.int16).cpu().numpy().view(np.uint16)
    ys = y[it].view(torch.int16).cpu().numpy().view(np.uint16)
    gis = gin[it].view(torch.int16).cpu().numpy().view(np.uint16)
    y_ref, c_packed = O.fwd(O.GELU, O.BF16, bits, s, xs)
    idx_ref = O.unpack(c_packed, xs.size, bits)
    check_y(ys, y_ref, "bf16", "y sampled")
    check_exact(_codes_at(codes, idx, bits), idx_ref.astype(np.int64), "codes sampled")
    gin_ref = O.bwd(O.BF16, bits, v, gs, c_packed)
    check_exact(gis, gin_ref, "grad_in sampled")
    del x, g, y, codes, gin
    torch.cuda.empty_cache()


@pytest.mark.parametrize("kernel", ["per-element", "table"])
def test_graph_capture_replays(kernel):
    # forward + backward captured into a graph after one eager call,
    # replayed several times with eager work and synchronisation in
    # between; every replay must equal the eager result bit for bit.  Both
    # fp16 / bf16 forward kernels.  (tests/test_gpu_capture_first.py makes a
    # process's first call inside a capture.)
    rng = np.random.default_rng(31)
    n = 3 * 65536 + 77
    spec, table = golden_table("gelu_bf16_lm_ffn_16x2048x8192/b3")
    table = table.with_flags(P.FLAG_ELEMENT_FWD if kernel == "per-element" else P.FLAG_TABLE_FWD)
    x = upload(O.round_array(O.BF16, rng.normal(0, 2, n)), "bf16")
    g = upload(O.round_array(O.BF16, rng.normal(0, 1, n)), "bf16")
    y, codes = P.fwd(table, x)
    gin = P.bwd(table, g, codes)
    torch.cuda.synchronize()
    y_ref, c_ref, gin_ref = y.clone(), codes.clone(), gin.clone()
    y2, c2, gin2 = torch.empty_like(y), torch.empty_like(codes), torch.empty_like(gin)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            P.fwd(table, x, y=y2, codes=c2)
            P.bwd(table, g, c2, grad_in=gin2)
    torch.cuda.current_stream().wait_stream(side)
    for rep in range(4):
        y2.fill_(0)
        c2.fill_(-1)
        gin2.fill_(0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y2.view(torch.int16), y_ref.view(torch.int16)), rep
        assert torch.equal(c2, c_ref), rep
        assert torch.equal(gin2.view(torch.int16), gin_ref.view(torch.int16)), rep


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_empty_tensors(dt):
    # n = 0 launches nothing and returns empty results
    from parity import torch_dtype
    s, v, table = _synthetic_table("gelu", 3)
    x = torch.empty(0, dtype=torch_dtype(dt), device="cuda")
    y, codes = P.fwd(table, x)
    gin = P.bwd(table, x, codes)
    torch.cuda.synchronize()
    assert y.numel() == 0 and gin.numel() == 0 and P.packed_words(0, 3) == 0


def test_misaligned_pointer_is_rejected():
    s, v, table = _synthetic_table("gelu", 3)
    x = torch.zeros(1000, dtype=torch.bfloat16, device="cuda")
    y = torch.zeros(1000, dtype=torch.bfloat16, device="cuda")
    c = torch.zeros(200, dtype=torch.int32, device="cuda")
    rc = P.fwd_raw(table, P.BF16, x.data_ptr() + 2, y.data_ptr(), c.data_ptr(), 10,
                   torch.cuda.current_stream().cuda_stream)
    assert rc == -3


def test_autograd_wrapper():
    rng = np.random.default_rng(15)
    n = 8 * 512 * 3 + 5
    s, v, table = _synthetic_table("gelu", 3)
    xb = O.round_array(O.BF16, rng.normal(0, 2, n))
    gb = O.round_array(O.BF16, rng.normal(0, 1, n))
    x = upload(xb, "bf16").requires_grad_(True)
    y = P.FewBitActivation.apply(x, table)
    y.backward(upload(gb, "bf16"))
    torch.cuda.synchronize()
    y_ref, c_ref = O.fwd(O.GELU, O.BF16, 3, s, xb, threads=THREADS)
    gin_ref = O.bwd(O.BF16, 3, v, gb, c_ref, threads=THREADS)
    check_y(download(y.detach(), "bf16"), y_ref, "bf16", "autograd y")
    check_exact(download(x.grad, "bf16"), gin_ref, "autograd grad")


def test_module_fits_its_own_table():
    m = P.FewBitAct("gelu", 3)
    assert len(m.table.s) == 7 and m.table.loss > 0
    x = torch.randn(4096 + 3, device="cuda", dtype=torch.float32, requires_grad=True)
    y = m(x)
    y.sum().backward()
    torch.cuda.synchronize()
    codes = O.fwd(O.GELU, O.F32, 3, np.float32(m.table.s),
                  x.detach().cpu().numpy().view(np.uint32), want_idx=True)[2]
    ref = np.float32(m.table.v)[codes]
    assert np.array_equal(x.grad.cpu().numpy(), ref)
