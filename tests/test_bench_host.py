"""Host-side logic of bench.py (no GPU): the kernel-source hash that ties
the committed HBM-traffic figures to the kernels they were measured on."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_code_tokens_ignore_comments_and_layout():
    a = "int f(int x) {\n  return x + 1;  // add one\n}\n/* block\n comment */\n"
    b = "int f(int x) { return x + 1; }"
    assert bench._code_tokens(a) == bench._code_tokens(b)


def test_code_tokens_keep_string_and_char_literals():
    src = 'const char* s = "// not a comment /* nor this */"; char c = \'/\'; // gone'
    assert bench._code_tokens(src) == 'const char* s = "// not a comment /* nor this */"; char c = \'/\';'


def test_code_change_changes_tokens():
    assert bench._code_tokens("a = b + 1;") != bench._code_tokens("a = b + 2;")


def test_committed_traffic_figures():
    # profiles/traffic.json holds rocprofv3 counter figures; bench.py reports
    # them only while they were taken on the current kernel code (else null)
    import json
    import pytest
    with open(os.path.join(ROOT, "profiles", "traffic.json")) as fh:
        rec = json.load(fh)
    if rec["kernel_source_hash"] != bench.kernel_source_hash():
        pytest.skip("kernel code changed since the counters were taken")
    assert bench.measured_traffic("gelu_bf16_lm_ffn_16x2048x8192", 3, "fwd") is not None
    for key, v in rec["launches"].items():
        assert 0.99 < v["hbm_bytes"] / v["algorithmic_bytes"] < 1.1, key


def test_ceiling_kernels_move_the_passes_bytes():
    # the streaming reference kernels move exactly the algorithmic bytes of
    # a pass per 512-element tile
    import ceiling as CL
    for dtype, s in (("bf16", 2), ("f16", 2), ("f32", 4)):
        for bits in (1, 2, 3, 4):
            per_tile = bench.algorithmic_bytes(512, dtype, bits)
            assert CL.tile_bytes("fwd", s, bits) == per_tile
            assert CL.tile_bytes("bwd", s, bits) == per_tile
        assert CL.tile_bytes("copy", s, 3) == 2 * 512 * s


def test_ceiling_rejects_bad_arguments_before_launching():
    import ceiling as CL
    f = CL._lib.ceiling_stream
    assert f(0, 64, 2, 3, None, None, None, 0, None) == 0          # nothing to move
    assert f(3, 64, 2, 3, 16, 16, 16, 1, None) == -1               # kind
    assert f(1, 128, 2, 3, 16, 16, 16, 1, None) == -1              # launch shape
    assert f(1, 513, 2, 3, 16, 16, 16, 1, None) == -1
    assert f(1, 512, 2, 3, None, None, None, 0, None) == 0         # persistent, nothing to move
    assert f(1, 64, 8, 3, 16, 16, 16, 1, None) == -1               # element size
    assert f(1, 64, 2, 5, 16, 16, 16, 1, None) == -1               # bits
    assert f(1, 64, 2, 3, 16, 16, None, 1, None) == -1             # codes missing
    assert f(0, 64, 2, 3, None, 16, None, 1, None) == -1           # source missing


def test_stats_record():
    rec = bench.stats_record([2.0, 1.0, 3.0, 10.0], bytes_pass=8e9)
    assert rec["ms"] == 4.0 and rec["median_ms"] == 2.5 and rec["min_ms"] == 1.0
    assert abs(rec["frac_peak"] - 8e9 / 4e-3 / 1e9 / bench.HBM_PEAK_GBPS) < 1e-4


def test_host_cpu():
    h = bench.host_cpu()
    assert h["cpus"] >= 1


def test_kernel_keys_of_rocprof_names():
    k = bench._kernel_key
    assert k("void (anonymous namespace)::stream_kernel<1, 2, 64, false>(unsigned char const*, "
             "unsigned char*, unsigned int*, long, int, unsigned int)") == "ceiling_fwd<64>"
    assert k("void (anonymous namespace)::stream_kernel<0, 4, 256, false>(...)") == "ceiling_copy<256>"
    assert k("void (anonymous namespace)::stream_kernel<2, 2, 64, true>(...)") == "ceiling_bwd<64,paired>"
    assert k("void (anonymous namespace)::persist_kernel<1, 2>(...)") == "ceiling_fwd<persistent>"
    assert k("void (anonymous namespace)::bwd_kernel<2, 3>(unsigned short const*, ...)") == \
        "bwd_kernel<bf16,3>"
    assert k("void (anonymous namespace)::fwd16_kernel<2, 3, 0>(...)") == \
        "fwd16_kernel<bf16,3,gelu>"


def test_summarize_sq_averages_per_dispatch(tmp_path, capsys):
    # two dispatches of a library kernel (one counter split over two rows,
    # as rocprofv3 writes per-block values) and one of a streaming kernel
    d = tmp_path / "pmc"
    d.mkdir()
    rows = [
        (1, "(anonymous namespace)::bwd_kernel<2, 3>(...)", "SQ_INSTS_VALU", 100.0e6),
        (1, "(anonymous namespace)::bwd_kernel<2, 3>(...)", "SQ_INSTS_VALU", 60.0e6),
        (1, "(anonymous namespace)::bwd_kernel<2, 3>(...)", "SQ_WAVE_CYCLES", 400.0),
        (1, "(anonymous namespace)::bwd_kernel<2, 3>(...)", "SQ_WAIT_ANY", 100.0),
        (2, "(anonymous namespace)::bwd_kernel<2, 3>(...)", "SQ_INSTS_VALU", 240.0e6),
        (2, "(anonymous namespace)::bwd_kernel<2, 3>(...)", "SQ_WAVE_CYCLES", 400.0),
        (2, "(anonymous namespace)::bwd_kernel<2, 3>(...)", "SQ_WAIT_ANY", 300.0),
        (3, "void (anonymous namespace)::stream_kernel<0, 2, 64, false>(...)", "SQ_INSTS_VALU", 7.0),
    ]
    with open(d / "run_counter_collection.csv", "w") as fh:
        fh.write('"Dispatch_Id","Kernel_Name","Counter_Name","Counter_Value"\n')
        for disp, name, c, v in rows:
            fh.write(f'{disp},"{name}","{c}",{v}\n')
    import workloads as WL
    w = WL.WORKLOADS["gelu3_bf16_bert_ffn_8x512x3072"]
    bench.summarize_sq([str(d)], w.name)
    out = capsys.readouterr().out
    # SQ_INSTS_VALU: dispatch 1 = 160e6, dispatch 2 = 240e6 -> 200e6 per dispatch
    assert f"VALU instructions per element {200e6 * 64 / w.n:.2f}" in out
    assert f"{200e6 * 64 / w.n:.2f}" != f"{240e6 * 64 / w.n:.2f}"
    # waiting share: (100/400 + 300/400) / 2 per dispatch averages -> 200 / 400
    assert "waiting share 0.50" in out
    assert "ceiling_copy<64>" in out


def test_forced_forward_kernel_choice():
    # --fwd-kernel forces the 16-bit forward kernel through the table flags,
    # and the reported kernel name follows the forced choice
    import paper_2202_00441_amd as P
    import workloads as WL
    w = WL.WORKLOADS["gelu_bf16_lm_ffn_16x2048x8192"]
    assert bench.fwd_kernel_flag(P, "auto") == 0
    assert bench.fwd_kernel_flag(P, "table") == P.FLAG_TABLE_FWD
    assert bench.fwd_kernel_flag(P, "element") == P.FLAG_ELEMENT_FWD
    assert bench.forced_min(P, w, 3, "auto") == P.fwd16_table_min("gelu", 3, "bf16")
    for choice, kernel in (("table", "fwd16_kernel"), ("element", "fwd16v_kernel")):
        tm = bench.forced_min(P, w, 3, choice)
        assert bench.kernel_name("fwd", "bf16", 3, "gelu", 1, tm).startswith(kernel + "<")
        assert bench.kernel_name("fwd", "bf16", 3, "gelu", w.n, tm).startswith(kernel + "<")
