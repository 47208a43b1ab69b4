"""CPU: the algorithmic byte and FLOP counts behind the benchmark's rooflines,
against values the model shapes and Table 1 fix on their own (bf16 K/V bytes
per token; the core's bf16 weight bytes; a mid-decode batch worked by hand)."""
import numpy as np

import bench
import cdbgen


def test_kv_bytes_per_token_and_layer_match_table_1():
    # Table 1, single slot, bf16: Ouro 192 KiB per token over its 24 layers,
    # Huginn 165 KiB over its 8 physical layers (2 prelude, 4 core, 2 coda)
    o, h = cdbgen.OURO, cdbgen.HUGINN
    assert bench.attention_bytes(o, [0]) - o.d * 6 == 192 * 1024 // o.n_core
    assert bench.attention_bytes(h, [0]) - h.d * 6 == 165 * 1024 // (h.n_prelude + h.n_core + h.n_coda)


def test_attention_bytes_count_every_visible_position():
    o = cdbgen.OURO
    assert bench.attention_bytes(o, np.array([0, 9, 640])) == (1 + 10 + 641) * 8192 + 3 * o.d * (4 + 2)


def test_step_bytes_and_flops_of_a_mid_decode_batch():
    o = cdbgen.OURO
    per_layer = 4 * o.d * o.d + 3 * o.d * o.d_ff  # q, k, v, o and gate, up, down, no biases
    w_core = o.n_core * per_layer * 2
    assert w_core == 2_466_250_752
    rows = {"pos": np.full(64, 640), "c": np.zeros(64, np.int64), "depth": np.full(64, 4)}
    kv_tok = 192 * 1024
    want = w_core + o.d * 2 + 64 * 641 * kv_tok + 64 * kv_tok + 64 * o.d * 4 * 2
    assert bench.step_bytes(o, rows) == want
    assert abs(want / 1e9 - 10.545) < 1e-3  # 1.32 ms at 8 TB/s
    assert bench.step_flops(o, rows) == 2 * 64 * o.n_core * per_layer + 4 * o.n_core * o.d * 64 * 641


def test_copy_on_exit_bytes_count_each_deeper_plane_read_and_written():
    o = cdbgen.OURO
    stay = {"pos": np.array([100]), "c": np.array([0]), "depth": np.array([2])}
    leave = {"pos": np.array([100]), "c": np.array([0]), "depth": np.array([1])}  # planes 2..4 take its entry
    assert bench.step_bytes(o, leave) - bench.step_bytes(o, stay) == (o.r_max - 1) * 2 * 192 * 1024


def test_huginn_core_weights_include_the_adapter():
    h = cdbgen.HUGINN
    per_layer = 4 * h.d * h.d + 3 * h.d * h.d_ff
    assert cdbgen.param_counts(h)["core"] * 2 == (h.n_core * per_layer + h.d * 2 * h.d) * 2 == 3_274_444_800


def test_idle_segments_of_a_synthetic_kernel_trace(tmp_path):
    # two decodes separated by 1 s of silence; the first has two overlapping
    # kernels (busy is their union), a 10 us gap and a nested kernel
    us = 1000
    kernels = [(0, 40 * us), (30 * us, 60 * us), (70 * us, 100 * us), (80 * us, 90 * us),
               (1_000_100 * us, 1_000_110 * us), (1_000_130 * us, 1_000_150 * us)]
    p = tmp_path / "run_kernel_trace.csv"
    p.write_text("Kernel_Name,Start_Timestamp,End_Timestamp\n" +
                 "".join(f"k{i},{a},{b}\n" for i, (a, b) in enumerate(kernels)))
    segs = bench.idle_segments(str(p))
    assert len(segs) == 2
    assert segs[0]["kernels"] == 4 and segs[0]["span_ms"] == 0.1 and segs[0]["busy_ms"] == 0.09
    assert segs[0]["idle_pct"] == 10.0 and segs[0]["largest_gaps_us"] == [10.0]
    assert segs[1]["kernels"] == 2 and segs[1]["span_ms"] == 0.05 and segs[1]["busy_ms"] == 0.03
    assert segs[1]["idle_pct"] == 40.0 and segs[1]["largest_gaps_us"] == [20.0]
