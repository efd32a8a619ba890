"""Host logic of bench.py: the algorithmic work it divides by, the grouping of
profiler dispatches into engine launches, the stale-counter rule and the
shader-clock readout.  CPU only."""

import csv

import pytest

import bench
import synth


def _allowed_pairs_brute(b):
    """Visible (query, key) pairs by enumeration: causal j <= i; prefix-LM
    j <= max(i, P - 1) (Section 3.3 batches; GLM's bidirectional context)."""
    n = 0
    for s in range(b.num_seqs):
        L = int(b.seqlens[s])
        P = int(b.prefix_len[s]) if b.mask == "prefix" else 0
        for i in range(L):
            n += sum(1 for j in range(L) if j <= max(i, P - 1))
    return n


@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_attention_pairs_match_enumeration(mask):
    b = synth.make_batch(3, 2, (5, 40), mask=mask, seed=4)
    w = synth.WORKLOADS["tiny_2blk_fp32"]
    fl = bench.algorithmic_flops(w, b)
    assert fl["pairs"] == _allowed_pairs_brute(b)


def test_gemm_flops_are_the_sum_of_the_block_products():
    """2 m n k per product: forward QKV (T x 3H x H), out-projection (T x H x
    H), FFN1 (T x F x H), FFN2 (T x H x F); the backward repeats each as an
    input-gradient and a weight-gradient product (input gradients only when
    the weights are frozen)."""
    b = synth.make_batch(2, 2, (9, 30), seed=1)
    for name in ("tiny_2blk_fp32", "chatglm6b_26blk_ragged_32x1_recompute",
                 "chatglm6b_26blk_ptuning128_ragged_32x1_recompute"):
        w = synth.WORKLOADS[name]
        H, F, T = w.shape.hidden, w.shape.ffn_hidden, b.total_tokens
        fwd = 2 * T * (3 * H * H + H * H + F * H + H * F)
        per_block = fwd * (1 + (1 if w.frozen else 2) if w.backward else 1)
        assert bench.algorithmic_flops(w, b)["gemm"] == pytest.approx(per_block * bench.total_layers(w), rel=1e-12)


def test_gemm_flops_follow_the_ffn_width():
    b = synth.make_batch(1, 1, (16, 16), seed=0)
    w = synth.WORKLOADS["tiny_2blk_fp32"]
    import dataclasses
    w2 = dataclasses.replace(w, shape=dataclasses.replace(w.shape, ffn_hidden=3 * w.shape.hidden))
    H, T = w.shape.hidden, b.total_tokens
    d = bench.algorithmic_flops(w, b)["gemm"] - bench.algorithmic_flops(w2, b)["gemm"]
    # one H-wide slice of FFN width less: 4 H^2 per token forward, x3 with the backward
    assert d == pytest.approx(3 * 4 * H * H * T * bench.total_layers(w), rel=1e-12)


def _disp(*names):
    return [("1", i, n, 1.0) for i, n in enumerate(names)]


GEMM_RES = "flglm::(anonymous namespace)::gemm_bf16_kernel<true, true, 2, 16>(G2Args)"
GEMM_TN = "flglm::(anonymous namespace)::gemm_bf16_kernel<false, false, 5, 4>(G2Args)"
LN = "void flglm::ln_fwd_kernel<bf16, 8>(...)"
DELTA, DKDV, DQ = "attn_delta_kernel<bf16, 128>", "flglm::(anonymous namespace)::dkdv_kernel<128>", \
    "flglm::(anonymous namespace)::dq_kernel<128>"


def test_fixup_dispatch_joins_its_launch():
    """A GEMM whose last round is split runs the same kernel twice in a row
    (main, then fix-up): one engine launch; the same GEMM again after another
    kernel is a new launch."""
    r = bench._class_launches(_disp(GEMM_RES, GEMM_RES, LN, GEMM_RES, LN, GEMM_TN, GEMM_TN, GEMM_TN))
    assert r["gemm_nt_bias_res"] == [2, 3.0]
    assert r["gemm_tn_acc"] == [1, 3.0]   # a reduction cut into three pieces
    assert r["layernorm_fwd"] == [2, 2.0]


def test_multi_kernel_class_counts_once():
    r = bench._class_launches(_disp(DELTA, DKDV, DQ, LN, DELTA, DKDV, DQ))
    assert r["attn_bwd"] == [2, 6.0]


PART, FIN = "void flglm::colsum_partial_kernel<bf16, 0>(...)", "flglm::colsum_finish_kernel(...)"
GELU_BWD = "flglm::(anonymous namespace)::gemm_bf16_kernel<true, false, 4, 8>(G2Args)"


def test_finish_after_a_gemm_is_a_column_sum_launch():
    """partial + finish, partial + finish + finish (LayerNorm gain and shift)
    and a finish of sums a GEMM epilogue formed: three column-sum launches."""
    r = bench._class_launches(_disp(PART, FIN, LN, PART, FIN, FIN, GELU_BWD, FIN))
    assert r["colsum"] == [3, 6.0]
    assert r["gemm_nn_gelu_bwd"] == [1, 1.0]


def test_queues_are_grouped_separately():
    d = [("1", 0, GEMM_RES, 1.0), ("2", 1, GEMM_RES, 1.0)]
    assert bench._class_launches(d)["gemm_nt_bias_res"] == [2, 2.0]


def test_summarize_trace_on_a_synthetic_run(tmp_path):
    rows = [(GEMM_RES, 0, 100), (GEMM_RES, 100, 130), (LN, 130, 140), (GEMM_RES, 140, 240)]
    with open(tmp_path / "run_kernel_trace.csv", "w", newline="") as fh:
        wr = csv.writer(fh)
        wr.writerow(["Queue_Id", "Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        for i, (n, a, e) in enumerate(rows):
            wr.writerow(["1", i, n, a * 1000, e * 1000])
    with open(tmp_path / "run_kernel_stats.csv", "w", newline="") as fh:
        wr = csv.writer(fh)
        wr.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage"])
        wr.writerow([GEMM_RES, 3, 230000, 76666.7, 95.8])
        wr.writerow([LN, 1, 10000, 10000, 4.2])
    out = bench.summarize_trace(str(tmp_path))
    line = [l for l in out.splitlines() if l.startswith("gemm_nt_bias_res")][0].split()
    assert int(line[1]) == 2 and float(line[2]) == pytest.approx(115.0)   # (130 + 100) us over 2 launches


def test_committed_traffic_goes_stale_with_the_sources(tmp_path, monkeypatch):
    h = bench.class_source_hash("gemm_tn_acc")
    f = tmp_path / "server_stack_kernels_w_hbm_traffic.txt"
    f.write_text(f"class gemm_tn_acc launches 4 hbm_bytes_per_launch 1234 src {h}\n"
                 f"class attn_fwd launches 4 hbm_bytes_per_launch 99 src 0000000000000000\n")
    monkeypatch.setattr(bench, "traffic_file", lambda w: str(f))
    assert bench.committed_traffic("gemm_tn_acc", "w") == 1234
    assert bench.committed_traffic("attn_fwd", "w") is None      # hash of other sources
    assert bench.committed_traffic("layernorm_fwd", "w") is None  # not measured


def test_source_hash_ignores_comments_but_not_code(tmp_path, monkeypatch):
    base = ('#pragma once\n// a kernel\n__global__ void k(float* p) { /* one */ p[0] = 1.0f; }\n'
            'asm volatile("s_nop 0 // kept: inside a string" ::: "memory");\n')
    variants = {
        "same": base.replace("// a kernel", "// the kernel, reworded").replace("/* one */", "/* two\n lines */"),
        "code": base.replace("1.0f", "2.0f"),
        "asm": base.replace("s_nop 0 //", "s_nop 1 //"),
    }
    monkeypatch.setattr(bench, "CSRC", str(tmp_path))
    monkeypatch.setattr(bench, "CLASS_SOURCES", {"": ("k.hip",)})

    def h(text):
        (tmp_path / "k.hip").write_text(text)
        return bench.class_source_hash("anything")
    h0 = h(base)
    assert h(variants["same"]) == h0
    assert h(variants["code"]) != h0
    assert h(variants["asm"]) != h0     # a string literal is code, even with // inside


@pytest.mark.parametrize("text,mhz", [("0: 500Mhz\n1: 1938Mhz *\n2: 2400Mhz\n", 1938.0),
                                      ("S: 112Mhz *\n0: 500Mhz\n1: 2400Mhz\n", 112.0),
                                      ("0: 500Mhz\n1: 2400Mhz\n", None)])
def test_clock_readout(tmp_path, text, mhz):
    f = tmp_path / "pp_dpm_sclk"
    f.write_text(text)
    assert bench.ClockSampler(str(f))._read() == mhz


def test_clock_sampler_mean_and_absent_source(tmp_path):
    import time
    f = tmp_path / "pp_dpm_sclk"
    f.write_text("0: 500Mhz\n1: 2000Mhz *\n")
    c = bench.ClockSampler(str(f)).start()
    time.sleep(0.08)
    assert c.stop() == 2000.0 and len(c.samples) >= 2
    assert bench.ClockSampler(None).start().stop() is None


def test_summarize_mfma_on_a_synthetic_run(tmp_path):
    rows = [(GEMM_RES, "MfmaFlopsBF16", 1000.0, 0, 100), (GEMM_RES, "MfmaUtil", 50.0, 0, 100),
            (GEMM_RES, "MfmaFlopsBF16", 24.0, 100, 110), (GEMM_RES, "MfmaUtil", 10.0, 100, 110),
            (LN, "MfmaFlopsBF16", 0.0, 110, 120), (LN, "MfmaUtil", 0.0, 110, 120)]
    with open(tmp_path / "run_counter_collection.csv", "w", newline="") as fh:
        wr = csv.writer(fh)
        wr.writerow(["Queue_Id", "Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
                     "End_Timestamp"])
        for i, (n, c, v, a, e) in enumerate(rows):
            wr.writerow(["1", i // 2, n, c, v, a, e])
    bj = tmp_path / "b.json"
    bj.write_text('{"kernels": {"gemm_nt_bias_res": {"tflops": 1e-6, "avg_launch_us": 1024.0}}}\n')
    out = bench.summarize_mfma(str(tmp_path), str(bj))
    line = [l for l in out.splitlines() if l.startswith("gemm_nt_bias_res")][0].split()
    # main + fix-up dispatch: one launch of 1024 flops; busy share weighted by duration
    assert int(line[1]) == 1 and float(line[2]) == 1024.0 and float(line[4]) == pytest.approx(1.0)
    assert float(line[5]) == pytest.approx((50.0 * 100 + 10.0 * 10) / 110, abs=0.05)
    assert not any(l.startswith("layernorm_fwd") for l in out.splitlines())


def test_spread_order_covers_the_length_distribution():
    """Every sequence once; the first picks are the median, then the
    quartiles, so a budget-limited prefix of the order samples the whole
    length distribution rather than its short end."""
    lens = [5, 1, 9, 3, 7, 2, 8, 4]
    o = bench.spread_order(lens)
    assert sorted(o) == list(range(len(lens)))
    assert [lens[i] for i in o[:3]] == [5, 3, 8]
    b = synth.WORKLOADS["chatglm6b_26blk_ragged_32x1_recompute"].batch()
    first = [int(b.seqlens[i]) for i in bench.spread_order(b.seqlens)[:3]]
    assert min(first) > int(b.seqlens.min()) and max(first) < int(b.seqlens.max())
    assert sorted(first)[1] == sorted(b.seqlens.tolist())[len(b.seqlens) // 2]


def test_cpu_baseline_is_the_float32_oracle():
    w = synth.WORKLOADS["tiny_2blk_fp32"]
    r = bench.cpu_baseline(w, w.batch(), budget_s=0.01)
    assert r["kind"] == "oracle" and r["value"] > 0 and r["cores"] >= 1
    assert "float32" in r["sample"] and "spread over" in r["sample"]
