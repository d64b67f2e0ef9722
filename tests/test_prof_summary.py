"""The counter summaries behind profiles/ (prof_summary), on small synthetic
rocprofv3 counter files: per-dispatch means per kernel, the wave-cycle
fractions and the MFMA rate.  No GPU."""
import csv

from paper_2605_30876_amd import prof_summary as P

K1 = "void dmoe::(anonymous namespace)::ffn_tile_bf16_kernel<true, 2>(dmoe::(anonymous namespace)::FfnParams, int)"
K2 = "void dmoe::(anonymous namespace)::ffn_tile_bf16_kernel<false, 2>(dmoe::(anonymous namespace)::FfnParams, int)"


def _csv(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (k, c, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": k, "Counter_Name": c, "Counter_Value": v})


def test_stalls_fractions(tmp_path, capsys):
    rows = []
    for wave_cyc, wait, wait_i, act in ((1000, 500, 200, 300), (3000, 1500, 600, 900)):  # two dispatches of K1
        rows += [(K1, "SQ_WAVE_CYCLES", wave_cyc), (K1, "SQ_WAIT_ANY", wait), (K1, "SQ_WAIT_INST_ANY", wait_i),
                 (K1, "SQ_ACTIVE_INST_ANY", act), (K1, "SQ_ACTIVE_INST_LDS", 40), (K1, "SQ_WAIT_INST_LDS", 20)]
    rows += [(K2, "SQ_WAVE_CYCLES", 100), (K2, "SQ_WAIT_ANY", 25), (K2, "SQ_WAIT_INST_ANY", 25),
             (K2, "SQ_ACTIVE_INST_ANY", 50), (K2, "SQ_ACTIVE_INST_LDS", 10), (K2, "SQ_WAIT_INST_LDS", 5)]
    f = tmp_path / "c.csv"
    _csv(f, rows)
    P.main(["stalls", "--csv", str(f), "--kernel", "ffn_tile_bf16_kernel<true, 2>", "ffn_tile_bf16_kernel<false, 2>"])
    out = capsys.readouterr().out.splitlines()
    # K1: means 2000 wave-cycles, 1000 waiting (50 %), 400 to issue (20 %), 600 issuing (30 %), LDS 40 / 2000
    assert "| `ffn_tile_bf16_kernel<true, 2>` | 2 | 2e+03 | 50.0% | 20.0% | 30.0% | 2.0% | 1.0% |" in out
    assert "| `ffn_tile_bf16_kernel<false, 2>` | 1 | 100 | 25.0% | 25.0% | 50.0% | 10.0% | 5.0% |" in out


def test_mfma_rate(tmp_path, capsys):
    # 2e9 MOPs per dispatch = 1024 GFLOP (512 flops a MOP); over 1000 us that is 1024 TFLOP/s, 41.0 % of 2.5 PFLOP/s
    rows = [(K1, "SQ_VALU_MFMA_BUSY_CYCLES", 10), (K1, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 2e9), (K1, "GRBM_GUI_ACTIVE", 5)]
    f = tmp_path / "m.csv"
    _csv(f, rows)
    P.main(["mfma", "--csv", str(f), "--kernel", "ffn_tile_bf16_kernel<true, 2>", "--avg-us", "1000"])
    out = capsys.readouterr().out
    assert "| 1024.0 | 1000.0 | 1024 | 41.0% |" in out


def test_groups_and_copy_reference():
    assert P.group_of(K1) == "ffn"
    assert P.group_of("void dmoe::(anonymous namespace)::combine_kernel<float, true, void>(...)") == "combine"
    assert P.group_of("void dmoe::(anonymous namespace)::layer_router_kernel(...)") == "layer"
    assert P.group_of("void dmoe::(anonymous namespace)::schedule_kernel(...)") == "route"
    assert P.group_of("void dmoe::(anonymous namespace)::pack_down_bf16_kernel(...)") is None
    assert P.group_of("void at::native::elementwise_kernel<...>") is None
    # the copy reference: the median of the large plain-copy dispatches (small ones are other traffic)
    copy = "void at::native::elementwise_kernel<128, 2, direct_copy_kernel_cuda>"
    rows = [(0, copy, 10.0), (1, copy, 524288.0), (2, copy, 524300.0), (3, copy, 524290.0), (4, K1, 9e9)]
    assert P.copy_kib(rows) == 524290.0
