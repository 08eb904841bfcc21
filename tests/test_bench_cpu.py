"""The benchmark's host logic (no GPU): the stratified frame sample reproduces the
stream's mean context, and the multi-GPU request is refused with a message."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("steps", [1, 5, 20, 37, 100, 999])
def test_stratified_frames_cover_the_stream(steps):
    t = bench.stratified(1000, steps)
    assert len(t) == steps == len(set(t)) and t == sorted(t)
    assert 0 <= t[0] and t[-1] < 1000
    # one frame from the middle of each of `steps` equal stretches
    for i, x in enumerate(t):
        assert i * 1000 // steps <= x < (i + 1) * 1000 // steps + 1
    # memory t * 10 rows: the sample's mean context is the stream's (1041 + 4995), within half a stretch
    mean_ctx = 1041 + 10 * sum(t) / steps
    assert abs(mean_ctx - 6036) <= 10 * 500 / steps + 1e-9


def test_whole_stream_when_steps_equal_its_length():
    assert bench.stratified(1000, 1000) == list(range(1000))
    from paper_2609_23286_amd import synth
    cfg = synth.CONFIGS["vitl_stack_1000"]
    assert bench.workload_key(cfg, 1000, 1000, []) == "vitl_stack_1000"
    assert bench.workload_key(cfg, 1000, 20, []) == "vitl_stack_1000__20of1000"
    assert bench.workload_key(cfg, 1000, 20, ["gamma 0.02"]) is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


# ---- the profile summaries (written into a temporary profiles/ directory) --------------

def _lines(path):
    with open(path) as fh:
        return fh.read()


def test_unit_rates_summary_derives_the_rates(tmp_path, monkeypatch):
    """Two MFMA waves at 16 ns per 32-cycle MFMA mean a 2.00 GHz clock; at 2.4 GHz, 32 FMAs
    in 32 ns from one wave are 2.4 cycles each, 64 in 40 ns from two are 1.5; 32
    exponentials in 160 ns from one wave are 12 cycles each, 64 in 240 ns from two 9.0
    (6.0x the two-wave FMA); the chained body then costs 16 x 9.0 + 32 x 1.5 = 192 cycles."""
    import json
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    ns = {"mfma_wave": 80.0, "valu_wave": 200.0, "mfma_wave_and_valu_wave": 208.0, "one_wave_both": 210.0,
          "two_mfma_waves": 128.0, "two_mfma_waves_zero_operands": 120.0, "two_valu_waves": 256.0,
          "fma_wave": 32.0, "two_fma_waves": 40.0, "exp_wave": 160.0, "two_exp_waves": 240.0}
    src = tmp_path / "ur.json"
    src.write_text(json.dumps({"ns_per_iter": ns, "cus": 256, "iterations": 4000}) + "\n")
    bench.unit_rates_summary(str(src))
    text = _lines(tmp_path / "unit_rates__mi355x.md")
    assert "16.0 ns per 32x32x16 bf16 MFMA" in text and "runs at 2.00 GHz (83 %" in text
    assert "2.4 SIMD cycles each from one wave (one wave's issue limit), 1.5 from two" in text
    assert "12.0 SIMD cycles each from one wave, 9.0 from two" in text and "6.0x as long as an FMA" in text
    assert "= 307 cycles per body against 192 at the single-unit costs" in text  # 256 * 2.4 / 2
    assert "hidden under VALU work on the same SIMD (one wave of each): 90 %" in text  # (80 + 200 - 208) / 80


def test_unit_rates_counters_summary(tmp_path, monkeypatch):
    """Counter rows per probe mode: the clock is GUI cycles per XCD over the duration, the
    vector-ALU share 4 x SQ_ACTIVE_INST_VALU over the SIMD cycles."""
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    d = tmp_path / "ur"
    d.mkdir()
    header = ("Correlation_Id,Dispatch_Id,Agent_Id,Queue_Id,Process_Id,Thread_Id,Grid_Size,Kernel_Id,Kernel_Name,"
              "Workgroup_Size,LDS_Block_Size,Scratch_Size,VGPR_Count,Accum_VGPR_Count,SGPR_Count,Counter_Name,"
              "Counter_Value,Start_Timestamp,End_Timestamp\n")
    rows = []
    dur = 1_000_000  # 1 ms
    gui = 8 * 2_000_000  # 2.0 GHz on each of 8 XCDs
    simd = 2_000_000 * 1024
    values = {"GRBM_GUI_ACTIVE": gui, "SQ_ACTIVE_INST_VALU": simd / 4 * 0.5, "SQ_VALU_MFMA_BUSY_CYCLES": simd * 0.25,
              "SQ_INSTS_VALU": 256 * 8 * 4000 * 48, "SQ_INSTS_VALU_TRANS_F32": 256 * 8 * 4000 * 16}
    for disp, kernel in ((1, "unit_rate_kernel<6>"), (2, "unit_rate_kernel<6>"), (3, "issue_rate_kernel<9>")):
        for name, v in values.items():
            rows.append(f'{disp},{disp},"Agent 1",1,1,1,131072,7,"void (anonymous namespace)::{kernel}'
                        f'(float*, int)",512,0,0,40,0,16,"{name}",{v},1000,{1000 + dur}\n')
    (d / "ur_counter_collection.csv").write_text(header + "".join(rows))
    bench.unit_rates_counters(str(d))
    text = _lines(tmp_path / "unit_rates__mi355x__counters.md")
    assert "| two VALU waves | 250.0 | 2.00 | 50.0 % | 25.0 % | 48.0 | 16.0 |" in text
    # the exponential probe issues from four waves per workgroup: twice the instructions per wave
    assert "| one exp wave | 250.0 | 2.00 | 50.0 % | 25.0 % | 96.0 | 32.0 |" in text


def test_library_context_summary(tmp_path, monkeypatch):
    """The comparison table: TFLOP/s from 4 N H d (M + N) flops per call, speed-up against
    the faster torch backend."""
    import json
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    flops = bench.attention_flops(1041, 16, 64, 1041 + 9990)
    r = {"config": "vitl_stack_1000", "tokens": 1041, "heads": 16, "head_dim": 64, "reps": 50,
         "rows": [{"mem_len": 9990, "context": 11031, "flops": flops, "rv_us": 50.0, "flash_us": 400.0,
                   "efficient_us": 300.0, "flash_max_abs_diff": 1e-5, "efficient_max_abs_diff": 2e-5}],
         "gemm_bf16": {"m": 8192, "n": 8192, "k": 8192, "us": 1000.0, "tflops": 1099.5},
         "torch": "t", "hip": "h"}
    src = tmp_path / "lc.json"
    src.write_text(json.dumps(r) + "\n")
    bench.library_context_summary(str(src))
    text = _lines(tmp_path / "attention_vs_torch_sdpa__vitl_stack_1000_layer_step.md")
    tf = flops / 50.0 / 1e6
    assert f"| 9990 | 50.0 | {tf:.0f} ({100 * tf / bench.PEAK_BF16_TFLOPS:.1f} %) | 400.0 | 300.0 | 6.00x | 2e-05 |" in text
    assert "1100 TFLOP/s" in text


def test_traffic_summary_scales_by_the_calibration_copy(tmp_path, monkeypatch):
    """The counters' KiB per dispatch become bytes through the factors the 256 MiB copy
    gives (here: FETCH_SIZE reads half the copy's bytes, WRITE_SIZE all of them), and the
    benchmark reads the figure back only for the code it was taken with."""
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    header = ("Correlation_Id,Dispatch_Id,Agent_Id,Queue_Id,Process_Id,Thread_Id,Grid_Size,Kernel_Id,Kernel_Name,"
              "Workgroup_Size,LDS_Block_Size,Scratch_Size,VGPR_Count,Accum_VGPR_Count,SGPR_Count,Counter_Name,"
              "Counter_Value,Start_Timestamp,End_Timestamp\n")
    copy_kib = bench.COPY_CALIBRATION_BYTES / 1024.0
    kib = {"attn_fwd_kernel": (1000.0, 500.0), "attn_merge_kernel": (300.0, 100.0), "sal_kernel": (2000.0, 50.0),
           "select_kernel": (80.0, 60.0)}
    for counter, half, sub, col in (("FETCH_SIZE", copy_kib / 2, "fetch", 0), ("WRITE_SIZE", copy_kib, "write", 1)):
        d = tmp_path / sub
        d.mkdir()
        rows = [f'1,1,"Agent 1",1,1,1,1,1,"void at::native::neg_kernel(float*)",256,0,0,8,0,8,"{counter}",{half},0,1\n']
        for i, (k, v) in enumerate(kib.items()):
            rows.append(f'{i + 2},{i + 2},"Agent 1",1,1,1,1,1,"rv::(anonymous namespace)::{k}(rv::Args)",256,0,0,8,0,8,'
                        f'"{counter}",{v[col]},0,1\n')
        (d / f"{sub}_counter_collection.csv").write_text(header + "".join(rows))
    bench.summarize_pmc(str(tmp_path / "fetch"), str(tmp_path / "write"), "w")
    for k, (f, w) in kib.items():
        expect = f * 1024 * 2 + w * 1024 * 1
        assert bench.recorded_traffic(k, "w") == pytest.approx(expect)
    assert bench.attention_traffic("w") == pytest.approx((1000 * 2 + 500 + 300 * 2 + 100) * 1024)
    assert bench.admission_traffic("w") == pytest.approx((2000 * 2 + 50 + 80 * 2 + 60) * 1024)


def test_summary_commands_quote_the_benchmark_arguments_only(monkeypatch):
    """Each summary option's own arguments are dropped from the quoted benchmark command."""
    monkeypatch.setattr(sys, "argv", ["bench.py", "--steps", "20", "--mfma-summary", "a", "b", "c", "t.json",
                                      "--warmup", "5"])
    assert bench.bench_args() == "--steps 20 --warmup 5"
    monkeypatch.setattr(sys, "argv", ["bench.py", "--trace-summary", "d", "t.json", "--staged", "--pmc-summary",
                                      "f", "w"])
    assert bench.bench_args() == "--staged"


def test_profile_summaries_keep_the_timed_frames_dispatches():
    """Generator and warm-up dispatches precede the timed frames: the window starts at the
    first of the last steps x layers attention launches (or the frame-staging launch
    before it), and without steps and layers nothing is left out."""
    d = [("gen_qkv_kernel", 1), ("attn_fwd_kernel", 10), ("attn_merge_kernel", 11), ("attn_fwd_kernel", 12),
         ("sal_kernel", 13), ("select_kernel", 14),                                  # warm-up frame
         ("attn_fwd_kernel", 20), ("attn_fwd_kernel", 22), ("attn_merge_kernel", 23), ("sal_kernel", 24),
         ("select_kernel", 25), ("attn_fwd_kernel", 30), ("attn_fwd_kernel", 32), ("sal_kernel", 34),
         ("select_kernel", 35)]                                                      # two timed frames
    assert bench.timed_start(d, 2, 2) == 20
    assert bench.timed_start(d, None, 2) is None and bench.timed_start(d, 9, 2) is None
    staged = [("stage_layers_kernel", 5)] + d[:6] + [("stage_layers_kernel", 19)] + d[6:11] + \
             [("stage_layers_kernel", 29)] + d[11:]
    assert bench.timed_start(staged, 2, 2) == 19
    rows = [{"Dispatch_Id": str(i), "Kernel_Name": n, "Start_Timestamp": str(t), "Counter_Name": c}
            for i, (n, t) in enumerate(d) for c in ("FETCH_SIZE", "WRITE_SIZE")]
    kept = bench.timed_counter_rows(rows, 2, 2)
    assert len(kept) == 2 * 9 and min(int(r["Start_Timestamp"]) for r in kept) == 20
    assert bench.timed_counter_rows(rows, None, None) == rows
