"""Host-side helpers of bench.py (CPU only): the chained Stage II batch and the
algorithmic byte counts the roofline figures are built on."""
import numpy as np

import bench
from paper_2605_29657_amd import synth


def test_chained_stage_keeps_registers_and_the_kept_rows_in_order():
    txt = synth.make_stage("llava15", "txt", B=3)
    R = txt.R
    kept_idx = np.array([0, 5, 7, 2, 300, 575], dtype=np.int32)
    kept_off = np.array([0, 3, 3, 6])                        # sample 1 keeps nothing
    ch = bench.chained_stage(txt, kept_idx, kept_off)
    assert list(ch.N) == [3, 0, 3]
    assert list(ch.k_off) == [0, R + 3, 2 * R + 3, 3 * R + 6]
    for b in range(3):
        kb, ckb = txt.k_off[b], ch.k_off[b]
        assert np.array_equal(ch.k[ckb:ckb + R], txt.k[kb:kb + R])            # registers
        for i, v in enumerate(kept_idx[kept_off[b]:kept_off[b + 1]]):
            assert np.array_equal(ch.k[ckb + R + i], txt.k[kb + R + v])
    # Payload rows follow the same selection with each tensor's own layout.
    co = np.concatenate([[0], np.cumsum(txt.N)])
    cco = np.concatenate([[0], np.cumsum(ch.N)])
    for pl, cpl in zip(txt.payload, ch.payload):
        assert (cpl.pad_rows, cpl.row0) == (pl.pad_rows, pl.row0)
        for b in range(3):
            for i, v in enumerate(kept_idx[kept_off[b]:kept_off[b + 1]]):
                src = co[b] + b * pl.pad_rows + pl.row0 + v
                dst = cco[b] + b * cpl.pad_rows + cpl.row0 + i
                assert np.array_equal(cpl.rows[dst], pl.rows[src])
    assert ch.q is txt.q and np.array_equal(ch.T, txt.T)


def test_stage_bytes_of_the_headline_image():
    # Per LLaVA-NeXT image: Stage II keys 2884 x 32 x 128 bf16, 128 x 32 x 128 query
    # rows, 4 B per score; 40 survivors gather 24 KB rows (read and write) plus 4 B each.
    sb = synth.make_stage("llava_next", "txt", B=1)
    got = bench.stage_bytes(sb, np.array([40]))
    assert got["keys"] == 2884 * 32 * 128 * 2
    assert got["q"] == 128 * 32 * 128 * 2
    assert got["scores"] == 2884 * 4
    assert got["gather"] == 2 * 40 * (4096 + 32 * 128 + 32 * 128) * 2 + 4 * 40
    assert got["total"] == got["keys"] + got["q"] + got["scores"] + got["gather"]


def _counter_csv(path, rows):
    import csv
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, counter, value) in enumerate(rows):
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter,
                        "Counter_Value": value})


def test_traffic_from_counters_scales_by_the_calibration_copy(tmp_path):
    # Two scoring dispatches and a 1 GiB copy whose FETCH_SIZE reads half its bytes: the
    # kernel's fetch is doubled, its write kept; the earlier copyBuffer dispatches are set-up.
    score = "void occam::text_score_kernel<8, false, true>(occam::Prob, ...)"
    copy = "__amd_rocclr_copyBuffer"
    fetch = tmp_path / "fetch.csv"
    write = tmp_path / "write.csv"
    _counter_csv(fetch, [(copy, "FETCH_SIZE", 7.0), (score, "FETCH_SIZE", 1000.0),
                         (score, "FETCH_SIZE", 1200.0), (copy, "FETCH_SIZE", 524288.0)])
    _counter_csv(write, [(copy, "WRITE_SIZE", 9.0), (score, "WRITE_SIZE", 10.0),
                         (score, "WRITE_SIZE", 14.0), (copy, "WRITE_SIZE", 1048576.0)])
    tj = bench.traffic_from_counters(str(fetch), str(write), "llava_next")
    assert tj["fetch_scale"] == 2.0 and tj["write_scale"] == 1.0
    assert tj["fetch_bytes"] == 1100 * 2 * 1024
    assert tj["write_bytes"] == 12 * 1024
    assert tj["bytes_per_launch"] == tj["fetch_bytes"] + tj["write_bytes"]
    assert tj["dispatches"] == [2, 2]
    assert tj["source_sha256"] == bench.score_source_sha256()


def test_trace_summary_finds_the_step_sequence_and_the_lone_scoring_loop(tmp_path):
    import csv
    names = [k for k, _ in bench.STEP_KERNELS]
    rows, t = [], 0

    def launch(name, us):
        nonlocal t
        rows.append({"Kernel_Name": "void occam::%s(occam::Prob, ...)" % name,
                     "Start_Timestamp": t, "End_Timestamp": t + int(us * 1000)})
        t += int(us * 1000) + 500

    launch("at::native::fill", 3.0)                    # set-up work is skipped
    for rep in range(65):                              # 40 settling + 5 warm-up + 20 timed
        for k, n in enumerate(names):
            launch(n, 10.0 * (k + 1) + (rep >= 45) * 1.0)
        if rep == 7:
            launch("at::native::copy", 2.0)
    for i in range(31):                                # settling + 20 timed, alone
        launch("text_score_kernel<8, false, true>", 190.0 + i)
    launch("text_stats_kernel<8, false, false, 4, 1>", 150.0)   # the next measurement
    launch("text_score_kernel<8, false, true>", 999.0)
    for rep in range(30):                              # ablation steps: the same sequence
        for k, n in enumerate(names):
            launch(n, 500.0)
    path = tmp_path / "trace.csv"
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        w.writerows(rows)
    got = bench.trace_summary(str(path), warmup=5, steps=20)
    assert [x["avg_us"] for x in got["steps"]] == [10.0 * (k + 1) + 1.0 for k in range(len(names))]
    assert got["matched_steps"] == 65
    assert got["text_score_alone"]["n"] == 20
    assert got["text_score_alone"]["min_us"] == 201.0 and got["text_score_alone"]["max_us"] == 220.0


def test_fetch_summary_scales_every_kernel(tmp_path):
    # Per-kernel means of FETCH_SIZE / WRITE_SIZE, scaled by the calibration copy (a 1 GiB
    # copy whose FETCH_SIZE reads half its bytes); PyTorch's own kernels are skipped.
    stats = "void occam::text_stats_kernel<8, false, false, 4, 1>(occam::Prob, ...)"
    score = "void occam::text_score_kernel<8, false, false>(occam::Prob, ...)"
    copy = "__amd_rocclr_copyBuffer"
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    _counter_csv(fetch, [("at::native::fill", "FETCH_SIZE", 5.0), (stats, "FETCH_SIZE", 100.0),
                         (stats, "FETCH_SIZE", 300.0), (score, "FETCH_SIZE", 50.0),
                         (copy, "FETCH_SIZE", 524288.0)])
    _counter_csv(write, [(stats, "WRITE_SIZE", 4.0), (stats, "WRITE_SIZE", 6.0),
                         (score, "WRITE_SIZE", 1.0), (copy, "WRITE_SIZE", 1048576.0)])
    got = bench.fetch_summary(str(fetch), str(write))
    assert got["fetch_scale"] == 2.0 and got["write_scale"] == 1.0
    ks = got["kernels"]
    assert set(ks) == {"text_stats_kernel<8, false, false, 4, 1>", "text_score_kernel<8, false, false>"}
    assert ks["text_stats_kernel<8, false, false, 4, 1>"] == {"fetch_bytes": 200 * 2 * 1024,
                                                           "write_bytes": 5 * 1024, "dispatches": 2}
    assert ks["text_score_kernel<8, false, false>"]["fetch_bytes"] == 50 * 2 * 1024


def test_step_description_covers_ragged_workloads():
    # The bench line's workload text for a ragged batch gives ranges (it used to format a
    # range as one integer and fail); the uniform headline text is unchanged.
    from paper_2605_29657_amd import synth
    v = synth.make_stage("qwen3vl_ragged", "vis", B=3)
    t = synth.make_stage("qwen3vl_ragged", "txt", B=3)
    desc = bench.step_desc("qwen3vl_ragged", v, t)
    assert "N=%d-%d visual tokens" % (v.N.min(), v.N.max()) in desc
    assert "d=72" in desc and "1152-wide hidden" in desc
    v = synth.make_stage("llava_next", "vis", B=2)
    t = synth.make_stage("llava_next", "txt", B=2)
    assert bench.step_desc("llava_next", v, t) == (
        "llava_next: B=2, R=4, N=2880 visual tokens; Stage I CLS row H=16 d=64 + 1024-wide hidden "
        "gather; Stage II 128 text rows H=32 d=128 over all 2880 tokens + hidden/K/V gather")


def test_cycler_runs_the_copies_in_turn():
    # Every timed loop of the bench calls one cycled function per step: copy 0, 1, 2, 0, ...
    seen = []
    one = bench.cycler([lambda i=i: seen.append(i) for i in range(bench.NCOPY)])
    for _ in range(2 * bench.NCOPY + 1):
        one()
    assert seen == list(range(bench.NCOPY)) * 2 + [0]
    assert bench.NCOPY >= 3
