"""Host logic of the measurement: the kernel-source hash that ties the stored
traffic counters to the code they were taken on, the counter scaling and
derived figures, and the timed loop read out of a kernel trace (small
synthetic rocprofv3 CSVs)."""
from paper_2501_12162_amd import profiling


def test_hash_ignores_comments_and_whitespace_only():
    code = "int f(int a) {\n  return a + 1;  // one more\n}\n/* block\n comment */\n"
    same = "int f(int a) { return a + 1; }   // another comment\n"
    changed = "int f(int a) { return a + 2; }\n"
    assert profiling._code_only(code) == profiling._code_only(same)
    assert profiling._code_only(code) != profiling._code_only(changed)
    assert profiling._code_only("a/*x*/b") == "a b"


def test_source_hash_is_stable_and_short():
    h = profiling.kernel_source_hash()
    assert h == profiling.kernel_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0


ATTN = "void adaserve::(anonymous namespace)::tree_attn_bf16_kernel<128>(adaserve::TreeAttnArgs)"
MERGE = "void adaserve::(anonymous namespace)::tree_attn_combine_kernel<128>(adaserve::TreeAttnArgs)"
COPY = "__amd_rocclr_copyBuffer"


def _write_counters(path, rows):
    """A rocprofv3 counter_collection.csv with the columns the summaries read."""
    import csv
    path.mkdir(parents=True, exist_ok=True)
    with open(path / "s_counter_collection.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
                                          "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for i, (name, counter, value, dur) in enumerate(rows, 1):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value,
                        "Start_Timestamp": 1000 * i, "End_Timestamp": 1000 * i + dur})


def test_traffic_scaled_by_the_calibration_copy(tmp_path):
    """The copy of 256 MiB before the first attention dispatch reads
    128 Ki KiB on FETCH_SIZE (factor 2) and 256 Ki KiB on WRITE_SIZE (factor
    1); per-kernel bytes are medians over dispatches times those factors.
    Copies after the first attention dispatch are not the calibration."""
    kib = 1024.0
    fetch = [(COPY, "FETCH_SIZE", 999.0, 5), (COPY, "FETCH_SIZE", 128 * 1024.0, 5),
             (ATTN, "FETCH_SIZE", 100.0, 5), (MERGE, "FETCH_SIZE", 3.0, 5),
             (ATTN, "FETCH_SIZE", 300.0, 5), (MERGE, "FETCH_SIZE", 3.0, 5),
             (ATTN, "FETCH_SIZE", 200.0, 5), (COPY, "FETCH_SIZE", 7.0, 5)]
    write = [(COPY, "WRITE_SIZE", 256 * 1024.0, 5), (ATTN, "WRITE_SIZE", 10.0, 5),
             (ATTN, "WRITE_SIZE", 30.0, 5)]
    _write_counters(tmp_path / "f", fetch)
    _write_counters(tmp_path / "w", write)
    res = profiling.traffic_summary(str(tmp_path / "f"), str(tmp_path / "w"), 9, "cmd")
    assert res["fetch_factor"] == 2.0 and res["write_factor"] == 1.0
    attn = res["kernels"]["tree_attn"]
    assert attn["fetch_bytes"] == 200.0 * kib * 2.0      # median of 100, 300, 200
    assert attn["write_bytes"] == 20.0 * kib             # median of 10, 30
    assert attn["dispatches"] == 3
    assert res["kernels"]["tree_attn_combine"]["write_bytes"] == 0.0
    assert res["kernel_source_sha"] == profiling.kernel_source_hash()


def test_counter_summary_derived_figures(tmp_path):
    """Counters summed over 8 XCDs: 8e6 GUI cycles over a 1 ms dispatch is
    a 1 GHz clock per XCD; MFMA busy over (cycles per XCD x SIMDs)."""
    rows = [(ATTN, "GRBM_GUI_ACTIVE", 8.0e6, 1_000_000), (ATTN, "SQ_VALU_MFMA_BUSY_CYCLES", 2.56e8, 1_000_000),
            (ATTN, "SQ_INSTS_VALU", 50.0, 1_000_000), (ATTN, "SQ_INSTS_MFMA", 10.0, 1_000_000),
            (ATTN, "SQ_LDS_IDX_ACTIVE", 100.0, 1_000_000), (ATTN, "SQ_LDS_BANK_CONFLICT", 25.0, 1_000_000),
            (COPY, "GRBM_GUI_ACTIVE", 1.0, 5)]
    _write_counters(tmp_path / "c", rows)
    k = profiling.counter_summary([str(tmp_path / "c")], 4, "cmd")["kernels"]
    assert set(k) == {"tree_attn"}
    a = k["tree_attn"]
    assert a["cycles_per_xcd"] == 1.0e6 and abs(a["clock_ghz"] - 1.0) < 1e-12
    assert a["mfma_busy_frac"] == 0.25          # 2.56e8 / (1e6 * 1024)
    assert a["valu_per_mfma"] == 4.0 and a["lds_conflict_frac"] == 0.25


def test_timed_step_summary_picks_the_timed_loop(tmp_path):
    """Attention dispatches warmup .. warmup + steps - 1 are the timed loop;
    the merge launch right after each is the step's second launch; start to
    start spans the first to the last timed step."""
    import csv
    path = tmp_path / "trace.csv"
    rows, t, did = [], 0, 0

    def launch(name, dur_ns, gap_ns=1000):
        nonlocal t, did
        did += 1
        rows.append({"Dispatch_Id": did, "Kernel_Name": name, "Start_Timestamp": t, "End_Timestamp": t + dur_ns})
        t += dur_ns + gap_ns
    launch(COPY, 500)
    for step in range(7):                     # 2 warm-up, 3 timed, 2 after
        slow = step < 2 or step >= 5
        launch(ATTN, 300_000 if slow else 200_000)
        launch(MERGE, 9_000 if slow else 8_000)
    launch(COPY, 500)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        # dispatch order, not file order, decides
        w.writerows(reversed(rows))
    res = profiling.timed_step_summary(str(path), 2, 3)
    assert res["steps"] == 3
    assert res["tree_attn_us"] == 200.0 and res["tree_attn_combine_us"] == 8.0
    assert res["start_to_start_us"] == (200_000 + 1000 + 8_000 + 1000) / 1e3


STATS = "void adaserve::(anonymous namespace)::sampled_stats_kernel<true>(adaserve::SampledArgs)"
WALK = "void adaserve::(anonymous namespace)::sampled_accept_kernel<true>(adaserve::SampledArgs)"


def test_sampled_traffic_has_its_own_kernels_and_hash(tmp_path):
    """The sampled summary keeps the statistics and walk kernels only, under
    the hash of the sampled sources (which the attention hash does not
    cover, and the other way round)."""
    fetch = [(COPY, "FETCH_SIZE", 128 * 1024.0, 5), (ATTN, "FETCH_SIZE", 100.0, 5),
             (STATS, "FETCH_SIZE", 40.0, 5), (WALK, "FETCH_SIZE", 4.0, 5), (STATS, "FETCH_SIZE", 60.0, 5)]
    write = [(COPY, "WRITE_SIZE", 256 * 1024.0, 5), (ATTN, "WRITE_SIZE", 10.0, 5), (STATS, "WRITE_SIZE", 1.0, 5)]
    _write_counters(tmp_path / "f", fetch)
    _write_counters(tmp_path / "w", write)
    res = profiling.traffic_summary(str(tmp_path / "f"), str(tmp_path / "w"), 3, "cmd", sampled=True)
    assert set(res["kernels"]) == {"sampled_stats", "sampled_accept"}
    assert res["kernels"]["sampled_stats"]["fetch_bytes"] == 50.0 * 1024 * 2.0
    assert res["kernel_source_sha"] == profiling.sampled_source_hash() != profiling.kernel_source_hash()
