"""Host logic of the bench's profile summaries: cutting a hash run's counter
records into calls and picking one series out of them, and the batch case's
algorithmic bytes."""
import csv
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
import bench  # noqa: E402

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]


def write_counters(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(FIELDS, r)))


def line_with(cases):
    return {"hash": {name: {"calls": calls} for name, calls in cases}}


def test_counter_calls_end_at_the_chain_or_fused_kernel(tmp_path):
    # dispatch order, not file order, decides; other kernels are skipped
    rows = [
        (3, "void ea::(anonymous namespace)::sha256_chain_split<int>(...)", "FETCH_SIZE", 30),
        (1, "void ea::(anonymous namespace)::hash_offsets_partials(...)", "FETCH_SIZE", 10),
        (2, "void ea::(anonymous namespace)::sha256_midstates<int>(...)", "FETCH_SIZE", 20),
        (4, "at::native::vectorized_elementwise_kernel(...)", "FETCH_SIZE", 99),
        (5, "void ea::(anonymous namespace)::hash_offsets_partials(...)", "FETCH_SIZE", 11),
        (6, "void ea::(anonymous namespace)::sha256_fused_scan(...)", "FETCH_SIZE", 40),
        (6, "void ea::(anonymous namespace)::sha256_fused_scan(...)", "WRITE_SIZE", 7),
    ]
    p = tmp_path / "c.csv"
    write_counters(p, rows)
    calls = bench._hash_counter_calls(str(p), "FETCH_SIZE")
    assert [[v for _, v in c] for c in calls] == [[10.0, 20.0, 30.0], [11.0, 40.0]]


def test_series_is_located_by_the_recorded_counts():
    # two cases, each a check call then two series of (untimed, timed) calls
    line = line_with([("a", {"device_offsets": [2, 3], "host_offsets": [1, 2]}),
                      ("b", {"device_offsets": [4, 2], "host_offsets": [1, 1]})])
    n = (1 + 2 + 3 + 1 + 2) + (1 + 4 + 2 + 1 + 1)
    calls = [[("k", float(i))] for i in range(n)]
    got = bench._hash_series(line, calls, "b", "device_offsets")
    # case a takes calls 0..8; b's check call is 9, its untimed 10..13
    assert [c[0][1] for c in got] == [14.0, 15.0]
    got = bench._hash_series(line, calls, "a", "host_offsets")
    assert [c[0][1] for c in got] == [7.0, 8.0]
    with pytest.raises(SystemExit):
        bench._hash_series(line, calls[:-1], "a", "host_offsets")


def test_batch_bytes_count_each_byte_once():
    n, t, b = bench.HASH_BATCH
    assert bench.hash_batch_bytes() == n * t * 4 + 2 * (n + 1) * 8 + n * (t // b) * 32
    assert bench.hash_batch_bytes() == 67108864 + 1048592 + 33554432
