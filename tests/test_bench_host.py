"""Host logic of bench.py (no GPU): the algorithmic byte counts behind the reported roofline and rates, and the
refusal of a multi-GPU run.

The byte counts are checked against the per-unit figures of the measurement plan written out term by term
here (K read once per scored row and KV head, queries, positions, one row of group sums per block of merged KV
heads written by the scorer and read by the fold, u read and written, the newcomer's K/V rows read and written
once), so a dropped or doubled term in bench.py fails."""
import json
import os
import subprocess
import sys

import bench
from workload import LLAMA8B, QWEN, SCOREFREE128K

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_steady_step_bytes_8b():
    """The 8B steady step: n = B + 1 = 3,278 rows, the scorer merging 4 KV heads (the figures quoted in the
    profiles and the benchmark record)."""
    L, b, hq, hkv, d, n, e = 32, 8, 32, 8, 128, 3278, 2
    k_rows = L * b * hkv * n * d * e          # every cached row of every KV head, and the newcomer's
    queries = L * b * hq * d * e
    positions = b * n * 4
    sums = L * b * (hkv // 4) * n * 4        # one row of group sums per block of 4 KV heads
    by = bench.step_bytes(LLAMA8B, n, merge=4)
    assert by["score"] == k_rows + queries + positions + sums == 1_727_531_456
    assert by["fold"] == sums + b * n * 4 * 3 == 7_028_032      # sums read; u read and written; pos read
    assert by["place"] == 2 * 2 * L * b * hkv * d * e + 2 * b * 8 == 2_097_280
    assert by["total"] == 1_736_656_768


def test_steady_step_bytes_scale_with_merge_and_dtype():
    n = QWEN.budget + 1
    one, two = bench.step_bytes(QWEN, n, merge=1), bench.step_bytes(QWEN, n, merge=2)
    rows_saved = QWEN.layers * QWEN.batch * (QWEN.n_kv_heads // 2) * n * 4
    assert one["score"] - two["score"] == rows_saved and one["fold"] - two["fold"] == rows_saved
    f32 = LLAMA8B.scaled(dtype="f32")
    # K, queries and the newcomer's rows double with 4-byte elements; the fp32 bookkeeping does not
    assert (bench.step_bytes(f32, 3278)["score"] - bench.step_bytes(LLAMA8B, 3278)["score"]
            == 32 * 8 * 8 * 3278 * 128 * 2 + 32 * 8 * 32 * 128 * 2)


def test_first_step_bytes_charge_logits_only_on_the_logits_path():
    """Step 1: the chunk-exchange scorer (path 1) keeps the logits in LDS; only the logits path (2) writes them
    and reads them back."""
    cfg, n = SCOREFREE128K, SCOREFREE128K.prefill_len + 1
    holes = [11_773, 11_779]
    exchange, logits = bench.step1_bytes(cfg, n, holes, 1), bench.step1_bytes(cfg, n, holes, 2)
    assert logits - exchange == 2 * cfg.layers * cfg.batch * cfg.n_q_heads * n * 4
    # every moved row: K and V of every layer and KV head read and written, its utility and position
    fewer = bench.step1_bytes(cfg, n, [holes[0] - 1, holes[1]], 1)
    assert exchange - fewer == 2 * 2 * cfg.layers * cfg.n_kv_heads * cfg.head_dim * 2 + 16
    # group sums of 4 KV heads added by the scorer: a quarter of the rows written and read back
    merged = bench.step1_bytes(cfg, n, holes, 1, merge=4)
    assert exchange - merged == 2 * cfg.layers * cfg.batch * (cfg.n_kv_heads - cfg.n_kv_heads // 4) * n * 4


def test_nonrefresh_bytes():
    n = LLAMA8B.budget
    assert bench.nonrefresh_bytes(LLAMA8B, n) == 8 * n * 8 + 2 * 2 * 32 * 8 * 8 * 128 * 2 + 8 * 8


def test_more_than_one_gpu_is_refused():
    """One GPU is measured; --gpus 2 exits with status 2 and a JSON line that says so (before any GPU work)."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]
