"""bench.py's host-side contract: it measures one GPU only and says so for
any other count, and its stage accounting covers the compression calls."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one MI355X" in r.stderr and r.stdout == ""


def test_stage_bytes_cover_the_compression_calls():
    import bench
    from paper_2607_16213_amd import synth
    w = synth.WORKLOADS["ctx100k"]
    m = int(w.seq_len * w.budgets[0])
    sb, per_decode, full = bench.stage_bytes(w, m)
    assert tuple(sb) == bench.STAGES
    heads = w.layers * w.batch * w.n_heads_kv
    # decode reads K and V of the compressed cache once (bf16) plus the bias, per call
    assert per_decode == w.batch * w.n_heads_kv * (2 * m * w.head_dim * 2 + 4 * m) + \
        w.batch * w.n_heads_kv * w.group * w.head_dim * (2 + 4)
    # the score pass reads K and V of the whole cache at least once
    assert sb["score"] >= heads * 2 * w.seq_len * w.head_dim * 2
    assert full > 3.9 * per_decode
