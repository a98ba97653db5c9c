"""The plain-C consumer of the ABI (paper_2607_16213_amd/examples/selkv_c_demo.c).

It runs in a process of its own with no Python or torch: buffers from
hipMalloc, then score, select, merge, bias and one biased decode step in the
order of Algorithm 1, with the defaults of selkv_params_init in fp32 storage.
Its outputs are checked against the float64 oracle on the same stored inputs,
to the same bars as the Python-driven parity tests."""
import os
import subprocess

import numpy as np
import pytest

from oracle import selkv_oracle as O
from paper_2607_16213_amd import build as B
from paper_2607_16213_amd import synth
from tests.parity_util import SCORE_RTOL, TOL, assert_close_elem, assert_close_rows, compare_end_to_end

BUCKET, ALPHA = 32, 0.5     # selkv_params_init defaults (Appendix F)


def test_c_demo_is_built_and_checks_its_arguments():
    assert os.path.exists(B.DEMO), "build() compiles the C consumer beside its source"
    r = subprocess.run([B.DEMO], capture_output=True, text=True, timeout=60)
    assert r.returncode == 1 and "usage" in r.stderr


CASES = {
    "tiny": synth.WORKLOADS["tiny"],
    # two sequences, odd group, d = 128, ragged n, short window
    "ragged": synth.WORKLOADS["tiny"].replace(name="c_demo_ragged", batch=2, n_heads_kv=2, group=3,
                                              head_dim=128, seq_len=1000, window=20),
}


def _take(buf, off, dtype, count):
    a = np.frombuffer(buf, dtype=dtype, count=count, offset=off)
    return a, off + a.nbytes


@pytest.mark.gpu
@pytest.mark.parametrize("name", sorted(CASES))
def test_c_demo_matches_oracle(name, tmp_path):
    w = CASES[name]
    assert w.dtype == "fp32"
    t = synth.make_layer(w, 0, "cpu")
    q = synth.make_decode_queries(w, 0, 1, "cpu")[0]
    Bn, H, G, d, n, W = w.batch, w.n_heads_kv, w.group, w.head_dim, w.seq_len, w.window
    K, V, Qw, q = (x.numpy().astype(np.float32) for x in (t["K"], t["V"], t["Qwin"], q))
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as f:
        f.write(np.array([Bn, H, G, d, n, W], np.int32).tobytes())
        for x in (K, V, Qw, q):
            f.write(np.ascontiguousarray(x).tobytes())
    print(f"c demo {name}: B={Bn} H={H} G={G} d={d} n={n} W={W}", flush=True)
    r = subprocess.run([B.DEMO, str(src), str(dst)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    buf = dst.read_bytes()
    (m, mr), off = _take(buf, 0, np.int32, 2)
    m, mr = int(m), int(mr)
    ne = n - m
    kept, off = _take(buf, off, np.int32, Bn * H * m)
    evicted, off = _take(buf, off, np.int32, Bn * H * ne)
    target, off = _take(buf, off, np.int32, Bn * H * ne)
    gate, off = _take(buf, off, np.float32, Bn * H * ne)
    K_out, off = _take(buf, off, np.float32, Bn * H * m * d)
    V_out, off = _take(buf, off, np.float32, Bn * H * m * d)
    bias, off = _take(buf, off, np.float32, Bn * H * m)
    out, off = _take(buf, off, np.float32, Bn * H * G * d)
    attn, off = _take(buf, off, np.float32, Bn * H * n)
    score, off = _take(buf, off, np.float32, Bn * H * (n - mr))
    assert off == len(buf)
    kept, evicted, target, gate = (x.reshape(Bn, H, -1) for x in (kept, evicted, target, gate))
    K_out, V_out = K_out.reshape(Bn, H, m, d), V_out.reshape(Bn, H, m, d)
    bias, attn, score = bias.reshape(Bn, H, m), attn.reshape(Bn, H, n), score.reshape(Bn, H, n - mr)
    out = out.reshape(Bn, H * G, d)

    K64, V64, Q64, q64 = (x.astype(np.float64) for x in (K, V, Qw, q))
    tol = TOL["fp32"]
    for b in range(Bn):
        for h in range(H):
            ch = O.compress_head(K64[b, h], V64[b, h], Q64[b, h * G:(h + 1) * G], window=W)
            assert (m, mr) == (ch["m"], ch["mr"])
            assert_close_elem(attn[b, h], ch["attn"], SCORE_RTOL, "attn")
            assert_close_elem(score[b, h], ch["score"], SCORE_RTOL, "score")
            gpu = dict(attn=attn[b, h].astype(np.float64), score=score[b, h].astype(np.float64),
                       kept=kept[b, h], evicted=evicted[b, h], target=target[b, h],
                       gate=gate[b, h].astype(np.float64), v_out=V_out[b, h].astype(np.float64),
                       bias=bias[b, h].astype(np.float64), K_out=K_out[b, h].astype(np.float64))
            counts = compare_end_to_end(gpu, ch, K64[b, h], n, BUCKET, tol, ALPHA)
            print(f"c demo {name} b={b} h={h}: {counts}")
    # the decode step over the cache the demo built (its own K_out, V_out, bias)
    ref = O.decode_batched(q64, K_out.astype(np.float64), V_out.astype(np.float64), bias.astype(np.float64), G,
                           1.0 / np.sqrt(d))
    assert_close_rows(out, ref, tol, "decode")
