"""Host-side checks of bench.py: the multi-GPU refusal, the source digest that
gates the committed traffic figures, and the algorithmic byte and flop counts
the roofline objects use."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_figures_follow_the_kernel_sources():
    # the committed summaries carry the digest of the step kernel's sources;
    # bench.py reads their byte counts only while the digest matches
    got = bench.measured_traffic("llama8b-32k")
    path = bench.TRAFFIC_FILE.format(workload="llama8b-32k")
    digest = [l for l in open(path) if l.startswith("- source_digest")][0].split("`")[1]
    if digest == bench.source_digest():
        assert isinstance(got, int) and got > 0
    else:
        assert got is None
    assert bench.measured_traffic("no-such-workload") is None


def test_algorithmic_bytes_per_token_at_32k():
    # K read once + the query window + the gather, per prefix token: 74,240 B
    L, b, H, HQ, T, d, B, Wn, es = 32, 1, 8, 32, 32768, 128, 1024, 64, 2
    step = L * b * (H * T * d * es + HQ * Wn * d * es + 4 * H * B * d * es)
    assert step // T == 74240


def test_repeated_layers_are_copies_of_the_generated_ones():
    # the other-workload leg generates n_gen layers and repeats them; every
    # layer is its own memory and equals the generated layer l % n_gen
    import numpy as np
    import torch

    import synth
    w = synth.workload(0)
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    q, k, v = bench.gen_inputs(w, torch.device("cpu"), dt, n_gen=1)
    assert q.shape[0] == k.shape[0] == v.shape[0] == w.n_layers >= 2
    for x in (q, k, v):
        assert x[1].data_ptr() != x[0].data_ptr()
        assert torch.equal(x[1], x[0])
    k0 = synth.keys(w, 0, 0)
    got = k[0, 0].numpy() if dt == torch.float32 else k[0, 0].view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, k0)
    q2, k2, _ = bench.gen_inputs(w, torch.device("cpu"), dt)
    assert torch.equal(k2[0], k[0]) and not torch.equal(k2[1], k2[0])
