"""GPU parity of the entry points that take the window rows' normalisers from
the caller (the log-sum-exp of the layer's prefill attention), through the C
ABI, against the float64 oracle: scores within 2e-3, the whole step with the
same end-to-end bar as kvec_evict_model, and agreement with kvec_score."""
import sys

import numpy as np
import pytest

import oracle as orc
import synth
from kvec_testlib import SCORE_RTOL, layer_inputs, oracle_scores, rel_err, to_device
from test_gpu_parity import SCORE_CASES, _e2e, _small

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _lse_dev(w, layer):
    import torch
    return torch.from_numpy(np.stack([
        orc.to_f32(orc.window_lse(synth.to_f64(synth.queries(w, layer, b), w.dtype),
                                  synth.to_f64(synth.keys(w, layer, b), w.dtype)))
        for b in range(w.batch)])).cuda()


@pytest.mark.parametrize("w", SCORE_CASES, ids=lambda w: w.name)
def test_score_lse_parity(gpu_lib, w):
    import torch
    kv = gpu_lib
    _say(f"[score-lse] {w.name} T={w.seq_len} O={w.window} Wn={w.rows} H={w.n_kv_heads} G={w.group}")
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    Tc = w.candidates
    layer = 0
    q = torch.stack([to_device(layer_inputs(w, layer, b)[0], w) for b in range(w.batch)])
    k = torch.stack([to_device(layer_inputs(w, layer, b)[1], w) for b in range(w.batch)])
    lse = _lse_dev(w, layer)
    p = torch.empty((w.batch, w.n_kv_heads, Tc), dtype=torch.float32, device="cuda")
    pe = torch.empty_like(p)
    imp = torch.empty((w.batch, Tc), dtype=torch.float32, device="cuda")
    kv.kvec_score_lse(cfg, q, lse, k, p, pe, imp, ws)
    # the two-pass scores of the same inputs, for the agreement of the paths
    p2 = torch.empty_like(p)
    pe2 = torch.empty_like(p)
    imp2 = torch.empty_like(imp)
    kv.kvec_score(cfg, q, k, p2, pe2, imp2, ws)
    torch.cuda.synchronize()
    for b in range(w.batch):
        rp, rpe, rimp = oracle_scores(w, layer, b)
        e = (rel_err(p[b].cpu().numpy(), rp), rel_err(pe[b].cpu().numpy(), rpe),
             rel_err(imp[b].cpu().numpy(), rimp))
        _say(f"   seq {b}: rel err P {e[0]:.2e} P' {e[1]:.2e} I {e[2]:.2e}")
        assert max(e) <= SCORE_RTOL, e
        d = (rel_err(p[b].cpu().numpy(), p2[b].cpu().numpy()),
             rel_err(imp[b].cpu().numpy(), imp2[b].cpu().numpy()))
        assert max(d) <= SCORE_RTOL, d


def test_score_lse_strided(gpu_lib):
    """lse rows taken out of a wider [b][HQ][T] log-sum-exp array (the layout a
    prefill attention returns): the head stride is T, the window rows its tail."""
    import torch
    kv = gpu_lib
    w = _small("lse-strided", 900, 16, 32, 4, 2, 128, "bf16", batch=2)
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    q = torch.stack([to_device(layer_inputs(w, 0, b)[0], w) for b in range(w.batch)])
    k = torch.stack([to_device(layer_inputs(w, 0, b)[1], w) for b in range(w.batch)])
    full = torch.full((w.batch, w.n_q_heads, w.seq_len), float("nan"), device="cuda")
    full[:, :, w.seq_len - w.rows:] = _lse_dev(w, 0)
    lse = full[:, :, w.seq_len - w.rows:]
    assert lse.stride() == (w.n_q_heads * w.seq_len, w.seq_len, 1)
    Tc = w.candidates
    p = torch.empty((w.batch, w.n_kv_heads, Tc), dtype=torch.float32, device="cuda")
    pe = torch.empty_like(p)
    imp = torch.empty((w.batch, Tc), dtype=torch.float32, device="cuda")
    kv.kvec_score_lse(cfg, q, lse, k, p, pe, imp, ws)
    torch.cuda.synchronize()
    for b in range(w.batch):
        rp, rpe, rimp = oracle_scores(w, 0, b)
        e = (rel_err(p[b].cpu().numpy(), rp), rel_err(pe[b].cpu().numpy(), rpe),
             rel_err(imp[b].cpu().numpy(), rimp))
        assert max(e) <= SCORE_RTOL, e


def test_e2e_lse_tiny_fp32(gpu_lib):
    _e2e(gpu_lib, synth.workload(0), lse=True)


def test_e2e_lse_small_bf16(gpu_lib):
    _e2e(gpu_lib, _small("e2e-lse-small", 2500, 32, 64, 8, 4, 128, "bf16", B=200, layers=6),
         lse=True)


def test_e2e_lse_batch2_o64(gpu_lib):
    _e2e(gpu_lib, _small("e2e-lse-b2", 3000, 64, 128, 8, 4, 128, "bf16", batch=2, B=300,
                         layers=4, pool=5), lse=True)


def test_full_llama8b_32k_lse_sampled_layers(gpu_lib):
    """The benchmark's 32k workload through kvec_evict_model_lse."""
    _e2e(gpu_lib, synth.workload(2), check_layers=[0, 1, 31], lse=True)


def test_e2e_lse_window_equals_extended(gpu_lib):
    """O' = O: no extended-window stages in the given-lse pipeline."""
    _e2e(gpu_lib, _small("e2e-lse-wn-eq-o", 1800, 16, 16, 4, 2, 64, "bf16", B=120, layers=3),
         lse=True)


def test_e2e_lse_group7_entropy(gpu_lib):
    """GQA group 7 (the Qwen2.5-7B grouping) with the entropy criterion."""
    _e2e(gpu_lib, _small("e2e-lse-g7-ent", 2600, 32, 64, 4, 7, 128, "bf16", B=256, layers=3,
                         criterion="entropy"), lse=True)


def test_lse_keep_everything_when_budget_covers(gpu_lib):
    """T <= B: every token is kept; the row normalisers are required but unread."""
    import torch
    kv = gpu_lib
    w = _small("lse-keep-all", 100, 8, 16, 2, 2, 64, "bf16", B=128, layers=2)
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(max(kv.kvec_workspace_size(cfg), 256), dtype=torch.uint8, device="cuda")
    from kvec_testlib import model_tensors
    q, k, v = model_tensors(w)
    lse = torch.full((2, 1, 4, w.rows), float("nan"), dtype=torch.float32, device="cuda")
    bits = torch.zeros((1, 2, 2), dtype=torch.int64, device="cuda")
    idx = torch.empty((2, 1, 2, 128), dtype=torch.int32, device="cuda")
    ko = torch.empty((2, 1, 2, 128, 64), dtype=k.dtype, device="cuda")
    vo = torch.empty_like(ko)
    kv.kvec_evict_model_lse(cfg, q, lse, k, v, bits, idx, ko, vo, ws)
    torch.cuda.synchronize()
    gi = idx.cpu().numpy()
    assert np.all(gi[:, :, :, :100] == np.arange(100))
    assert np.all(gi[:, :, :, 100:] == -1)
    assert torch.equal(ko[:, :, :, :100], k)


def test_layer_lse_calls_match_model_step(gpu_lib):
    """kvec_evict_layer_lse called layer by layer (as inside a prefill loop)
    reproduces kvec_evict_model_lse exactly."""
    import torch
    from test_gpu_parity import oracle_lse_tensor
    from kvec_testlib import model_tensors
    kv = gpu_lib
    w = _small("layerwise-lse", 3000, 32, 64, 4, 4, 128, "bf16", batch=2, B=256, layers=4)
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    q, k, v = model_tensors(w)
    lse = oracle_lse_tensor(w)
    L, H, B, T, d = w.n_layers, w.n_kv_heads, w.budget, w.seq_len, w.head_dim
    W = (T + 63) // 64
    bits_m = torch.empty((w.batch, L, W), dtype=torch.int64, device="cuda")
    idx_m = torch.empty((L, w.batch, H, B), dtype=torch.int32, device="cuda")
    ko_m = torch.empty((L, w.batch, H, B, d), dtype=k.dtype, device="cuda")
    vo_m = torch.empty_like(ko_m)
    kv.kvec_evict_model_lse(cfg, q, lse, k, v, bits_m, idx_m, ko_m, vo_m, ws)
    bits_l = torch.zeros_like(bits_m)
    idx_l = torch.empty_like(idx_m)
    ko_l = torch.empty_like(ko_m)
    vo_l = torch.empty_like(vo_m)
    for l in range(L):
        kv.kvec_evict_layer_lse(cfg, l, q[l], lse[l], k[l], v[l], bits_l, idx_l[l], ko_l[l],
                                vo_l[l], ws)
    torch.cuda.synchronize()
    assert torch.equal(idx_m, idx_l)
    assert torch.equal(bits_m, bits_l)
    assert torch.equal(ko_m.view(torch.int16), ko_l.view(torch.int16))
    assert torch.equal(vo_m.view(torch.int16), vo_l.view(torch.int16))
