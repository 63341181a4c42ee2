"""kvec_evict_model_steps and kvec_evict_model_lse_steps: several independent
steps in one pipelined call.

Every step's outputs (bitmap rows, indices, kept K and V) must be
bit-identical to a kvec_evict_model (kvec_evict_model_lse) call on that step's
inputs, with layer counts below and above the pipeline depth (so that up to
several steps share a launch), distinct inputs per step, and a step stride of
0 (one prefill evicted repeatedly).  The single-step paths are checked against
the oracle elsewhere; this pins the multi-step plumbing to them.
"""
import sys

import pytest

import synth
from kvec_testlib import model_tensors
from test_gpu_parity import oracle_lse_tensor

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _wl(L, seed, T=1500, H=4, G=4, d=128, batch=2, B=200):
    return synth.Workload(f"steps-L{L}-s{seed}", L, H, H * G, d, T, batch, 32, 64, B, 7, "bf16", seed,
                          rope=True, hh_count=T // 50, n_adjust_heads=2)


def _outs(kv, w, n):
    import torch
    L, H, B, T, d = w.n_layers, w.n_kv_heads, w.budget, w.seq_len, w.head_dim
    bits = torch.zeros((n, w.batch, L, (T + 63) // 64), dtype=torch.int64, device="cuda")
    idx = torch.full((n, L, w.batch, H, B), -7, dtype=torch.int32, device="cuda")
    ko = torch.zeros((n, L, w.batch, H, B, d), dtype=torch.bfloat16, device="cuda")
    return bits, idx, ko, torch.zeros_like(ko)


def _check(kv, ws_list, n_steps, shared, lse=False):
    import torch
    w0 = ws_list[0]
    cfg = kv.Config.from_workload(w0)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    ins = [model_tensors(w) + ((oracle_lse_tensor(w),) if lse else ()) for w in ws_list]
    if shared:
        stacked = [x.unsqueeze(0).expand(n_steps, *x.shape) for x in ins[0]]
        ins = [ins[0]] * n_steps
    else:
        stacked = [torch.stack([x[i] for x in ins]) for i in range(len(ins[0]))]
    bits, idx, ko, vo = _outs(kv, w0, n_steps)
    if lse:
        q, k, v, ls = stacked
        kv.kvec_evict_model_lse_steps(cfg, q, ls, k, v, bits, idx, ko, vo, ws)
    else:
        q, k, v = stacked
        kv.kvec_evict_model_steps(cfg, q, k, v, bits, idx, ko, vo, ws)
    torch.cuda.synchronize()
    for s in range(n_steps):
        b1, i1, k1, v1 = (x[0] for x in _outs(kv, w0, 1))
        if lse:
            kv.kvec_evict_model_lse(cfg, ins[s][0], ins[s][3], ins[s][1], ins[s][2], b1, i1, k1, v1, ws)
        else:
            kv.kvec_evict_model(cfg, ins[s][0], ins[s][1], ins[s][2], b1, i1, k1, v1, ws)
        torch.cuda.synchronize()
        assert torch.equal(bits[s], b1), f"step {s}: bitmap rows differ"
        assert torch.equal(idx[s], i1), f"step {s}: indices differ"
        assert torch.equal(ko[s].view(torch.int16), k1.view(torch.int16)), f"step {s}: K differs"
        assert torch.equal(vo[s].view(torch.int16), v1.view(torch.int16)), f"step {s}: V differs"
        assert int((i1 >= 0).sum()) > 0


@pytest.mark.parametrize("L", [4, 13])
def test_steps_match_single_calls(gpu_lib, L):
    n = 3
    _say(f"[steps] L={L} n={n}, distinct inputs")
    _check(gpu_lib, [_wl(L, 40 + s) for s in range(n)], n, shared=False)


def test_steps_shared_prefill(gpu_lib):
    _say("[steps] L=6 n=4, step stride 0")
    _check(gpu_lib, [_wl(6, 50)], 4, shared=True)


def test_steps_keep_everything(gpu_lib):
    _say("[steps] T <= B: keep everything")
    w = _wl(3, 60, T=150, B=200)
    _check(gpu_lib, [w, _wl(3, 61, T=150, B=200)], 2, shared=False)


@pytest.mark.parametrize("L", [3, 10])
def test_lse_steps_match_single_calls(gpu_lib, L):
    n = 3
    _say(f"[steps-lse] L={L} n={n}, distinct inputs and normalisers")
    _check(gpu_lib, [_wl(L, 70 + s) for s in range(n)], n, shared=False, lse=True)


def test_lse_steps_shared_prefill(gpu_lib):
    _say("[steps-lse] L=5 n=3, step stride 0")
    _check(gpu_lib, [_wl(5, 80)], 3, shared=True, lse=True)


def test_lse_steps_keep_everything(gpu_lib):
    _say("[steps-lse] T <= B: keep everything")
    _check(gpu_lib, [_wl(2, 90, T=150, B=200), _wl(2, 91, T=150, B=200)], 2, shared=False, lse=True)
