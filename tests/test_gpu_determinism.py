"""Run-twice determinism of the GPU path, through the C ABI.

Every entry point runs twice on the same inputs with its workspace refilled
with a different byte pattern before each run (zeros, then 0xA5).  The
outputs must be bit-identical: no result may depend on the order in which
work-groups finish or on what an earlier call left in the scratch memory
(the library keeps no state between calls).
"""
import sys

import numpy as np
import pytest

import synth
from kvec_testlib import model_tensors, layer_inputs

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _wl(T=3000, layers=4, batch=2, H=8, G=4, d=128, dtype="bf16", O=32, Wn=64, B=256):
    return synth.Workload(f"det-{dtype}-T{T}", layers, H, H * G, d, T, batch, O, Wn, B, 7, dtype, 23,
                          rope=True, hh_count=T // 50, n_adjust_heads=3)


def _bits(t):
    import torch
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16)
    if t.dtype == torch.float32:
        return t.view(torch.int32)
    return t


def _same(a, b, what):
    import torch
    assert torch.equal(_bits(a), _bits(b)), f"{what} differs between two runs"


@pytest.mark.parametrize("lse", [False, True], ids=["two-pass", "given-lse"])
def test_model_step_twice(gpu_lib, lse):
    import torch
    kv = gpu_lib
    w = _wl()
    _say(f"[det] model step {w.name} L={w.n_layers} b={w.batch} lse={lse}")
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    q, k, v = model_tensors(w)
    L, H, B, T, d = w.n_layers, w.n_kv_heads, w.budget, w.seq_len, w.head_dim
    lse_t = None
    if lse:
        # any fixed normalisers serve for determinism: log-sum-exp of the
        # window rows' logits in float32
        qf = q.float()
        kf = k.float().repeat_interleave(w.group, dim=2)
        s = torch.matmul(qf, kf.transpose(-1, -2).contiguous()) / np.sqrt(d)
        pos = torch.arange(T, device="cuda")
        rows = T - w.rows + torch.arange(w.rows, device="cuda")
        s = s.masked_fill(pos[None, :] > rows[:, None], float("-inf"))
        lse_t = torch.logsumexp(s, dim=-1).contiguous()
    outs = []
    for fill in (0x00, 0xA5):
        ws.fill_(fill)
        bits = torch.empty((w.batch, L, (T + 63) // 64), dtype=torch.int64, device="cuda")
        idx = torch.empty((L, w.batch, H, B), dtype=torch.int32, device="cuda")
        ko = torch.empty((L, w.batch, H, B, d), dtype=k.dtype, device="cuda")
        vo = torch.empty_like(ko)
        if lse:
            kv.kvec_evict_model_lse(cfg, q, lse_t, k, v, bits, idx, ko, vo, ws)
        else:
            kv.kvec_evict_model(cfg, q, k, v, bits, idx, ko, vo, ws)
        torch.cuda.synchronize()
        outs.append((bits, idx, ko, vo))
    for name, a, b in zip(("bitmap rows", "indices", "K cache", "V cache"), outs[0], outs[1]):
        _same(a, b, name)
    assert int((outs[0][1] >= 0).sum()) > 0


@pytest.mark.parametrize("dtype,T", [("bf16", 2999), ("f32", 1500)])
def test_scores_twice(gpu_lib, dtype, T):
    import torch
    kv = gpu_lib
    w = _wl(T=T, layers=1, batch=2, G=2 if dtype == "f32" else 4, d=128 if dtype == "bf16" else 64,
            dtype=dtype)
    _say(f"[det] scores {w.name}")
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    q, k, _ = model_tensors(w)
    q, k = q[0].contiguous(), k[0].contiguous()
    outs = []
    for fill in (0x00, 0xA5):
        ws.fill_(fill)
        p = torch.empty((w.batch, w.n_kv_heads, w.candidates), dtype=torch.float32, device="cuda")
        pe = torch.empty_like(p)
        imp = torch.empty((w.batch, w.candidates), dtype=torch.float32, device="cuda")
        kv.kvec_score(cfg, q, k, p, pe, imp, ws)
        torch.cuda.synchronize()
        outs.append((p, pe, imp))
    for name, a, b in zip(("P", "P over O'", "I"), outs[0], outs[1]):
        _same(a, b, name)


def test_decode_twice(gpu_lib):
    import torch
    kv = gpu_lib
    g = torch.Generator().manual_seed(3)
    w = _wl(T=4096, layers=1, batch=2, B=1024)
    cfg = kv.Config.from_workload(w)
    n_ctx = 1100
    _say(f"[det] decode b={w.batch} H={w.n_kv_heads} n_ctx={n_ctx}")
    q = torch.randn((w.batch, w.n_q_heads, w.head_dim), generator=g).to(torch.bfloat16).cuda()
    kc = torch.randn((w.batch, w.n_kv_heads, n_ctx, w.head_dim), generator=g).to(torch.bfloat16).cuda()
    vc = torch.randn_like(kc.float().cpu()).to(torch.bfloat16).cuda()
    idx = torch.randint(-1, w.seq_len, (w.batch, w.n_kv_heads, w.budget), generator=g,
                        dtype=torch.int32).cuda()
    ws = torch.empty(kv.kvec_decode_workspace_size(cfg, n_ctx), dtype=torch.uint8, device="cuda")
    outs = []
    for fill in (0x00, 0xA5):
        ws.fill_(fill)
        out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
        kv.kvec_decode_attention(cfg, q, kc, vc, out, ws, idx=idx)
        torch.cuda.synchronize()
        outs.append(out)
    _same(outs[0], outs[1], "decode output")
