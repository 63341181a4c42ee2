"""GPU parity of kvec_decode_attention (a decode token's attention over the
compacted cache) against the float64 oracle, through the C ABI.

Bar: |out - oracle| <= 1e-4 * max|V| element-wise (fp32 accumulation of a
convex combination of the V rows; the inputs are exact on both sides)."""
import sys

import numpy as np
import pytest

import oracle as orc
import synth
from kvec_testlib import model_tensors
from test_gpu_parity import _small

pytestmark = pytest.mark.gpu
DEC_TOL = 1e-4


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _f64(t):
    import torch
    return t.float().cpu().numpy().astype(np.float64) if t.dtype == torch.bfloat16 else \
        t.cpu().numpy().astype(np.float64)


def _check(kv, cfg, q, kc, vc, n_ctx=None, idx=None):
    import torch
    b, hq, d = q.shape
    n = kc.shape[2] if n_ctx is None else n_ctx
    ws = torch.empty(max(kv.kvec_decode_workspace_size(cfg, n), 16), dtype=torch.uint8,
                     device="cuda")
    out = torch.full((b, hq, d), float("nan"), dtype=torch.float32, device="cuda")
    kv.kvec_decode_attention(cfg, q, kc, vc, out, ws, idx=idx, n_ctx=n)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    qn, kn, vn = _f64(q), _f64(kc[:, :, :n]), _f64(vc[:, :, :n])
    ii = None if idx is None else idx.cpu().numpy()
    for s in range(b):
        valid = None
        if ii is not None:
            valid = np.ones((kn.shape[1], n), bool)
            valid[:, :ii.shape[2]] = ii[s] >= 0
        want = orc.decode_attention(qn[s], kn[s], vn[s], valid)
        err = np.max(np.abs(got[s] - want))
        scale = max(np.max(np.abs(vn[s])), 1e-30)
        _say(f"   seq {s}: max abs err {err:.2e} (V scale {scale:.2f})")
        assert err <= DEC_TOL * scale, err


CASES = [  # (H, G, d, n_ctx, batch, dtype)
    (8, 4, 128, 1024, 1, "bf16"),       # the 32k workload's cache shape, B = 1024
    (4, 7, 128, 1024, 1, "bf16"),       # Qwen2.5-7B grouping
    (8, 8, 64, 300, 3, "bf16"),
    (2, 1, 64, 77, 2, "f32"),
    (4, 3, 128, 2048, 1, "f32"),
    (1, 5, 128, 5000, 2, "bf16"),
]


@pytest.mark.parametrize("H,G,d,n,batch,dt", CASES,
                         ids=[f"h{c[0]}-g{c[1]}-d{c[2]}-n{c[3]}-b{c[4]}-{c[5]}" for c in CASES])
def test_decode_random_cache(gpu_lib, H, G, d, n, batch, dt):
    import torch
    kv = gpu_lib
    _say(f"[decode] H={H} G={G} d={d} n={n} batch={batch} {dt}")
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    cfg = kv.Config(batch=batch, n_layers=1, n_kv_heads=H, n_q_heads=H * G, head_dim=d,
                    seq_len=max(n, 64), window=32, window_ext=64, budget=min(n, 1024),
                    n_adjust_heads=min(3, H), dtype=kv.KVEC_BF16 if dt == "bf16" else kv.KVEC_F32)
    g = torch.Generator().manual_seed(1000 * H + 10 * G + d + n)
    q = (torch.randn((batch, H * G, d), generator=g) * 2).to(tdt).cuda()
    kc = (torch.randn((batch, H, n, d), generator=g) * 2).to(tdt).cuda()
    vc = torch.randn((batch, H, n, d), generator=g).to(tdt).cuda()
    _check(kv, cfg, q, kc, vc)


def test_decode_after_eviction_with_appended_rows(gpu_lib):
    """The compacted cache of a real eviction step (kvec_evict_model), copied
    into a larger buffer with 37 decode tokens appended after the B kept rows."""
    import torch
    kv = gpu_lib
    w = _small("decode-e2e", 2000, 32, 64, 4, 4, 128, "bf16", batch=2, B=160, layers=2)
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    q, k, v = model_tensors(w)
    L, H, B, T, d = w.n_layers, w.n_kv_heads, w.budget, w.seq_len, w.head_dim
    bits = torch.empty((w.batch, L, (T + 63) // 64), dtype=torch.int64, device="cuda")
    idx = torch.empty((L, w.batch, H, B), dtype=torch.int32, device="cuda")
    ko = torch.empty((L, w.batch, H, B, d), dtype=k.dtype, device="cuda")
    vo = torch.empty_like(ko)
    kv.kvec_evict_model(cfg, q, k, v, bits, idx, ko, vo, ws)
    extra = 37
    g = torch.Generator().manual_seed(5)
    kc = torch.empty((w.batch, H, B + extra + 11, d), dtype=k.dtype, device="cuda")
    vc = torch.empty_like(kc)
    kc[:, :, :B] = ko[1]
    vc[:, :, :B] = vo[1]
    kc[:, :, B:] = torch.randn(kc[:, :, B:].shape, generator=g).to(k.dtype).cuda()
    vc[:, :, B:] = torch.randn(vc[:, :, B:].shape, generator=g).to(k.dtype).cuda()
    qd = (torch.randn((w.batch, w.n_q_heads, d), generator=g) * 2).to(k.dtype).cuda()
    _check(kv, cfg, qd, kc, vc, n_ctx=B + extra, idx=idx[1])


def test_decode_masks_padding_when_everything_is_kept(gpu_lib):
    """T <= B: kvec_compact pads with zero rows (idx -1) that decode must skip."""
    import torch
    kv = gpu_lib
    w = _small("decode-keep-all", 100, 8, 16, 2, 2, 64, "bf16", B=128, layers=1)
    cfg = kv.Config.from_workload(w)
    q, k, v = model_tensors(w)
    ws = torch.empty(max(kv.kvec_workspace_size(cfg), 256), dtype=torch.uint8, device="cuda")
    bits = torch.zeros((1, 1, 2), dtype=torch.int64, device="cuda")
    idx = torch.empty((1, 1, 2, 128), dtype=torch.int32, device="cuda")
    ko = torch.empty((1, 1, 2, 128, 64), dtype=k.dtype, device="cuda")
    vo = torch.empty_like(ko)
    kv.kvec_evict_model(cfg, q, k, v, bits, idx, ko, vo, ws)
    g = torch.Generator().manual_seed(6)
    qd = (torch.randn((1, 4, 64), generator=g) * 3).to(k.dtype).cuda()
    _check(kv, cfg, qd, ko[0], vo[0], idx=idx[0])
