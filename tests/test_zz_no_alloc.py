"""kvec_decode_attention_noalloc (the allocation-free decode entry point)
against kvec_decode_attention, through the C ABI, on several calls in a row
(each reuses the library's fixed scratch that the calls before it left
behind; the second call is smaller than the first), and against the float64
oracle."""
import sys

import numpy as np
import pytest

import oracle as orc

pytestmark = pytest.mark.gpu
DEC_TOL = 1e-4  # |out - oracle| <= DEC_TOL * max|V|, as for kvec_decode_attention


def _cfg(kv, batch, H, G, d, dtype):
    return kv.Config(batch=batch, n_layers=32, n_kv_heads=H, n_q_heads=H * G, head_dim=d,
                     seq_len=32768, window=32, window_ext=64, budget=1024,
                     n_adjust_heads=min(3, H), dtype=dtype)


def _case(kv, batch, H, G, d, n_ctx, seed):
    import torch
    g = torch.Generator().manual_seed(seed)
    dt = torch.bfloat16
    cfg = _cfg(kv, batch, H, G, d, kv.KVEC_BF16)
    q = torch.randn((batch, H * G, d), generator=g).to(dt).cuda()
    kc = torch.randn((batch, H, n_ctx, d), generator=g).to(dt).cuda()
    vc = torch.randn((batch, H, n_ctx, d), generator=g).to(dt).cuda()
    idx = torch.randint(-1, 32768, (batch, H, cfg.budget), generator=g, dtype=torch.int32).cuda()
    ws = torch.empty(kv.kvec_decode_workspace_size(cfg, n_ctx), dtype=torch.uint8, device="cuda")
    ref = torch.full((batch, H * G, d), float("nan"), dtype=torch.float32, device="cuda")
    out = torch.full_like(ref, float("nan"))
    kv.kvec_decode_attention(cfg, q, kc, vc, ref, ws, idx=idx)
    kv.kvec_decode_attention_noalloc(cfg, q, kc, vc, out, idx=idx)
    torch.cuda.synchronize()
    assert torch.equal(out, ref), float((out - ref).abs().max())
    # and the oracle, on the same bytes
    got = out.cpu().numpy()
    qn = q.float().cpu().numpy().astype(np.float64)
    kn = kc.float().cpu().numpy().astype(np.float64)
    vn = vc.float().cpu().numpy().astype(np.float64)
    ii = idx.cpu().numpy()
    for s in range(batch):
        valid = np.ones((H, n_ctx), bool)
        valid[:, :cfg.budget] = ii[s] >= 0
        want = orc.decode_attention(qn[s], kn[s], vn[s], valid)
        assert np.max(np.abs(got[s] - want)) <= DEC_TOL * np.max(np.abs(vn[s]))
    print(f"   batch {batch} H {H} G {G} d {d} n_ctx {n_ctx}: equal to kvec_decode_attention",
          file=sys.stderr, flush=True)


def test_noalloc_decode_matches_workspace_entry(gpu_lib):
    kv = gpu_lib
    _case(kv, 3, 8, 4, 128, 1500, 1)   # larger first
    _case(kv, 1, 4, 7, 128, 1030, 2)   # then smaller, on the same scratch
    _case(kv, 2, 2, 2, 64, 1024, 3)


def test_noalloc_decode_many_chunks_and_repeats(gpu_lib):
    """One KV head over 4096 rows: 64 chunks, so the combine takes its
    two-pass order (more chunks than one batch of loads); the same call three
    times on the scratch the last one left behind."""
    kv = gpu_lib
    for rep in range(3):
        _case(kv, 1, 1, 8, 128, 4096, 4)
    _case(kv, 2, 1, 1, 64, 1024, 5)


def test_noalloc_decode_rejects_plans_beyond_its_scratch(gpu_lib):
    import torch
    kv = gpu_lib
    # 256 sequences x 8 KV heads: one chunk each, 256 x 32 x 130 floats > 4 MiB
    cfg = _cfg(kv, 256, 8, 4, 128, kv.KVEC_BF16)
    assert kv.kvec_decode_workspace_size(cfg, 1024) > 4 << 20
    q = torch.zeros((256, 32, 128), dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros((256, 8, 1024, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((256, 32, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(kv.KvecError) as e:
        kv.kvec_decode_attention_noalloc(cfg, q, kc, kc, out)
    assert e.value.status == kv.KVEC_ERR_WORKSPACE
