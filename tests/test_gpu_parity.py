"""GPU parity of libkvec against the float64 oracle, through the C ABI.

Scores: max relative error <= 2e-3.  Selection on oracle scores: bit-exact
indices, H_top and bitmaps.  Gather: byte-exact.  End to end: teacher-forced
agreement >= 99.5% with every mismatch within tolerance of the cut.
"""
import sys

import numpy as np
import pytest

import oracle as orc
import synth
from kvec_testlib import (AGREE_MIN, SCORE_RTOL, agreement, bits_to_bool, counts_before,
                          layer_inputs, model_tensors, oracle_scores, rel_err, to_device)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _small(name, T, O, Wn, H, G, D, dtype, batch=1, B=None, layers=2, pool=7, delta=3, lam=1.0,
           beta=0.25, hh=0.02, rope=True, seed=7, criterion="std"):
    B = B if B is not None else max(O + 8, T // 8)
    return synth.Workload(name, layers, H, H * G, D, T, batch, O, Wn, B, pool, dtype, seed,
                          rope=rope, hh_count=int(round(hh * T)), n_adjust_heads=min(delta, H),
                          lam=lam, beta=beta, criterion=criterion)


SCORE_CASES = [
    _small("f32-d64-g2", 1024, 32, 64, 4, 2, 64, "f32", rope=False),
    _small("f32-d64-g2-ragged", 301, 32, 64, 4, 2, 64, "f32", rope=False),
    _small("bf16-d128-g4", 1000, 32, 64, 8, 4, 128, "bf16"),
    _small("bf16-d128-g4-mixed", 777, 20, 40, 2, 4, 128, "bf16"),
    _small("bf16-d64-g1-pad", 530, 20, 40, 2, 1, 64, "bf16"),
    _small("bf16-d128-g2-h1", 3001, 24, 48, 1, 2, 128, "bf16"),
    _small("bf16-d128-g4-o64", 2048, 64, 128, 8, 4, 128, "bf16", batch=2),
    _small("bf16-d128-g8", 257, 5, 17, 2, 8, 128, "bf16"),
    _small("bf16-d64-g2-short", 70, 16, 64, 2, 2, 64, "bf16"),
    _small("f32-d128-g1", 200, 8, 8, 2, 1, 128, "f32"),
    _small("bf16-d128-g4-wn-eq-o", 600, 32, 32, 4, 4, 128, "bf16"),
    # the longest supported prefix (T = 2^18), one KV head
    _small("bf16-d64-g1-max-T", 1 << 18, 32, 64, 1, 1, 64, "bf16", B=2048),
    # key tiles of 256 (8192 <= T < 16384; shorter prefixes use 128, longer 512)
    _small("bf16-d128-g4-tile256", 9000, 32, 64, 8, 4, 128, "bf16"),
    # group sizes that are not powers of two (Qwen2.5: 7 for 7B, 5 for 14B/32B, 6 for 1.5B)
    _small("bf16-d128-g7-h4", 1500, 32, 64, 4, 7, 128, "bf16"),
    _small("bf16-d64-g3-ragged", 611, 12, 24, 2, 3, 64, "bf16"),
    _small("bf16-d128-g5-h8", 800, 16, 32, 8, 5, 128, "bf16"),
    _small("f32-d128-g6-h2", 500, 20, 40, 2, 6, 128, "f32"),
]


@pytest.mark.parametrize("w", SCORE_CASES, ids=lambda w: w.name)
def test_score_parity(gpu_lib, w):
    import torch
    kv = gpu_lib
    _say(f"[score] {w.name} T={w.seq_len} O={w.window} Wn={w.rows} H={w.n_kv_heads} G={w.group}")
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    Tc = w.candidates
    for layer in range(min(w.n_layers, 2)):
        qs, ks = [], []
        for b in range(w.batch):
            qa, ka, _ = layer_inputs(w, layer, b)
            qs.append(to_device(qa, w))
            ks.append(to_device(ka, w))
        q = torch.stack(qs)
        k = torch.stack(ks)
        p = torch.empty((w.batch, w.n_kv_heads, Tc), dtype=torch.float32, device="cuda")
        pe = torch.empty_like(p)
        imp = torch.empty((w.batch, Tc), dtype=torch.float32, device="cuda")
        kv.kvec_score(cfg, q, k, p, pe, imp, ws)
        torch.cuda.synchronize()
        for b in range(w.batch):
            rp, rpe, rimp = oracle_scores(w, layer, b)
            e = (rel_err(p[b].cpu().numpy(), rp), rel_err(pe[b].cpu().numpy(), rpe),
                 rel_err(imp[b].cpu().numpy(), rimp))
            _say(f"   layer {layer} seq {b}: rel err P {e[0]:.2e} P' {e[1]:.2e} I {e[2]:.2e}")
            assert max(e) <= SCORE_RTOL, e


SELECT_CASES = [
    _small("sel-base", 4096, 32, 64, 8, 4, 128, "bf16", B=128, layers=4),
    _small("sel-b2-pool5", 3000, 64, 128, 4, 4, 128, "bf16", batch=2, B=300, layers=3, pool=5),
    _small("sel-pool1-nodelta", 1500, 16, 32, 4, 2, 64, "bf16", B=100, layers=3, pool=1, delta=0),
    _small("sel-lam0", 1500, 16, 32, 4, 2, 64, "bf16", B=100, layers=3, lam=0.0),
    _small("sel-beta0", 1500, 16, 32, 4, 2, 64, "bf16", B=100, layers=3, beta=0.0),
    _small("sel-beta1", 1500, 16, 32, 4, 2, 64, "bf16", B=100, layers=3, beta=1.0),
    _small("sel-wn-eq-o", 1500, 16, 16, 4, 2, 64, "bf16", B=100, layers=3),
    _small("sel-ragged", 999, 7, 14, 2, 1, 64, "bf16", B=41, layers=3, pool=3),
    _small("sel-long", 20000, 32, 64, 8, 4, 128, "bf16", B=700, layers=3),
    # the entropy criterion of the head-selection ablation
    _small("sel-entropy", 4096, 32, 64, 8, 4, 128, "bf16", B=128, layers=4, criterion="entropy"),
    _small("sel-entropy-b2-d2", 3000, 64, 128, 4, 4, 128, "bf16", batch=2, B=300, layers=3,
           pool=5, delta=2, criterion="entropy"),
]


@pytest.mark.parametrize("w", SELECT_CASES, ids=lambda w: w.name)
def test_select_on_oracle_scores(gpu_lib, w):
    """Selection fed the oracle's fp32 scores is bit-exact with the oracle."""
    import torch
    kv = gpu_lib
    _say(f"[select] {w.name} T={w.seq_len} B={w.budget} layers={w.n_layers} batch={w.batch}")
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    T, Tc, H, B = w.seq_len, w.candidates, w.n_kv_heads, w.budget
    W = (T + 63) // 64
    bits = torch.zeros((w.batch, w.n_layers, W), dtype=torch.int64, device="cuda")
    idx = torch.empty((w.batch, H, B), dtype=torch.int32, device="cuda")
    htop = torch.empty((w.batch,), dtype=torch.int32, device="cuda")
    prev = [[] for _ in range(w.batch)]
    for layer in range(w.n_layers):
        sc = [orc.score_layer(synth.to_f64(synth.queries(w, layer, b), w.dtype),
                              synth.to_f64(synth.keys(w, layer, b), w.dtype), w.window)
              for b in range(w.batch)]
        p = torch.from_numpy(np.stack([s[0] for s in sc])).cuda()
        pe = torch.from_numpy(np.stack([s[1] for s in sc])).cuda()
        imp = torch.from_numpy(np.stack([s[2] for s in sc])).cuda()
        kv.kvec_select_cover(cfg, layer, p, pe, imp, bits, idx, htop, ws)
        torch.cuda.synchronize()
        gi = idx.cpu().numpy()
        gb = bits.cpu().numpy().view(np.uint64)
        gh = htop.cpu().numpy()
        for b in range(w.batch):
            n_t = orc.counts_from_bits(prev[b]) if prev[b] else np.zeros(T, np.int64)
            res = orc.evict_layer_from_scores(sc[b][0], sc[b][1], sc[b][2], n_t, layer, w)
            np.testing.assert_array_equal(gi[b], res.idx, err_msg=f"layer {layer} seq {b}")
            want_mask = sum(1 << int(h) for h in res.htop)
            assert int(gh[b]) & 0xFFFF == want_mask, (layer, b, gh[b], res.htop)
            np.testing.assert_array_equal(bits_to_bool(gb[b, layer], T), res.bits)
            prev[b].append(res.bits)
        _say(f"   layer {layer}: idx, H_top and bitmap bit-exact")


def test_keep_everything_when_budget_covers(gpu_lib):
    import torch
    kv = gpu_lib
    w = _small("keep-all", 100, 8, 16, 2, 2, 64, "bf16", B=128, layers=2)
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(max(kv.kvec_workspace_size(cfg), 256), dtype=torch.uint8, device="cuda")
    q, k, v = model_tensors(w)
    W = (w.seq_len + 63) // 64
    bits = torch.zeros((1, 2, W), dtype=torch.int64, device="cuda")
    idx = torch.empty((2, 1, 2, 128), dtype=torch.int32, device="cuda")
    ko = torch.empty((2, 1, 2, 128, 64), dtype=k.dtype, device="cuda")
    vo = torch.empty_like(ko)
    kv.kvec_evict_model(cfg, q, k, v, bits, idx, ko, vo, ws)
    torch.cuda.synchronize()
    gi = idx.cpu().numpy()
    assert np.all(gi[:, :, :, :100] == np.arange(100))
    assert np.all(gi[:, :, :, 100:] == -1)
    assert np.all(ko[:, :, :, 100:].float().cpu().numpy() == 0)
    assert torch.equal(ko[:, :, :, :100], k)


def test_compact_bit_exact(gpu_lib):
    import torch
    kv = gpu_lib
    w = _small("compact", 500, 8, 16, 4, 2, 128, "bf16", batch=2, B=64, layers=1)
    cfg = kv.Config.from_workload(w)
    g = torch.Generator().manual_seed(3)
    k = torch.randn((2, 4, 500, 128), generator=g).to(torch.bfloat16).cuda()
    v = torch.randn((2, 4, 500, 128), generator=g).to(torch.bfloat16).cuda()
    idx = torch.randint(-1, 500, (2, 4, 64), generator=g, dtype=torch.int32).cuda()
    ko = torch.empty((2, 4, 64, 128), dtype=torch.bfloat16, device="cuda")
    vo = torch.empty_like(ko)
    kv.kvec_compact(cfg, k, v, idx, ko, vo)
    torch.cuda.synchronize()
    ki = idx.cpu().numpy()
    kn, vn = k.cpu().view(torch.int16).numpy(), v.cpu().view(torch.int16).numpy()
    want_k = np.stack([orc.gather_rows(kn[b], ki[b]) for b in range(2)])
    want_v = np.stack([orc.gather_rows(vn[b], ki[b]) for b in range(2)])
    np.testing.assert_array_equal(ko.cpu().view(torch.int16).numpy(), want_k)
    np.testing.assert_array_equal(vo.cpu().view(torch.int16).numpy(), want_v)


def oracle_lse_tensor(w):
    """The oracle's window-row normalisers of every (layer, sequence), rounded to
    fp32, on the device: [L][b][HQ][Wn] (what a prefill attention would hand over)."""
    import torch
    out = np.empty((w.n_layers, w.batch, w.n_q_heads, w.rows), dtype=np.float32)
    for l in range(w.n_layers):
        for b in range(w.batch):
            out[l, b] = orc.to_f32(orc.window_lse(synth.to_f64(synth.queries(w, l, b), w.dtype),
                                                  synth.to_f64(synth.keys(w, l, b), w.dtype)))
    return torch.from_numpy(out).cuda()


def _e2e(kv, w, check_layers=None, lse=False, scores=None, same_as_model=False):
    """Run the whole-model driver and check layers teacher-forced (the oracle's
    layer l uses the device's bitmap rows of layers < l).

    The driver is kvec_evict_model_lse on the oracle's row normalisers when
    lse=True; else kvec_evict_model_scores (scores=True, the default), whose
    per-layer P, P over O' of the H_top heads and I are then compared element
    by element with the oracle at SCORE_RTOL, or kvec_evict_model.  With
    same_as_model=True kvec_evict_model also runs and must give bit-identical
    indices, bitmaps and caches (the scores variant runs the same pipeline)."""
    import torch
    scores = (not lse) if scores is None else scores
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    _say(f"[e2e] {w.name}{' (given lse)' if lse else ''}: generating inputs")
    q, k, v = model_tensors(w)
    L, H, B, T, d = w.n_layers, w.n_kv_heads, w.budget, w.seq_len, w.head_dim
    Tc = w.candidates
    W = (T + 63) // 64
    bits = torch.empty((w.batch, L, W), dtype=torch.int64, device="cuda")
    idx = torch.empty((L, w.batch, H, B), dtype=torch.int32, device="cuda")
    ko = torch.empty((L, w.batch, H, B, d), dtype=k.dtype, device="cuda")
    vo = torch.empty_like(ko)
    if lse:
        kv.kvec_evict_model_lse(cfg, q, oracle_lse_tensor(w), k, v, bits, idx, ko, vo, ws)
    elif scores:
        sp = torch.full((L, w.batch, H, Tc), float("nan"), dtype=torch.float32, device="cuda")
        spe = torch.full_like(sp, float("nan"))
        simp = torch.full((L, w.batch, Tc), float("nan"), dtype=torch.float32, device="cuda")
        shtop = torch.zeros((L, w.batch), dtype=torch.int32, device="cuda")
        kv.kvec_evict_model_scores(cfg, q, k, v, bits, idx, ko, vo, sp, spe, simp, shtop, ws)
    else:
        kv.kvec_evict_model(cfg, q, k, v, bits, idx, ko, vo, ws)
    torch.cuda.synchronize()
    _say(f"[e2e] {w.name}: device step done")
    if same_as_model:
        bits2, idx2 = torch.empty_like(bits), torch.empty_like(idx)
        ko2, vo2 = torch.empty_like(ko), torch.empty_like(vo)
        kv.kvec_evict_model(cfg, q, k, v, bits2, idx2, ko2, vo2, ws)
        torch.cuda.synchronize()
        raw = torch.int16 if k.dtype == torch.bfloat16 else torch.int32
        assert torch.equal(idx, idx2) and torch.equal(bits, bits2)
        assert torch.equal(ko.view(raw), ko2.view(raw)) and torch.equal(vo.view(raw), vo2.view(raw))
        _say("   kvec_evict_model gives the same indices, bitmaps and caches")
    gi = idx.cpu().numpy()
    gb = bits.cpu().numpy().view(np.uint64)
    if scores and not lse:
        gp, gpe, gimp, ght = (sp.cpu().numpy(), spe.cpu().numpy(), simp.cpu().numpy(),
                              shtop.cpu().numpy())
    ibits = torch.int16 if k.dtype == torch.bfloat16 else torch.int32
    M = B - w.window
    kp = orc.preserve_count(B, w.window, w.beta)
    layers = range(L) if check_layers is None else check_layers
    tot_m = tot = 0
    worst = 0.0
    cache = {}
    for l in layers:
        for b in range(w.batch):
            p, pe, imp = oracle_scores(w, l, b)
            if b == 0:
                cache[l] = (p, pe, imp)
            n_t = counts_before(gb[b], l, T)
            res = orc.evict_layer_from_scores(orc.to_f32(p), orc.to_f32(pe), orc.to_f32(imp),
                                              n_t, l, w)
            if scores and not lse:
                # the pipeline's own scores, element by element
                hs = [h for h in range(H) if (int(ght[l, b]) >> h) & 1]
                assert sorted(hs) == sorted(int(x) for x in res.htop), (l, b, hs, res.htop)
                e = [rel_err(gp[l, b], p), rel_err(gimp[l, b], imp)]
                if hs:
                    e.append(rel_err(gpe[l, b, hs], pe[hs]))
                worst = max(worst, max(e))
                assert max(e) <= SCORE_RTOL, (l, b, e)
            m, t, bad = agreement(gi[l, b], res, M, kp)
            tot_m += m
            tot += t
            assert not bad, f"layer {l} seq {b}: mismatches away from the cut {bad[:5]}"
            # the window, the layout and the bitmap row
            assert np.all(gi[l, b, :, M:] == np.arange(T - w.window, T))
            assert np.all(np.diff(gi[l, b, :, :M], axis=1) > 0)
            np.testing.assert_array_equal(bits_to_bool(gb[b, l], T),
                                          orc.layer_bits(gi[l, b], T))
            # gather of K and V is byte-exact for the GPU's own indices
            for src, out in ((k, ko), (v, vo)):
                xx = src[l, b].cpu().view(ibits).numpy()
                np.testing.assert_array_equal(out[l, b].cpu().view(ibits).numpy(),
                                              orc.gather_rows(xx, gi[l, b]))
        _say(f"   layer {l}: agreement so far {tot_m / tot:.5f}"
             + (f", worst score rel err {worst:.2e}" if scores and not lse else ""))
    assert tot_m / tot >= AGREE_MIN
    if check_layers is None and w.batch == 1:
        # free-running agreement (the oracle on its own bitmaps): reported only
        own, fm, ft = [], 0, 0
        for l in range(L):
            p, pe, imp = cache[l]
            n_t = orc.counts_from_bits(own) if own else np.zeros(T, np.int64)
            res = orc.evict_layer_from_scores(orc.to_f32(p), orc.to_f32(pe), orc.to_f32(imp),
                                              n_t, l, w)
            own.append(res.bits)
            for h in range(H):
                fm += len(set(gi[l, 0, h, :M].tolist()) & set(res.idx[h, :M].tolist()))
                ft += M
        _say(f"   free-running agreement (not gated): {fm / ft:.5f}")
    # coverage equals the union of the kept index sets
    cnt = torch.empty((w.batch,), dtype=torch.int64, device="cuda")
    kv.kvec_coverage(cfg, bits, L - 1, cnt)
    torch.cuda.synchronize()
    for b in range(w.batch):
        u = set()
        for l in range(L):
            u |= set(gi[l, b].ravel().tolist())
        u.discard(-1)
        assert int(cnt[b]) == len(u)


def test_e2e_tiny_fp32(gpu_lib):
    _e2e(gpu_lib, synth.workload(0))


def test_e2e_small_bf16(gpu_lib):
    _e2e(gpu_lib, _small("e2e-small", 2500, 32, 64, 8, 4, 128, "bf16", B=200, layers=6))


def test_e2e_max_prefix(gpu_lib):
    """The longest supported prefix, T = 2^18, two KV heads of group 2."""
    _e2e(gpu_lib, _small("e2e-max-T", 1 << 18, 32, 64, 2, 2, 64, "bf16", B=2048, layers=2))


def test_e2e_tile256_bf16(gpu_lib):
    _e2e(gpu_lib, _small("e2e-tile256", 10000, 32, 64, 8, 4, 128, "bf16", B=512, layers=3))


def test_e2e_entropy_bf16(gpu_lib):
    _e2e(gpu_lib, _small("e2e-entropy", 2500, 32, 64, 8, 4, 128, "bf16", B=200, layers=6,
                         criterion="entropy"))


def test_e2e_group7_bf16(gpu_lib):
    _e2e(gpu_lib, _small("e2e-g7", 3000, 32, 64, 4, 7, 128, "bf16", B=256, layers=4))


def test_layer_calls_match_model_step(gpu_lib):
    """kvec_evict_layer called layer by layer reproduces kvec_evict_model exactly."""
    import torch
    kv = gpu_lib
    w = _small("layerwise", 3000, 32, 64, 4, 4, 128, "bf16", batch=2, B=256, layers=5)
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    q, k, v = model_tensors(w)
    L, H, B, T, d = w.n_layers, w.n_kv_heads, w.budget, w.seq_len, w.head_dim
    W = (T + 63) // 64
    bits_m = torch.empty((w.batch, L, W), dtype=torch.int64, device="cuda")
    idx_m = torch.empty((L, w.batch, H, B), dtype=torch.int32, device="cuda")
    ko_m = torch.empty((L, w.batch, H, B, d), dtype=k.dtype, device="cuda")
    vo_m = torch.empty_like(ko_m)
    kv.kvec_evict_model(cfg, q, k, v, bits_m, idx_m, ko_m, vo_m, ws)
    bits_l = torch.zeros_like(bits_m)
    idx_l = torch.empty_like(idx_m)
    ko_l = torch.empty_like(ko_m)
    vo_l = torch.empty_like(vo_m)
    for l in range(L):
        kv.kvec_evict_layer(cfg, l, q[l], k[l], v[l], bits_l, idx_l[l], ko_l[l], vo_l[l], ws)
    torch.cuda.synchronize()
    assert torch.equal(idx_m, idx_l)
    assert torch.equal(bits_m, bits_l)
    assert torch.equal(ko_m.view(torch.int16), ko_l.view(torch.int16))
    assert torch.equal(vo_m.view(torch.int16), vo_l.view(torch.int16))


# ---------------------------------------------------------------------------
# Full-size workloads, run exactly as the benchmark runs them (kvec_evict_model
# over every layer with the library-sized workspace); the oracle checks every
# layer at 4k and sampled layers of the larger shapes, teacher-forced on the
# device's own bitmaps of the earlier layers.
# ---------------------------------------------------------------------------

def test_full_llama8b_4k_every_layer(gpu_lib):
    _e2e(gpu_lib, synth.workload(1))


def test_full_llama8b_32k_every_layer(gpu_lib):
    """The benchmarked workload: every layer's scores, indices, bitmaps and
    gathered K/V; kvec_evict_model must match the scores variant exactly."""
    _e2e(gpu_lib, synth.workload(2), same_as_model=True)


def test_full_llama8b_16k_batch8_layers(gpu_lib):
    _e2e(gpu_lib, synth.workload(3), check_layers=[0, 1, 2, 3, 15, 16, 30, 31])


def test_full_llama8b_128k_layers(gpu_lib):
    _e2e(gpu_lib, synth.workload(4), check_layers=list(range(0, 32, 4)) + [31])


def test_full_qwen7b_32k_sampled_layers(gpu_lib):
    """The Qwen2.5-7B shape (4 KV / 28 query heads, 28 layers) at 32k."""
    _e2e(gpu_lib, synth.workload(5), check_layers=[0, 1, 27])


@pytest.mark.parametrize("wi", [1, 2, 3, 4, 5], ids=["4k", "32k", "16k-b8", "128k", "qwen7b-32k"])
def test_full_size_scores(gpu_lib, wi):
    """kvec_score on one layer of a full-size shape against the oracle scores."""
    import torch
    kv = gpu_lib
    w = synth.workload(wi)
    w1 = w.with_(batch=1)
    cfg = kv.Config.from_workload(w1)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    layer = w.n_layers - 1
    qa, ka, _ = layer_inputs(w1, layer, 0)
    q = to_device(qa, w1)[None]
    k = to_device(ka, w1)[None]
    Tc = w1.candidates
    p = torch.empty((1, w1.n_kv_heads, Tc), dtype=torch.float32, device="cuda")
    pe = torch.empty_like(p)
    imp = torch.empty((1, Tc), dtype=torch.float32, device="cuda")
    kv.kvec_score(cfg, q, k, p, pe, imp, ws)
    torch.cuda.synchronize()
    rp, rpe, rimp = oracle_scores(w1, layer, 0, qa, ka)
    e = (rel_err(p[0].cpu().numpy(), rp), rel_err(pe[0].cpu().numpy(), rpe),
         rel_err(imp[0].cpu().numpy(), rimp))
    _say(f"[score] {w.name} layer {layer}: rel err P {e[0]:.2e} P' {e[1]:.2e} I {e[2]:.2e}")
    assert max(e) <= SCORE_RTOL, e


# ---------------------------------------------------------------------------
# Exact ties at scale and the exact row-normaliser fallback
# ---------------------------------------------------------------------------

def test_all_ties_member_spill(gpu_lib):
    """Zero queries: every logit is 0, so P[t] = (H_T - H_{T-O}) / O for every
    candidate t (the closed form the oracle pins) and every head, I equals P,
    and every ranking is decided by the tie rule alone (score descending, index
    ascending; lower head first for sigma).  With 12000 candidates all in one
    histogram bin the selection's member lists exceed what LDS holds and take
    the spill path.  Indices and bitmaps are compared bit-exactly with the
    oracle run free on its own bitmaps."""
    import torch
    kv = gpu_lib
    w = _small("all-ties", 12032, 32, 64, 2, 2, 64, "bf16", B=256, layers=3, delta=1)
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    L, H, B, T, d, Tc = w.n_layers, w.n_kv_heads, w.budget, w.seq_len, w.head_dim, w.candidates
    _, k, v = model_tensors(w)
    q = torch.zeros((L, 1, w.n_q_heads, w.rows, d), dtype=k.dtype, device="cuda")
    W = (T + 63) // 64
    bits = torch.empty((1, L, W), dtype=torch.int64, device="cuda")
    idx = torch.empty((L, 1, H, B), dtype=torch.int32, device="cuda")
    ko = torch.empty((L, 1, H, B, d), dtype=k.dtype, device="cuda")
    vo = torch.empty_like(ko)
    sp = torch.empty((L, 1, H, Tc), dtype=torch.float32, device="cuda")
    spe = torch.empty_like(sp)
    simp = torch.empty((L, 1, Tc), dtype=torch.float32, device="cuda")
    sht = torch.empty((L, 1), dtype=torch.int32, device="cuda")
    kv.kvec_evict_model_scores(cfg, q, k, v, bits, idx, ko, vo, sp, spe, simp, sht, ws)
    torch.cuda.synchronize()
    gi, gp = idx.cpu().numpy(), sp.cpu().numpy()
    gb = bits.cpu().numpy().view(np.uint64)
    qz = np.zeros((w.n_q_heads, w.rows, d))
    own = []
    for l in range(L):
        # the device's scores are one value for every candidate of every head
        assert np.all(gp[l] == gp[l, 0, 0, 0]), l
        kf = synth.to_f64(synth.keys(w, l, 0), w.dtype)
        p, pe, imp = orc.score_layer(qz, kf, w.window)
        assert rel_err(gp[l, 0], p) <= SCORE_RTOL
        n_t = orc.counts_from_bits(own) if own else np.zeros(T, np.int64)
        res = orc.evict_layer_from_scores(p, pe, imp, n_t, l, w)
        np.testing.assert_array_equal(gi[l, 0], res.idx, err_msg=f"layer {l}")
        np.testing.assert_array_equal(bits_to_bool(gb[0, l], T), res.bits)
        assert int(sht[l, 0]) == 1, int(sht[l, 0])          # sigma tie -> head 0
        own.append(res.bits)
        _say(f"   layer {l}: {Tc} tied candidates, indices bit-exact")


def _fallback_inputs(w):
    """Random bf16 window queries and keys with two planted pairs whose logit is
    200 (about 288 in base 2): window row Wn-1 with key 200 (in the second key
    tile of 128 but not among its first 16 keys, so that tile's running sum
    overflows past its block reference) and window row Wn-2 with key 3 (among
    the first 16 keys of the first tile, so that tile's block reference is huge
    and the other rows' sums underflow)."""
    g = np.random.default_rng(11)
    d, T, Wn = w.head_dim, w.seq_len, w.rows
    q = (0.5 * g.standard_normal((w.n_q_heads, Wn, d))).astype(np.float32)
    k = g.standard_normal((w.n_kv_heads, T, d)).astype(np.float32)
    q[:, Wn - 1] = 0.0
    q[:, Wn - 1, 0] = 40.0
    k[:, 200] = 0.0
    k[:, 200, 0] = 40.0
    q[:, Wn - 2] = 0.0
    q[:, Wn - 2, 1] = 40.0
    k[:, 3] = 0.0
    k[:, 3, 1] = 40.0
    # bf16 storage by truncation (any bf16 values serve; 40 and 0 are exact)
    qb = (q.view(np.uint32) >> 16).astype(np.uint16)
    kb = (k.view(np.uint32) >> 16).astype(np.uint16)
    return qb, kb


def test_score_exact_normaliser_fallback(gpu_lib):
    """Key tiles whose partial sums leave the fp32 range of the fast path are
    recomputed exactly by the row-normaliser stage; the scores still match the
    oracle (both through kvec_score and through the pipeline)."""
    import torch
    kv = gpu_lib
    w = _small("fallback", 600, 8, 16, 1, 1, 64, "bf16", B=64, layers=2, hh=0.0)
    cfg = kv.Config.from_workload(w)
    ws = torch.empty(kv.kvec_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    qb, kb = _fallback_inputs(w)
    ref = orc.window_scores(synth.to_f64(qb, "bf16"), synth.to_f64(kb, "bf16"), w.window)
    q, k = to_device(qb, w)[None], to_device(kb, w)[None]
    Tc = w.candidates
    p = torch.empty((1, 1, Tc), dtype=torch.float32, device="cuda")
    pe, imp = torch.empty_like(p), torch.empty((1, Tc), dtype=torch.float32, device="cuda")
    kv.kvec_score(cfg, q, k, p, pe, imp, ws)
    torch.cuda.synchronize()
    e = (rel_err(p[0].cpu().numpy(), ref[0]), rel_err(pe[0].cpu().numpy(), ref[1]),
         rel_err(imp[0].cpu().numpy(), ref[2]))
    _say(f"   kvec_score: rel err P {e[0]:.2e} P' {e[1]:.2e} I {e[2]:.2e}")
    assert max(e) <= SCORE_RTOL, e
    # the two planted keys take nearly all of their rows' attention
    assert p[0, 0, 200] > 0.1 and p[0, 0, 3] > 0.1
    # the same inputs in both layers of the pipeline
    L = w.n_layers
    qq, kk = q[None].expand(L, -1, -1, -1, -1), k[None].expand(L, -1, -1, -1, -1)
    vv = torch.zeros_like(kk)
    bits = torch.empty((1, L, (w.seq_len + 63) // 64), dtype=torch.int64, device="cuda")
    idx = torch.empty((L, 1, 1, w.budget), dtype=torch.int32, device="cuda")
    ko = torch.empty((L, 1, 1, w.budget, w.head_dim), dtype=k.dtype, device="cuda")
    vo = torch.empty_like(ko)
    sp = torch.empty((L, 1, 1, Tc), dtype=torch.float32, device="cuda")
    spe = torch.empty_like(sp)
    simp = torch.empty((L, 1, Tc), dtype=torch.float32, device="cuda")
    sht = torch.empty((L, 1), dtype=torch.int32, device="cuda")
    kv.kvec_evict_model_scores(cfg, qq, kk, vv, bits, idx, ko, vo, sp, spe, simp, sht, ws)
    torch.cuda.synchronize()
    for l in range(L):
        e = [rel_err(sp[l, 0].cpu().numpy(), ref[0]), rel_err(simp[l, 0].cpu().numpy(), ref[2])]
        if int(sht[l, 0]) & 1:
            e.append(rel_err(spe[l, 0].cpu().numpy(), ref[1]))
        assert max(e) <= SCORE_RTOL, (l, e)
