"""GPU parity of every step against the CPU oracle, through the C ABI.

Indices bit-exact; routing weights within 1e-6 relative; expert and combined
outputs per row/token normwise within 1e-2 (bf16) or 3e-2 (fp8).  Small shapes span several
tiles and ragged tails; the full-size configurations are checked on every
index and on sampled tokens the oracle evaluates one by one."""
import ctypes as C
import json
import os

import numpy as np
import pytest

import oracle
from _helpers import BF16_TOL, FP8_TOL, layer_specs, normwise_rel_err
from workload import CONFIGS, bf16_bits, custom_config, make_layer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_18002_amd import load_library
    load_library()
    return torch.device("cuda:0")


def _route(dev, L, k, lb, El):
    from paper_2607_18002_amd import ops
    ids, w = ops.moe_topk_route(torch.from_numpy(L).to(dev), k, lb, El)
    torch.cuda.synchronize()
    return ids.cpu().numpy(), w.cpu().numpy()


# ----------------------------------------------------------------------------- a1 routing
@pytest.mark.parametrize("T,E,k", [(1, 8, 2), (257, 8, 2), (130, 64, 8), (77, 65, 3), (513, 256, 8),
                                   (33, 1000, 32), (19, 16, 16), (5, 3, 1)])
def test_route_random(dev, T, E, k):
    rng = np.random.default_rng(T * 7 + E)
    L = (rng.standard_normal((T, E)) * 2).astype(np.float32)
    for lb, El in [(0, E), (1, max(1, E // 4)), (E - 1, 1)]:
        ids, w = _route(dev, L, k, lb, El)
        oi, ow = oracle.route(L, k, lb, El)
        np.testing.assert_array_equal(ids, oi)
        np.testing.assert_allclose(w, ow, rtol=1e-6, atol=1e-9)


def test_route_ties_and_signed_zero(dev):
    rng = np.random.default_rng(9)
    L = rng.choice(np.array([-1.0, -0.0, 0.0, 0.5, 2.0], np.float32), size=(300, 40))
    for k in (1, 5, 32):
        ids, w = _route(dev, L, k, 0, 40)
        oi, ow = oracle.route(L, k, 0, 40)
        np.testing.assert_array_equal(ids, oi)
        np.testing.assert_allclose(w, ow, rtol=1e-6, atol=1e-9)


def test_route_worked_example(dev, golden_dir):
    g = json.load(open(os.path.join(golden_dir, "route_worked.json")))
    L = np.array(g["logits"], dtype=np.float32)
    ids, w = _route(dev, L, g["top_k"], g["local_begin"], g["E_local"])
    np.testing.assert_array_equal(ids, np.array(g["local_ids"]))
    np.testing.assert_allclose(w, np.array(g["weights"]), atol=g["weights_tol"])


def test_route_empty(dev):
    from paper_2607_18002_amd import ops
    ids, w = ops.moe_topk_route(torch.zeros((0, 8), device=dev), 2, 0, 8)
    assert ids.shape == (0, 2)


# ----------------------------------------------------------------------------- a2 permutation
def _permute(dev, ids, E, align, x, x_scales=None, capacity=None, maps_only=False):
    from paper_2607_18002_amd import ops
    from paper_2607_18002_amd.pipeline import bf16_tensor
    T, k = ids.shape
    H = x.shape[1]
    cap = capacity or T * min(k, E) + E * (align - 1)
    fp8 = x.dtype == np.uint8
    xd = torch.from_numpy(x).to(dev) if fp8 else bf16_tensor(x, dev)
    xs = torch.from_numpy(x_scales).to(dev) if fp8 else None
    out = dict(counts=torch.full((E,), -5, dtype=torch.int32, device=dev),
               offsets=torch.full((E + 1,), -5, dtype=torch.int32, device=dev),
               r2a=torch.full((cap,), -5, dtype=torch.int32, device=dev),
               a2r=torch.full((T * k,), -5, dtype=torch.int32, device=dev),
               xp=torch.full((cap, H), 7, dtype=torch.uint8 if fp8 else torch.int16, device=dev),
               xps=torch.full((cap, H // 128), 7.0, device=dev) if fp8 else None,
               ws=torch.zeros(ops.moe_permute_workspace_bytes(T, k, E), dtype=torch.uint8, device=dev),
               err=torch.zeros(1, dtype=torch.int32, device=dev))
    xp_arg = out["xp"] if fp8 else out["xp"].view(torch.bfloat16)
    if maps_only:                                            # the copy buffers are not passed
        xp_arg = out["xps"] = None
    ops.moe_permute(torch.from_numpy(ids).to(dev), E, xd, xs, align, cap, out["counts"], out["offsets"],
                    out["r2a"], out["a2r"], xp_arg, out["xps"], out["ws"], out["err"])
    torch.cuda.synchronize()
    res = {n: (t.cpu().numpy() if t is not None else None) for n, t in out.items()}
    if not fp8 and not maps_only:
        res["xp"] = res["xp"].view(np.uint16)
    return res, cap


@pytest.mark.parametrize("T,k,E,align", [(1, 1, 1, 1), (37, 8, 32, 128), (600, 8, 32, 32), (4096, 8, 32, 128),
                                         (5001, 4, 12, 16), (20000, 8, 32, 128), (300, 2, 1000, 8)])
def test_permute_bit_exact(dev, T, k, E, align):
    rng = np.random.default_rng(T + k * 31 + E)
    L = rng.standard_normal((T, max(E * 2, k))).astype(np.float32)
    L[:, 0] += 1.0                                           # a hot expert
    ids, _ = oracle.route(L, k, 0, E)
    H = 256
    x = rng.integers(0, 65535, size=(T, H), dtype=np.uint16)
    got, cap = _permute(dev, ids, E, align, x)
    ref = oracle.permute(ids, E, align, x, capacity=cap)
    used = int(ref.offsets[-1])
    np.testing.assert_array_equal(got["counts"], ref.counts)
    np.testing.assert_array_equal(got["offsets"], ref.offsets)
    np.testing.assert_array_equal(got["r2a"][:used], ref.row_to_assign[:used])
    np.testing.assert_array_equal(got["a2r"], ref.assign_to_row)
    np.testing.assert_array_equal(got["xp"][:used], ref.x_perm[:used])
    assert np.all(got["r2a"][used:] == -5), "rows past the last segment are left untouched"
    assert got["err"][0] == 0


def test_permute_workspace_reused_across_sizes(dev):
    """One zeroed workspace serves calls of different sizes in turn: the
    last-block ticket returns to zero after every call."""
    from paper_2607_18002_amd import ops
    rng = np.random.default_rng(21)
    E, k, align, H = 16, 4, 32, 128
    ws = torch.zeros(ops.moe_permute_workspace_bytes(3000, k, E), dtype=torch.uint8, device=dev)
    for T in (3000, 7, 1, 0, 1500, 3000):
        L = rng.standard_normal((max(T, 1), 2 * E)).astype(np.float32)[:T]
        ids, _ = oracle.route(L, k, 0, E) if T else (np.zeros((0, k), np.int32), None)
        cap = T * min(k, E) + E * (align - 1)
        counts = torch.full((E,), -5, dtype=torch.int32, device=dev)
        offsets = torch.full((E + 1,), -5, dtype=torch.int32, device=dev)
        r2a = torch.full((cap,), -5, dtype=torch.int32, device=dev)
        a2r = torch.full((max(T * k, 1),), -5, dtype=torch.int32, device=dev)
        err = torch.zeros(1, dtype=torch.int32, device=dev)
        x = torch.zeros((max(T, 1), H), dtype=torch.bfloat16, device=dev)[:T]
        ops.moe_permute(torch.from_numpy(ids).to(dev), E, x, None, align, cap, counts, offsets, r2a, a2r, None,
                        None, ws, err)
        torch.cuda.synchronize()
        ref = oracle.permute(ids, E, align, capacity=cap)
        used = int(ref.offsets[-1])
        assert int(err.item()) == 0
        np.testing.assert_array_equal(counts.cpu().numpy(), ref.counts)
        np.testing.assert_array_equal(offsets.cpu().numpy(), ref.offsets)
        np.testing.assert_array_equal(r2a.cpu().numpy()[:used], ref.row_to_assign[:used])
        np.testing.assert_array_equal(a2r.cpu().numpy()[:T * k], ref.assign_to_row)
        assert int(ws[:256].view(torch.int32).abs().sum().item()) == 0


@pytest.mark.parametrize("fp8", [False, True])
def test_permute_maps_only(dev, fp8):
    """Without x_perm the call builds the same maps (bit-exact), including the
    -1 of every padding row inside the segments."""
    rng = np.random.default_rng(12)
    T, k, E, align = 900, 8, 24, 64
    L = rng.standard_normal((T, 2 * E)).astype(np.float32)
    L[:, 1] += 1.0
    ids, _ = oracle.route(L, k, 0, E)
    if fp8:
        x = rng.integers(0, 255, size=(T, 256), dtype=np.uint8)
        xs = rng.random((T, 2), dtype=np.float32)
    else:
        x, xs = rng.integers(0, 1 << 15, size=(T, 256), dtype=np.uint16), None
    got, cap = _permute(dev, ids, E, align, x, xs, maps_only=True)
    ref = oracle.permute(ids, E, align, capacity=cap)
    used = int(ref.offsets[-1])
    assert got["err"][0] == 0
    assert (ref.row_to_assign[:used] == -1).any()
    np.testing.assert_array_equal(got["counts"], ref.counts)
    np.testing.assert_array_equal(got["offsets"], ref.offsets)
    np.testing.assert_array_equal(got["r2a"][:used], ref.row_to_assign[:used])
    np.testing.assert_array_equal(got["a2r"], ref.assign_to_row)


def test_permute_fp8_rows_and_scales(dev):
    rng = np.random.default_rng(5)
    T, k, E, H = 700, 8, 32, 512
    ids, _ = oracle.route(rng.standard_normal((T, 256)).astype(np.float32), k, 0, E)
    x = rng.integers(0, 255, size=(T, H), dtype=np.uint8)
    xs = rng.random((T, H // 128)).astype(np.float32)
    got, cap = _permute(dev, ids, E, 128, x, xs)
    ref = oracle.permute(ids, E, 128, x, cap, xs)
    used = int(ref.offsets[-1])
    np.testing.assert_array_equal(got["xp"][:used], ref.x_perm[:used])
    np.testing.assert_array_equal(got["xps"][:used], ref.x_perm_scales[:used])


def test_permute_bad_expert_is_reported(dev):
    ids = np.array([[0, 5], [1, -1], [-3, 2]], dtype=np.int32)     # 5 and -3 are outside [-1, 4)
    x = np.zeros((3, 128), dtype=np.uint16)
    got, cap = _permute(dev, ids, 4, 4, x)
    assert got["err"][0] == -7
    assert got["a2r"][1] == -1 and got["a2r"][4] == -1
    np.testing.assert_array_equal(got["counts"], [1, 1, 1, 0])


# ----------------------------------------------------------------------------- a7 combine
def test_combine_matches_oracle(dev):
    from paper_2607_18002_amd import ops
    from paper_2607_18002_amd.pipeline import bf16_tensor
    rng = np.random.default_rng(6)
    T, k, E, H = 333, 8, 32, 384
    L = rng.standard_normal((T, 128)).astype(np.float32)
    L[:7, :E] = -50.0                                          # tokens with no local slot
    ids, w = oracle.route(L, k, 0, E)
    p = oracle.permute(ids, E, 32)
    rows = len(p.row_to_assign)
    yp_bits = bf16_bits(rng.standard_normal((rows, H)).astype(np.float32))
    want = oracle.combine(oracle.bf16_to_f64(yp_bits), p.assign_to_row, w.astype(np.float32).astype(np.float64), T, k)
    for dt in (torch.float32, torch.bfloat16):
        y = ops.moe_combine(bf16_tensor(yp_bits, dev), torch.from_numpy(p.assign_to_row).to(dev),
                            torch.from_numpy(w.astype(np.float32)).to(dev), T, k, out_dtype=dt)
        got = y.float().cpu().numpy()
        assert np.all(got[:7] == 0.0)
        tol = 1e-6 if dt == torch.float32 else 8e-3
        assert normwise_rel_err(got, want) < tol


# ----------------------------------------------------------------------------- a3-a7 through the pipeline
def _run_pipeline(dev, specs, **kw):
    from paper_2607_18002_amd.pipeline import MoEPipeline
    pipe = MoEPipeline(specs, **kw)
    pipe.run()
    torch.cuda.synchronize()
    return pipe


def _check_op(pipe, i, cfg, lay, ph, tol=BF16_TOL, h_fp8=False):
    from paper_2607_18002_amd.pipeline import bits_of
    b = pipe.bufs[i]
    ref = oracle.moe_local_share(ph.logits, ph.x, lay.weights, cfg.top_k, cfg.local_begin, cfg.E_local,
                                 b.row_align, x_scales=ph.x_scales, capacity=b.capacity, h_fp8=h_fp8)
    np.testing.assert_array_equal(b.topk_ids.cpu().numpy(), ref["ids"])
    np.testing.assert_allclose(b.topk_w.cpu().numpy(), ref["w"], rtol=1e-6, atol=1e-9)
    p = ref["perm"]
    np.testing.assert_array_equal(b.counts.cpu().numpy(), p.counts)
    np.testing.assert_array_equal(b.offsets.cpu().numpy(), p.offsets)
    valid = p.row_to_assign >= 0
    yp = oracle.bf16_to_f64(bits_of(b.y_perm))
    err_rows = normwise_rel_err(yp[valid], ref["y_perm"][valid])
    err_y = normwise_rel_err(b.y.float().cpu().numpy(), ref["y"])
    assert err_rows < tol, f"y_perm rows: {err_rows}"
    assert err_y < tol, f"y: {err_y}"
    return err_rows, err_y


# fp8: the kernel forms h in fp32 and the oracle in float64; the two differ by
# the rounding of fp32 sums, which grows with the sum of the magnitudes of the
# terms, not with |h| (measured: within 2.4e-6 of sum |x w| on these shapes,
# the sqrt(K) * 2^-24 growth of an fp32 sum).  Where that difference decides
# an h code -- the oracle's value lies within the bound of a rounding
# midpoint -- every code the bound reaches is valid.
FP8_GAMMA = 2.0 ** -16


def _h_code_bounds(p, weights, h, sc, g_sc):
    """Lowest and highest valid h code values (scaled units) per element."""
    xp = oracle.dequant_rows(p.x_perm, p.x_perm_scales)
    I = weights["w_down"].shape[2]
    bound = np.zeros_like(h)
    for e in range(len(p.counts)):
        m, r0 = int(p.counts[e]), int(p.offsets[e])
        if m == 0:
            continue
        gu = oracle.dequant_weight(weights["w_gate_up"][e], weights["w_gate_up_scales"][e])
        x = xp[r0:r0 + m]
        g, u = x @ gu[:I].T, x @ gu[I:].T
        sg = 1.0 / (1.0 + np.exp(-g))
        silu, dsilu = g * sg, sg * (1.0 + g * (1.0 - sg))
        bound[r0:r0 + m] = FP8_GAMMA * (np.abs(dsilu * u) * (np.abs(x) @ np.abs(gu[:I]).T) +
                                        np.abs(silu) * (np.abs(x) @ np.abs(gu[I:]).T))
    valid = p.row_to_assign >= 0
    s = np.repeat(sc, 128, axis=1)
    v = h[valid] / s
    dv = bound[valid] / s + np.abs(v) * np.repeat(np.abs(g_sc - sc) / sc, 128, axis=1)
    return oracle.e4m3_to_f64(oracle.e4m3_quantize(v - dv)), oracle.e4m3_to_f64(oracle.e4m3_quantize(v + dv))


def _check_fp8_op(pipe, i, cfg, lay, ph, tol=BF16_TOL):
    """Indices bit-exact; h scales within 1e-3 and every h code within the
    fp32 bound of the oracle's (_h_code_bounds); y_perm and y within `tol` of
    the oracle's down projection and combine applied to the GPU's own h."""
    from paper_2607_18002_amd.pipeline import bits_of
    b = pipe.bufs[i]
    ids, w = oracle.route(ph.logits, cfg.top_k, cfg.local_begin, cfg.E_local)
    np.testing.assert_array_equal(b.topk_ids.cpu().numpy(), ids)
    np.testing.assert_allclose(b.topk_w.cpu().numpy(), w, rtol=1e-6, atol=1e-9)
    p = oracle.permute(ids, cfg.E_local, b.row_align, ph.x, b.capacity, ph.x_scales)
    np.testing.assert_array_equal(b.counts.cpu().numpy(), p.counts)
    np.testing.assert_array_equal(b.offsets.cpu().numpy(), p.offsets)
    valid = p.row_to_assign >= 0
    if b.x_perm is not None:                                 # else the FFN gathered x rows itself
        np.testing.assert_array_equal(b.x_perm.cpu().numpy()[valid], p.x_perm[valid])
        np.testing.assert_array_equal(b.x_perm_scales.cpu().numpy()[valid], p.x_perm_scales[valid])
    h = oracle.grouped_hidden(oracle.dequant_rows(p.x_perm, p.x_perm_scales), p.counts, p.offsets, lay.weights)
    codes, sc = oracle.quantize_rows(h[valid])
    g_codes, g_sc = b.h.cpu().numpy()[valid], b.h_scales.cpu().numpy()[valid].astype(np.float64)
    assert np.max(np.abs(g_sc - sc) / sc) < 1e-3
    lo, hi = _h_code_bounds(p, lay.weights, h, sc, g_sc)
    gv = oracle.e4m3_to_f64(g_codes)
    ok = (gv >= lo) & (gv <= hi)
    assert ok.all(), f"{(~ok).sum()} h codes outside the fp32 bound"
    assert (g_codes == codes).mean() > 0.99
    h_gpu = np.zeros_like(h)
    h_gpu[valid] = oracle.dequant_rows(g_codes, g_sc)
    y_perm = oracle.grouped_down(h_gpu, p.counts, p.offsets, lay.weights)
    err_rows = normwise_rel_err(oracle.bf16_to_f64(bits_of(b.y_perm))[valid], y_perm[valid])
    y = oracle.combine(y_perm, p.assign_to_row, w, ids.shape[0], cfg.top_k)
    err_y = normwise_rel_err(b.y.float().cpu().numpy(), y)
    assert err_rows < tol, f"y_perm rows: {err_rows}"
    assert err_y < tol, f"y: {err_y}"
    return err_rows, err_y


def test_tiny_config_both_phases_one_launch(dev):
    cfg = CONFIGS[1]
    specs, lay, _ = layer_specs(cfg, 0, dev)
    pipe = _run_pipeline(dev, specs, trace_capacity=4096)
    assert pipe.statuses() == (0, 0)
    for i, ph in enumerate(lay.phases):
        _check_op(pipe, i, cfg, lay, ph)


@pytest.mark.parametrize("H,I,T_p,T_d,E_g,E_l,k", [(512, 256, 700, 90, 64, 8, 4), (256, 768, 300, 300, 16, 16, 2),
                                                   (768, 512, 1100, 45, 128, 12, 8)])
@pytest.mark.parametrize("fused", [False, True], ids=["x_perm", "gathered"])
def test_small_ragged_configs(dev, H, I, T_p, T_d, E_g, E_l, k, fused):
    cfg = custom_config(2, cfg_id=200 + H + I, H=H, I=I, prefill_tokens=T_p, decode_tokens=T_d,
                        E_global=E_g, E_local=E_l, top_k=k, zipf_s=(1.3,))
    lay = make_layer(cfg, 0)
    lay.phases[0].logits[:, 3] = -100.0                      # local expert 3 receives no prefill row
    specs, lay, _ = layer_specs(cfg, 0, dev, lay=lay)
    pipe = _run_pipeline(dev, specs, trace_capacity=1 << 16, fused_gather=fused)
    assert pipe.statuses() == (0, 0)
    assert pipe.bufs[0].counts.cpu().numpy()[3] == 0
    for i, ph in enumerate(lay.phases):
        _check_op(pipe, i, cfg, lay, ph)


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_gathered_operand_matches_the_copy_bitwise(dev, dtype):
    """GEMM-1 reading x through row_to_assign performs the same arithmetic as
    reading the permuted copy: h and y_perm are bit-identical."""
    base = 2 if dtype == "bf16" else 5
    cfg = custom_config(base, cfg_id=700 + base, H=512, I=512, prefill_tokens=500, decode_tokens=37,
                        E_global=64, E_local=8, top_k=4, zipf_s=(1.3,))
    specs, lay, _ = layer_specs(cfg, 0, dev)
    a = _run_pipeline(dev, specs)
    b = _run_pipeline(dev, specs, fused_gather=True)
    assert a.statuses() == (0, 0) and b.statuses() == (0, 0)
    for ba, bb in zip(a.bufs, b.bufs):
        valid = (ba.row_to_assign >= 0).cpu().numpy()
        assert torch.equal(ba.row_to_assign, bb.row_to_assign)
        assert np.array_equal(ba.h.view(torch.uint8).cpu().numpy()[valid], bb.h.view(torch.uint8).cpu().numpy()[valid])
        assert np.array_equal(ba.y_perm.view(torch.int16).cpu().numpy()[valid],
                              bb.y_perm.view(torch.int16).cpu().numpy()[valid])
        assert torch.equal(ba.y.view(torch.int16), bb.y.view(torch.int16))


def test_token_without_local_expert_is_exact_zero(dev):
    cfg = custom_config(2, cfg_id=301, H=256, I=256, prefill_tokens=64, decode_tokens=0, E_global=64, E_local=8,
                        top_k=2)
    lay = make_layer(cfg, 0)
    lay.phases[0].logits[:10, :8] = -100.0
    specs, lay, _ = layer_specs(cfg, 0, dev, lay=lay)
    pipe = _run_pipeline(dev, specs)
    y = pipe.bufs[0].y.float().cpu().numpy()
    assert np.all(y[:10] == 0.0)
    _check_op(pipe, 0, cfg, lay, lay.phases[0])


def _sampled_full_size(dev, cfg_id, layers=(0,), n_sample=10, tol=BF16_TOL, h_fp8_tol=None, fused_gather=False):
    """Full-size configuration: every index bit-exact, sampled tokens' outputs
    against the oracle evaluated token by token."""
    from paper_2607_18002_amd.pipeline import bits_of
    cfg = CONFIGS[cfg_id]
    specs, lays = [], []
    for layer in layers:
        s, lay, _ = layer_specs(cfg, layer, dev)
        specs += s
        lays += [(lay, ph) for ph in lay.phases]
    pipe = _run_pipeline(dev, specs, trace_capacity=0, fused_gather=fused_gather)
    assert pipe.statuses() == (0, 0)
    rng = np.random.default_rng(cfg_id)
    worst = 0.0
    for i, (lay, ph) in enumerate(lays):
        b = pipe.bufs[i]
        ids, w = oracle.route(ph.logits, cfg.top_k, cfg.local_begin, cfg.E_local)
        np.testing.assert_array_equal(b.topk_ids.cpu().numpy(), ids)
        np.testing.assert_allclose(b.topk_w.cpu().numpy(), w, rtol=1e-6, atol=1e-9)
        p = oracle.permute(ids, cfg.E_local, b.row_align, capacity=b.capacity)
        np.testing.assert_array_equal(b.counts.cpu().numpy(), p.counts)
        np.testing.assert_array_equal(b.offsets.cpu().numpy(), p.offsets)
        used = int(p.offsets[-1])
        np.testing.assert_array_equal(b.row_to_assign.cpu().numpy()[:used], p.row_to_assign[:used])
        np.testing.assert_array_equal(b.assign_to_row.cpu().numpy(), p.assign_to_row)
        # sampled tokens: the hottest expert's first and last rows, the last expert's last row, random others
        has_local = np.nonzero((ids >= 0).any(axis=1))[0]
        c = p.counts
        pick = {p.row_to_assign[p.offsets[0]] // cfg.top_k, p.row_to_assign[p.offsets[0] + c[0] - 1] // cfg.top_k}
        last = int(np.nonzero(c)[0][-1])
        pick.add(p.row_to_assign[p.offsets[last] + c[last] - 1] // cfg.top_k)
        pick.update(rng.choice(has_local, size=min(n_sample, len(has_local)), replace=False).tolist())
        pick = sorted(int(t) for t in pick)
        y = b.y.float().cpu().numpy()
        xf = oracle.dequant_rows(ph.x, ph.x_scales)
        cache = {}
        want = np.stack([oracle.token_output(xf[t], ids[t], w[t], lay.weights, cache) for t in pick])
        err = normwise_rel_err(y[pick], want)
        worst = max(worst, err)
        assert err < tol, (i, err)
        if h_fp8_tol is not None:                            # against the oracle that also stores h in fp8
            want_q = np.stack([oracle.token_output(xf[t], ids[t], w[t], lay.weights, cache, h_fp8=True)
                               for t in pick])
            err_q = normwise_rel_err(y[pick], want_q)
            assert err_q < h_fp8_tol, (i, err_q)
    return worst


def test_full_size_decode_config(dev):
    _sampled_full_size(dev, 2)


def test_full_size_prefill_config(dev):
    _sampled_full_size(dev, 3)


def test_full_size_mixed_config_two_layers(dev):
    _sampled_full_size(dev, 4, layers=(0, 1), n_sample=6)


def test_full_size_mixed_config_gathered(dev):
    """The mixed configuration with GEMM-1 reading x through row_to_assign."""
    _sampled_full_size(dev, 4, n_sample=6, fused_gather=True)


def test_full_size_fp8_mixed_config_gathered(dev):
    _sampled_full_size(dev, 5, n_sample=6, tol=FP8_TOL, fused_gather=True)


def test_full_size_fp8_mixed_config(dev):
    """fp8 e4m3 with 128 x 128 weight scales and 1 x 128 activation scales,
    H 6144, I 2048, 4096 prefill + 1024 decode tokens in one launch: within
    3e-2 of the float64 oracle (h unquantized)."""
    _sampled_full_size(dev, 5, n_sample=8, tol=FP8_TOL)


@pytest.mark.parametrize("H,I,T_p,T_d,E_g,E_l,k", [(512, 256, 600, 70, 64, 8, 4), (256, 512, 200, 200, 16, 16, 2),
                                                   (768, 768, 900, 33, 128, 12, 8)])
@pytest.mark.parametrize("fused", [False, True], ids=["x_perm", "gathered"])
def test_fp8_small_configs(dev, H, I, T_p, T_d, E_g, E_l, k, fused):
    """fp8 path on ragged shapes: 32- to 128-row tiles, several row tiles per
    expert, an expert without rows; checked stage by stage (_check_fp8_op).
    At these small widths the fp8 rounding of h alone can exceed 3e-2 against
    the unquantized oracle, so the end-to-end 3e-2 bound is checked at the
    full-size shape."""
    cfg = custom_config(5, cfg_id=600 + H + I, H=H, I=I, prefill_tokens=T_p, decode_tokens=T_d,
                        E_global=E_g, E_local=E_l, top_k=k, zipf_s=(1.3,))
    lay = make_layer(cfg, 0)
    lay.phases[0].logits[:, 2] = -100.0                      # local expert 2 receives no prefill row
    specs, lay, _ = layer_specs(cfg, 0, dev, lay=lay)
    pipe = _run_pipeline(dev, specs, trace_capacity=1 << 16, fused_gather=fused)
    assert pipe.statuses() == (0, 0)
    assert pipe.bufs[0].counts.cpu().numpy()[2] == 0
    assert pipe.bufs[0].row_align == 32
    for i, ph in enumerate(lay.phases):
        _check_fp8_op(pipe, i, cfg, lay, ph)


def test_pack_weights_layout_fp8(dev):
    """fp8 layout: chunk c of 32-row block b holds, for kk = 0..1, half = 0..1
    and lane = 0..63, row 32b + lane%32, columns 128c + 64kk + (lane/32)*32 +
    16*half .. +16 (bit copy)."""
    from paper_2607_18002_amd import ops
    rng = np.random.default_rng(37)
    E, N, K = 2, 64, 384
    w = rng.integers(0, 256, size=(E, N, K), dtype=np.uint8)
    got = ops.moe_pack_weights(torch.from_numpy(w).to(dev)).cpu().numpy().reshape(E, -1)
    want = np.empty((E, N * K), dtype=np.uint8)
    pos = 0
    for b in range(N // 32):
        for c in range(K // 128):
            for kk in range(2):
                for half in range(2):
                    for lane in range(64):
                        row = 32 * b + lane % 32
                        col = 128 * c + 64 * kk + (lane // 32) * 32 + 16 * half
                        want[:, pos:pos + 16] = w[:, row, col:col + 16]
                        pos += 16
    np.testing.assert_array_equal(got, want)


def test_buffers_reused_across_launches_with_new_inputs(dev):
    """Second launch on the same buffers with different inputs and weights:
    the persistent kernel never invalidates caches on its h handoff, so a
    stale copy from the first launch would show up here."""
    from paper_2607_18002_amd.pipeline import MoEPipeline, bf16_tensor
    cfg = custom_config(2, cfg_id=501, H=512, I=512, prefill_tokens=900, decode_tokens=200, E_global=64,
                        E_local=16, top_k=4, zipf_s=(1.1, 0.7), n_layers=2)
    specs, lay0, w = layer_specs(cfg, 0, dev)
    pipe = MoEPipeline(specs)
    for layer in (0, 1, 0):
        lay = make_layer(cfg, layer)
        for s, ph in zip(specs, lay.phases):
            s.logits.copy_(torch.from_numpy(ph.logits).to(dev))
            s.x.copy_(bf16_tensor(ph.x, dev))
        w.load(bf16_tensor(lay.weights["w_gate_up"], dev), bf16_tensor(lay.weights["w_down"], dev))
        pipe.run()
        torch.cuda.synchronize()
        assert pipe.statuses() == (0, 0)
        for i, ph in enumerate(lay.phases):
            _check_op(pipe, i, cfg, lay, ph)


def test_pack_weights_layout(dev):
    """moe_pack_weights writes the documented layout: chunk c of 32-row block b
    holds, for q = 0..3 and lane = 0..63, row 32b + lane%32, columns
    64c + (lane/32)*32 + 8q .. +8 (bit copy)."""
    from paper_2607_18002_amd import ops
    from paper_2607_18002_amd.pipeline import bf16_tensor, bits_of
    rng = np.random.default_rng(31)
    E, N, K = 3, 96, 192
    w = rng.integers(0, 65535, size=(E, N, K), dtype=np.uint16)
    got = bits_of(ops.moe_pack_weights(bf16_tensor(w, dev))).reshape(E, -1)
    want = np.empty((E, N * K), dtype=np.uint16)
    pos = 0
    for b in range(N // 32):
        for c in range(K // 64):
            for q in range(4):
                for lane in range(64):
                    row, col = 32 * b + lane % 32, 64 * c + (lane // 32) * 32 + 8 * q
                    want[:, pos:pos + 8] = w[:, row, col:col + 8]
                    pos += 8
    np.testing.assert_array_equal(got, want)


def test_gathered_operand_argument_errors(dev):
    """The GEMM-1 operand is exactly one of x_perm and x; a gathered operand
    needs its row map, T and top_k.  Rejected on the host, nothing launched."""
    from paper_2607_18002_amd import _lib
    from paper_2607_18002_amd.pipeline import MoEPipeline
    cfg = custom_config(2, cfg_id=710, H=256, I=256, prefill_tokens=64, decode_tokens=0, E_global=16, E_local=8,
                        top_k=2)
    specs, _, _ = layer_specs(cfg, 0, dev)
    pipe = MoEPipeline(specs)
    lib = _lib.load_library()
    d = pipe.descs[0]
    cases = [dict(x=specs[0].x.data_ptr()),                                            # both operands
             dict(x_perm=None, x=specs[0].x.data_ptr()),                              # no row map
             dict(x_perm=None, x=specs[0].x.data_ptr(), row_to_assign=pipe.bufs[0].row_to_assign.data_ptr(),
                  T=64, top_k=0),
             dict(x_perm=None)]                                                        # neither
    for kw in cases:
        bad = _lib.OpDesc.from_buffer_copy(d)
        for k, v in kw.items():
            setattr(bad, k, v)
        arr = (_lib.OpDesc * 1)(bad)
        rc = lib.moe_grouped_ffn_persistent(arr, 1, C.byref(pipe.cfg), pipe.ffn_ws.data_ptr(),
                                            pipe.status.data_ptr(), None)
        assert rc == _lib.MOE_ERR_INVALID_ARG, (kw, rc)
    torch.cuda.synchronize()
    assert int(pipe.status.item()) == 0


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_batched_calls_match_per_op_calls(dev, dtype):
    """moe_topk_route_batch / moe_permute_batch / moe_combine_batch over the
    ops of one launch (2 layers x 2 phases) give bitwise the results of the
    per-op calls."""
    from paper_2607_18002_amd.pipeline import MoEPipeline
    base = 2 if dtype == "bf16" else 5
    cfg = custom_config(base, cfg_id=710 + base, H=512, I=512, prefill_tokens=700, decode_tokens=90, E_global=64,
                        E_local=12, top_k=6, zipf_s=(1.2, 0.7), n_layers=2)
    specs = []
    for layer in range(2):
        s, _, _ = layer_specs(cfg, layer, dev)
        specs += s
    outs = []
    for batched in (False, True):
        pipe = MoEPipeline(specs, fused_gather=True)
        pipe.route(batched=batched)
        pipe.permute(batched=batched)
        pipe.ffn()
        pipe.combine(batched=batched)
        torch.cuda.synchronize()
        assert pipe.statuses() == (0, 0)
        outs.append([(b.topk_ids.cpu(), b.topk_w.cpu(), b.counts.cpu(), b.offsets.cpu(), b.row_to_assign.cpu(),
                      b.assign_to_row.cpu(), b.y.view(torch.int16).cpu()) for b in pipe.bufs])
    for a, b in zip(*outs):
        for ta, tb in zip(a, b):
            assert torch.equal(ta, tb)


@pytest.mark.parametrize("dtype,y_f32", [("bf16", False), ("fp8", False), ("bf16", True)])
def test_fused_combine_matches_separate_combine(dev, dtype, y_f32):
    """Combine tiles inside the persistent kernel give moe_combine's y bit for
    bit (the same fp32 accumulation order) for every op of a 2-layer mixed
    launch, including an op none of whose tokens routes to a local expert: it
    runs no GEMM tile, and its combine tiles write zeros."""
    import dataclasses
    from paper_2607_18002_amd.pipeline import MoEPipeline
    base = 2 if dtype == "bf16" else 5
    cfg = custom_config(base, cfg_id=720 + base, H=512, I=512, prefill_tokens=700, decode_tokens=90, E_global=64,
                        E_local=12, top_k=6, zipf_s=(1.2, 0.7), n_layers=2)
    specs = []
    for layer in range(2):
        s, _, _ = layer_specs(cfg, layer, dev)
        specs += s
    last = specs[-1]
    lg = last.logits.clone()
    lg[:, last.local_begin:last.local_begin + last.E_local] = -1.0e4
    specs[-1] = dataclasses.replace(last, logits=lg)
    ydt = torch.float32 if y_f32 else torch.bfloat16
    outs = []
    for fused in (False, True):
        pipe = MoEPipeline(specs, fused_gather=True, fused_combine=fused, y_dtype=ydt)
        for b in pipe.bufs:
            b.y.fill_(3.0)                                   # every element must be written
        pipe.run()
        torch.cuda.synchronize()
        assert pipe.statuses() == (0, 0)
        assert int(pipe.bufs[-1].counts.sum().item()) == 0
        outs.append([b.y.view(torch.int32 if y_f32 else torch.int16).cpu() for b in pipe.bufs])
    for a, b in zip(*outs):
        assert torch.equal(a, b)
    assert not outs[1][-1].any()


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("prefill_too", [False, True], ids=["decode", "both"])
def test_masked_layout(dev, dtype, prefill_too):
    """Ops in the masked layout (routing places each local slot in its
    expert's fixed region; no permute pass): counts, offsets and both maps
    equal the oracle's masked layout bit for bit over three steps on the same
    buffers, the outputs match the oracle, and y equals the contiguous
    layout's bit for bit (each row is computed on its own)."""
    from paper_2607_18002_amd import MOE_DECODE
    from paper_2607_18002_amd.pipeline import MoEPipeline
    base = 2 if dtype == "bf16" else 5
    cfg = custom_config(base, cfg_id=740 + base, H=512, I=512, prefill_tokens=600, decode_tokens=77, E_global=64,
                        E_local=12, top_k=6, zipf_s=(1.2, 0.7), n_layers=2)
    specs, lays = [], []
    for layer in range(2):
        s, lay, _ = layer_specs(cfg, layer, dev)
        specs += s
        lays += [(lay, ph) for ph in lay.phases]
    ref = MoEPipeline(specs, fused_gather=True)
    msk = MoEPipeline(specs, fused_gather=True, masked_decode=True, masked_prefill=prefill_too)
    for step in range(3):
        for p in (ref, msk):
            p.run()
        torch.cuda.synchronize()
        assert ref.statuses() == (0, 0) and msk.statuses() == (0, 0)
        for i, (br, bm) in enumerate(zip(ref.bufs, msk.bufs)):
            lay, ph = lays[i]
            assert torch.equal(br.topk_ids, bm.topk_ids) and torch.equal(br.topk_w, bm.topk_w)
            assert torch.equal(br.counts, bm.counts)
            assert torch.equal(br.y.view(torch.int16), bm.y.view(torch.int16))
            masked = bm.spec.phase == MOE_DECODE or prefill_too
            assert (bm.slots > 0) == masked
            if not masked:
                continue
            ids = bm.topk_ids.cpu().numpy()
            o = oracle.permute_masked(ids, cfg.E_local, bm.slots)
            np.testing.assert_array_equal(bm.counts.cpu().numpy(), o.counts)
            np.testing.assert_array_equal(bm.offsets.cpu().numpy(), o.offsets)
            np.testing.assert_array_equal(bm.assign_to_row.cpu().numpy(), o.assign_to_row)
            r2a = bm.row_to_assign.cpu().numpy()
            for e in range(cfg.E_local):
                lo = e * bm.slots
                np.testing.assert_array_equal(r2a[lo:lo + o.counts[e]], o.row_to_assign[lo:lo + o.counts[e]])
            # bf16 outputs against the oracle; fp8 outputs equal the contiguous
            # layout's bit for bit (above), whose h codes, scales and outputs are
            # checked stage by stage against the oracle in test_fp8_small_configs
            if step == 0 and dtype == "bf16":
                want = oracle.moe_local_share(ph.logits, ph.x, lay.weights, cfg.top_k, cfg.local_begin, cfg.E_local,
                                              32, slots=bm.slots)
                assert normwise_rel_err(bm.y.float().cpu().numpy(), want["y"]) < BF16_TOL


@pytest.mark.parametrize("T_seq,E,E_l,k", [((1000, 300, 1000, 5, 1), 64, 16, 8), ((257, 64), 1000, 300, 32),
                                           ((3, 130), 8, 8, 2), ((5000, 2048, 2049, 700, 5000), 64, 8, 4)])
def test_masked_placement_calls_share_a_workspace(dev, T_seq, E, E_l, k):
    """Routing with masked placement, called repeatedly on one placement
    workspace with changing token counts (the workspace sized for the
    largest): every call's counts and maps equal the oracle's masked layout,
    including E_local above one thread per expert and k = 32."""
    from paper_2607_18002_amd import ops
    Tmax = max(T_seq)
    slots = (Tmax + 31) // 32 * 32
    ws = torch.zeros((ops.moe_route_place_workspace_bytes(Tmax, E_l),), dtype=torch.uint8, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    counts = torch.full((E_l,), -5, dtype=torch.int32, device=dev)
    for n, T in enumerate(T_seq):
        rng = np.random.default_rng(1000 * n + T)
        L = rng.standard_normal((T, E)).astype(np.float32)
        L[:, : E_l // 3] += 2.0                              # many local selections
        logits = torch.from_numpy(L).to(dev)
        ids = torch.empty((T, k), dtype=torch.int32, device=dev)
        w = torch.empty((T, k), dtype=torch.float32, device=dev)
        a2r = torch.full((T * k,), -7, dtype=torch.int32, device=dev)
        r2a = torch.full((E_l * slots,), -9, dtype=torch.int32, device=dev)
        ops.moe_topk_route_batch([ops.route_args(logits, k, 0, E_l, ids, w, slots=slots, counts=counts, place_ws=ws,
                                                 assign_to_row=a2r, row_to_assign=r2a, error_flag=err)])
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        oi, ow = oracle.route(L, k, 0, E_l)
        np.testing.assert_array_equal(ids.cpu().numpy(), oi)
        o = oracle.permute_masked(oi, E_l, slots)
        np.testing.assert_array_equal(counts.cpu().numpy(), o.counts)
        np.testing.assert_array_equal(a2r.cpu().numpy(), o.assign_to_row)
        got = r2a.cpu().numpy()
        valid = o.row_to_assign >= 0
        np.testing.assert_array_equal(got[valid], o.row_to_assign[valid])
        assert np.all(got[~valid] == -9)                     # rows past a region's count are not written


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_plain_grid_baseline_matches_persistent_bitwise(dev, dtype):
    """The comparison baseline (the same tiles as plain per-op grids, no device
    scheduler) computes h and y_perm bit for bit like the persistent kernel,
    for a 2-layer mixed launch with the masked decode layout."""
    from paper_2607_18002_amd.pipeline import MoEPipeline
    base = 2 if dtype == "bf16" else 5
    cfg = custom_config(base, cfg_id=760 + base, H=512, I=512, prefill_tokens=700, decode_tokens=90, E_global=64,
                        E_local=12, top_k=6, zipf_s=(1.2, 0.7), n_layers=2)
    specs = []
    for layer in range(2):
        s, _, _ = layer_specs(cfg, layer, dev)
        specs += s
    pipe = MoEPipeline(specs, fused_gather=True, masked_decode=True)
    pipe.route()
    pipe.permute()
    outs = []
    for plain in (False, True):
        for b in pipe.bufs:
            b.h.zero_()
            b.y_perm.zero_()
        if plain:
            pipe.ffn_plain()
        else:
            pipe.ffn()
        torch.cuda.synchronize()
        assert pipe.statuses() == (0, 0)
        outs.append([(b.h.view(torch.uint8).clone(), b.y_perm.view(torch.int16).clone()) for b in pipe.bufs])
    for (h0, y0), (h1, y1), b in zip(outs[0], outs[1], pipe.bufs):
        valid = (b.row_to_assign >= 0)
        if b.slots:                                          # masked: rows past a region's count are not outputs
            r = torch.arange(b.capacity, device=dev)
            e = r // b.slots
            valid = (r - e * b.slots) < b.counts.long()[e]
        assert torch.equal(h0[valid], h1[valid])
        assert torch.equal(y0[valid], y1[valid])


def test_prefill_128_row_tiles_match_oracle(dev):
    """With prefill_tile_rows = 128 the bf16 prefill op of a mixed launch runs
    the 128-row tiles (every traced prefill tile has at most 128 rows and the
    op's tile count follows Eq. (3) at M_t = 128); both ops still match the
    oracle."""
    cfg = custom_config(2, cfg_id=403, H=512, I=512, prefill_tokens=1500, decode_tokens=200, E_global=64,
                        E_local=16, top_k=4, zipf_s=(1.1,))
    specs, lay, _ = layer_specs(cfg, 0, dev)
    pipe = _run_pipeline(dev, specs, trace_capacity=1 << 16, fused_gather=True, prefill_tile_rows=128)
    assert pipe.statuses() == (0, 0)
    tr = pipe.trace_records()
    st = pipe.op_stats()
    for i, ph in enumerate(lay.phases):
        _check_op(pipe, i, cfg, lay, ph)
        mine = tr[tr["op"] == i]
        assert len(mine) and int(mine["rows"].max()) <= 128
        counts = pipe.bufs[i].counts.cpu().numpy()
        assert int(st["x_moe"][i]) == oracle.x_moe(counts, 128)
