"""The persistent kernel's scheduler, observed through its per-tile trace and
per-op statistics: every tile runs exactly once (Eq. (3) tile counts),
GEMM-2 tiles start after their row tile's GEMM-1 tiles committed, ops start
only after their release condition, lone phases use every workgroup, the
decode quota holds under contention, results are bitwise independent of the
schedule, and abort / never-released ops end cleanly (forced from the host
with a small spin limit; every wait in the kernel is bounded)."""
import numpy as np
import pytest

import oracle
from _helpers import layer_specs
from workload import CONFIGS, custom_config, make_layer

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TICK_NS = 10.0   # 100 MHz device wall clock


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_18002_amd import load_library
    load_library()
    return torch.device("cuda:0")


def _mixed_cfg():
    return custom_config(2, cfg_id=401, H=512, I=512, prefill_tokens=2048, decode_tokens=256, E_global=64,
                         E_local=16, top_k=4, zipf_s=(1.1,))


def _pipe(dev, specs, **kw):
    from paper_2607_18002_amd.pipeline import MoEPipeline
    p = MoEPipeline(specs, **kw)
    p.run()
    torch.cuda.synchronize()
    return p


def _tiles_per_op(pipe, i):
    b = pipe.bufs[i]
    counts = b.counts.cpu().numpy()
    H, I = b.spec.weights.H, b.spec.weights.I
    from paper_2607_18002_amd import ops
    bm, bn, _ = ops.moe_ffn_tile_shape(b.spec.phase, b.spec.weights.dtype)
    xm = oracle.x_moe(counts, bm)                         # Eq. (3) at the tallest tile height
    return xm, xm * (I // (bn // 2)) + xm * (H // bn)


def test_every_tile_exactly_once_and_dependencies(dev):
    cfg = _mixed_cfg()
    specs, lay, _ = layer_specs(cfg, 0, dev)
    pipe = _pipe(dev, specs, trace_capacity=1 << 16)
    assert pipe.statuses() == (0, 0)
    tr = pipe.trace_records()
    st = pipe.op_stats()
    for i in range(len(specs)):
        xm, ntiles = _tiles_per_op(pipe, i)
        mine = tr[tr["op"] == i]
        assert st["x_moe"][i] == xm                           # Eq. (3) on the device
        assert st["n_tiles"][i] == ntiles == len(mine)
        keys = set(zip(mine["stage"], mine["expert"], mine["mblk"], mine["nblk"]))
        assert len(keys) == len(mine), "a tile ran twice"
        for (e, mb) in set(zip(mine["expert"], mine["mblk"])):
            g1 = mine[(mine["stage"] == 1) & (mine["expert"] == e) & (mine["mblk"] == mb)]
            g2 = mine[(mine["stage"] == 2) & (mine["expert"] == e) & (mine["mblk"] == mb)]
            assert len(g1) and len(g2)
            assert g2["t_start"].min() >= g1["t_end"].max(), "GEMM-2 started before its GEMM-1 row tile committed"
        assert np.all(mine["t_claim"] >= st["t_ready"][i])
        assert st["t_done"][i] >= mine["t_end"].max()                 # done is published after every commit
        assert st["t_done"][i] - mine["t_end"].max() < 2000           # ... promptly (20 us)
        assert np.all(mine["t_start"] <= mine["t_end"])


def test_release_delay_and_layer_dependency(dev):
    """Decode released 10 us after the start, later layers after the previous
    layer of the same phase is done plus a gap."""
    cfg = custom_config(2, cfg_id=402, H=512, I=512, prefill_tokens=1024, decode_tokens=128, E_global=64,
                        E_local=16, top_k=4, zipf_s=(1.1, 0.8), n_layers=2)
    specs = []
    for layer in range(2):
        ready = {"prefill": dict(depends_on_op=(-1 if layer == 0 else 0)),
                 "decode": dict(release_after_ns=10_000 if layer == 0 else -1,
                                depends_on_op=(-1 if layer == 0 else 1), gap_ns=20_000)}
        s, _, _ = layer_specs(cfg, layer, dev, **ready)
        specs += s
    pipe = _pipe(dev, specs, trace_capacity=1 << 16)
    assert pipe.statuses() == (0, 0)
    st = pipe.op_stats()
    t0 = pipe.kernel_t0()
    assert t0 > 0
    assert st["t_ready"][0] >= t0
    assert st["t_ready"][1] >= t0 + int(10_000 / TICK_NS)                    # decode layer 0: 10 us after start
    assert st["t_ready"][2] >= st["t_done"][0]                               # prefill layer 1 after layer 0
    assert st["t_ready"][3] >= st["t_done"][1] + int(20_000 / TICK_NS)       # decode layer 1 after gap


def test_lone_phase_uses_every_workgroup(dev):
    cfg = custom_config(2, cfg_id=403, H=1024, I=1024, prefill_tokens=4096, decode_tokens=0, E_global=64,
                        E_local=16, top_k=8)
    specs, _, _ = layer_specs(cfg, 0, dev)
    pipe = _pipe(dev, specs, trace_capacity=1 << 16, decode_quota_wg=64)
    tr = pipe.trace_records()
    assert len(np.unique(tr["wg"])) == 256
    assert set(np.unique(tr["xcc"]).tolist()) == set(range(8))


HOW_PREFERRED, HOW_OTHER, HOW_AHEAD, HOW_COMBINE = 0, 1, 2, 3


def _claim_lower_bounds(tr):
    """A time no later than each tile's claim atomic: its boundary's polls
    returned (t_polled) before the claim; a tile claimed ahead was claimed
    during the workgroup's previous tile, after that tile started."""
    lb = tr["t_polled"].astype(np.int64).copy()
    ahead = np.nonzero(tr["how"] == HOW_AHEAD)[0]
    for i in ahead:
        m = (tr["wg"] == tr["wg"][i]) & (tr["t_start"] < tr["t_start"][i])
        lb[i] = int(tr["t_start"][m].max())
    return lb


def _check_policy(tr, st, phases_of_op):
    """Every tile's recorded decision inputs (q' used, phases with claimable
    work in its polls, path) against the policy: a workgroup below q' prefers
    decode, the others prefill; a tile of the non-preferred phase is taken only
    when the preferred phase had no tile left to claim -- and then every tile of
    the preferred phase's active op had been claimed before that decision
    (a claim's atomic precedes the stamp of the failed attempt that followed it).
    Returns the number of decode tiles claimed while both phases were active."""
    lb = _claim_lower_bounds(tr)
    phase = phases_of_op[tr["op"]]
    contended = 0
    for i in range(len(tr)):
        how = int(tr["how"][i])
        if how in (HOW_AHEAD, HOW_COMBINE):
            continue
        pref = 1 if tr["wg"][i] < tr["quota_seen"][i] else 0     # 1 decode, 0 prefill
        if how == HOW_PREFERRED:
            assert phase[i] == pref, ("tile of the non-preferred phase recorded as preferred", tr[i])
        else:
            assert phase[i] != pref, tr[i]
            if tr["phases_seen"][i] & (1 if pref == 1 else 2):
                # the preferred phase was active: all its active op's tiles had been claimed
                ops = [o for o in np.nonzero(phases_of_op == pref)[0]
                       if st["t_ready"][o] <= tr["t_polled"][i] and st["t_done"][o] >= tr["t_polled"][i]]
                for o in ops:
                    mine = tr["op"] == o
                    assert np.all(lb[mine] < int(tr["t_claim"][i])), (
                        "the other phase was taken while the preferred phase still had unclaimed tiles", tr[i])
        if phase[i] == 1 and tr["phases_seen"][i] == 3:
            contended += 1
            if how == HOW_PREFERRED:
                assert tr["wg"][i] < tr["quota_seen"][i]
    return contended


def test_decode_quota_under_contention(dev):
    """While prefill has claimable tiles, decode tiles run only on workgroups
    below q' (decided from the inputs each decision recorded, no time windows),
    and workgroups at or above q' take decode tiles only once every prefill
    tile has been claimed."""
    cfg = custom_config(2, cfg_id=404, H=1024, I=1024, prefill_tokens=8192, decode_tokens=256, E_global=64,
                        E_local=16, top_k=8)
    specs, _, _ = layer_specs(cfg, 0, dev, decode=dict(release_after_ns=40_000))
    pipe = _pipe(dev, specs, trace_capacity=1 << 17, decode_quota_wg=64)
    assert pipe.statuses() == (0, 0)
    tr = pipe.trace_records()
    st = pipe.op_stats()
    assert st["quota"][1] == 64
    contended = _check_policy(tr, st, np.array([s.phase for s in specs]))
    assert contended > 0, "no decode tile ran while prefill was active: the test checked nothing"
    dec = tr[(tr["op"] == 1) & (tr["phases_seen"] == 3) & (tr["how"] != HOW_OTHER)]
    assert len(dec) and dec["wg"].max() < 64


@pytest.mark.parametrize("release_us", [10, 45, 130])
def test_bounded_preemption(dev, release_us):
    """Bounded tile-level preemption, term by term from the trace: a decode op
    released while prefill tiles run is seen at the first tile boundary of a
    workgroup below q' after its release (so no later than the remaining time
    of those workgroups' prefill tiles, plus one boundary) and activated by
    that workgroup (its template was built ahead, so no instantiation is
    left), which takes the op's first tile in the same boundary.  The epoch
    (one boundary's decision) is the longest boundary measured in the same
    launch."""
    cfg = custom_config(2, cfg_id=405, H=1024, I=1024, prefill_tokens=8192, decode_tokens=256, E_global=64,
                        E_local=16, top_k=8)
    specs, _, _ = layer_specs(cfg, 0, dev, decode=dict(release_after_ns=release_us * 1000))
    pipe = _pipe(dev, specs, trace_capacity=1 << 17, decode_quota_wg=64)
    assert pipe.statuses() == (0, 0)
    tr = pipe.trace_records()
    st = pipe.op_stats()
    t0 = pipe.kernel_t0()
    R = t0 + int(release_us * 1000 / TICK_NS)
    q = int(st["quota"][1])
    epoch = int((tr["t_claim"] - tr["t_boundary"]).max())
    pre = tr[tr["op"] == 0]
    # each decode-preferring workgroup decides again right after the first of
    # its tiles to end after the release (a tile in flight at the release, or
    # one it claimed at a decision taken just before it)
    rem = []
    for w in range(q):
        m = tr[(tr["wg"] == w) & (tr["t_end"] > R)]
        if len(m):
            rem.append(int(m["t_end"].min()) - R)
    seen, ready = int(st["t_seen"][1]), int(st["t_ready"][1])
    first = int(tr[tr["op"] == 1]["t_start"].min())
    us = lambda t: t * TICK_NS / 1000.0  # noqa: E731
    print(f"release {release_us} us: seen +{us(seen - R):.1f} us (bound {us(min(rem) + epoch):.1f}), activated "
          f"in {us(ready - seen):.1f} us, first tile +{us(first - ready):.1f} us after (epoch {us(epoch):.1f}); "
          f"wait {us(first - R):.1f} us, longest prefill tile {us(int((pre['t_end'] - pre['t_start']).max())):.1f} us")
    assert seen >= R
    assert seen - R <= min(rem) + epoch
    assert ready == seen
    assert first - ready <= epoch
    # the first decode tile ran on the workgroup that activated the op, or on another below q'
    fd = tr[(tr["op"] == 1)]
    assert fd[np.argmin(fd["t_start"])]["wg"] < q


def test_results_independent_of_schedule(dev):
    cfg = _mixed_cfg()
    outs = []
    for kw in (dict(), dict(decode_quota_wg=0), dict(decode_quota_wg=256, decode_quota_max_wg=256),
               dict(n_workgroups=24)):
        specs, _, _ = layer_specs(cfg, 0, dev, decode=dict(release_after_ns=3_000))
        pipe = _pipe(dev, specs, **kw)
        assert pipe.statuses() == (0, 0)
        outs.append([b.y.view(torch.int16).cpu().numpy().copy() for b in pipe.bufs])
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("n_ops,n_wg", [(16, 0), (16, 24), (2, 0)])
def test_every_op_finished_when_workgroups_leave_early(dev, n_ops, n_wg):
    """Workgroups leave as soon as every op is activated and every queue is
    empty; an op whose last commit no polling workgroup saw must still be
    finished (done word, statistics) by the workgroup that committed it."""
    cfg = custom_config(2, cfg_id=402, H=256, I=256, prefill_tokens=96, decode_tokens=32, E_global=16,
                        E_local=8, top_k=2, n_layers=n_ops // 2, zipf_s=(1.1, 0.7))
    specs = []
    for layer in range(n_ops // 2):
        s, _, _ = layer_specs(cfg, layer, dev)
        specs += s
    for _ in range(3):
        pipe = _pipe(dev, specs, n_workgroups=n_wg, trace_capacity=1 << 16)
        assert pipe.statuses() == (0, 0)
        st = pipe.op_stats()
        for i in range(len(specs)):
            xm, ntiles = _tiles_per_op(pipe, i)
            assert int(pipe.bufs[i].done_word.item()) == 1, i
            assert st["x_moe"][i] == xm and st["n_tiles"][i] == ntiles and st["t_done"][i] > 0, i


def test_adaptive_quota_eq4(dev):
    cfg = _mixed_cfg()
    specs, _, _ = layer_specs(cfg, 0, dev)
    pipe = _pipe(dev, specs, decode_quota_wg=64, x_moe_expected=4, decode_quota_max_wg=128, round_multiple=8)
    st = pipe.op_stats()
    xm = int(st["x_moe"][1])
    assert st["quota"][1] == oracle.decode_quota(64, xm, 4, 128, 8)


def test_abort_word_stops_the_kernel(dev):
    cfg = _mixed_cfg()
    abort = torch.ones(1, dtype=torch.int32, device=dev)
    specs, _, _ = layer_specs(cfg, 0, dev)
    pipe = _pipe(dev, specs, abort_word=abort)
    assert pipe.statuses()[1] == -5


def test_never_released_op_times_out(dev):
    cfg = _mixed_cfg()
    never = torch.zeros(1, dtype=torch.int32, device=dev)
    specs, _, _ = layer_specs(cfg, 0, dev, decode=dict(release_word=never))
    pipe = _pipe(dev, specs, spin_limit=20000, trace_capacity=1 << 16)
    assert pipe.statuses()[1] == -6
    st = pipe.op_stats()
    assert st["t_done"][0] > 0                                 # the released prefill op still completed
    assert st["t_ready"][1] == 0


def test_release_word_set_before_launch(dev):
    cfg = _mixed_cfg()
    word = torch.ones(1, dtype=torch.int32, device=dev)
    specs, lay, _ = layer_specs(cfg, 0, dev, decode=dict(release_word=word))
    pipe = _pipe(dev, specs)
    assert pipe.statuses() == (0, 0)
    assert int(pipe.bufs[1].done_word.item()) == 1 and int(pipe.bufs[0].done_word.item()) == 1


def test_static_partition_never_borrows(dev):
    """The comparison mode of a static split: decode tiles run only on
    workgroups below q, prefill tiles only on the others, even while one side
    idles; results stay bitwise those of tile-level sharing."""
    cfg = _mixed_cfg()
    specs, _, _ = layer_specs(cfg, 0, dev, decode=dict(release_after_ns=3_000))
    shared = _pipe(dev, specs, decode_quota_wg=64)
    want = [b.y.view(torch.int16).cpu().numpy().copy() for b in shared.bufs]
    specs, _, _ = layer_specs(cfg, 0, dev, decode=dict(release_after_ns=3_000))
    pipe = _pipe(dev, specs, decode_quota_wg=64, static_partition=True, trace_capacity=1 << 16)
    assert pipe.statuses() == (0, 0)
    tr = pipe.trace_records()
    assert tr[tr["op"] == 1]["wg"].max() < 64
    assert tr[tr["op"] == 0]["wg"].min() >= 64
    for b, w in zip(pipe.bufs, want):
        np.testing.assert_array_equal(b.y.view(torch.int16).cpu().numpy(), w)


def test_fused_combine_tiles_follow_gemm_and_precede_dependants(dev):
    """With a fused combine, each op's combine tiles (trace stage 3, row-block
    field = tile index) run exactly once each, none is claimed before the op's
    last GEMM tile committed, the op's t_done follows its last combine tile,
    and the next layer of the same phase starts only after that."""
    from paper_2607_18002_amd.pipeline import MoEPipeline
    cfg = custom_config(2, cfg_id=731, H=512, I=512, prefill_tokens=900, decode_tokens=70, E_global=64, E_local=12,
                        top_k=6, zipf_s=(1.1,), n_layers=2)
    specs, _, _ = layer_specs(cfg, 0, dev)                      # op 0 prefill, op 1 decode
    s1, _, _ = layer_specs(cfg, 1, dev, prefill=dict(depends_on_op=0), decode=dict(depends_on_op=1))
    specs += s1
    assert [sp.depends_on_op for sp in specs] == [-1, -1, 0, 1]
    pipe = MoEPipeline(specs, fused_gather=True, fused_combine=True, trace_capacity=1 << 16)
    pipe.run()
    torch.cuda.synchronize()
    assert pipe.statuses() == (0, 0)
    tr, st = pipe.trace_records(), pipe.op_stats()
    for o, b in enumerate(pipe.bufs):
        m = tr[tr["op"] == o]
        comb, gemm = m[m["stage"] == 3], m[m["stage"] != 3]
        n3 = (b.T + 31) // 32
        assert sorted(comb["mblk"].tolist()) == list(range(n3))
        if len(gemm):
            assert comb["t_claim"].min() >= gemm["t_end"].max()
        assert int(st["t_done"][o]) >= int(comb["t_end"].max())
        dep = specs[o].depends_on_op
        if dep >= 0:
            assert m["t_claim"].min() >= int(st["t_done"][dep])


@pytest.mark.parametrize("fused_combine", [False, True])
def test_templates_built_ahead_then_activated(dev, fused_combine):
    """Ops whose inputs are in place at the launch and that wait for a
    dependency or a release time are built ahead and then activated by one
    transition of their state word: seen and ready at the same tick, no
    earlier than their release condition allows.  An op with no local rows
    finishes at its activation (with a fused combine: after its combine
    tiles, which write zeros) and releases its dependant; an op with a
    release word is instantiated after its release, as before.  Outputs are
    bitwise those of the same ops all ready at the launch."""
    cfg = custom_config(2, cfg_id=732, H=512, I=512, prefill_tokens=1024, decode_tokens=96, E_global=64,
                        E_local=12, top_k=4, zipf_s=(1.1,), n_layers=3)
    word = torch.ones(1, dtype=torch.int32, device=dev)

    def build(chained):
        specs = []
        for layer in range(3):
            ready = {"prefill": {}, "decode": {}}
            if chained:
                ready["prefill"] = dict(depends_on_op=-1 if layer == 0 else 2 * (layer - 1))
                ready["decode"] = (dict(release_after_ns=15_000) if layer == 0 else
                                   dict(depends_on_op=2 * layer - 1, gap_ns=10_000))
                if layer == 2:
                    ready["decode"]["release_word"] = word
            s, _, _ = layer_specs(cfg, layer, dev, **ready)
            specs += s
        # layer 1's decode op routes no token to a local expert: no row tiles
        lg = specs[3].logits.clone()
        lg[:, cfg.local_begin:cfg.local_begin + cfg.E_local] = -50.0
        specs[3].logits = lg
        from paper_2607_18002_amd.pipeline import MoEPipeline
        p = MoEPipeline(specs, fused_gather=True, fused_combine=fused_combine, trace_capacity=1 << 16)
        p.run()
        torch.cuda.synchronize()
        assert p.statuses() == (0, 0)
        return specs, p

    base_specs, base = build(False)
    specs, pipe = build(True)
    st = pipe.op_stats()
    t0 = pipe.kernel_t0()
    assert st["x_moe"][3] == 0 and st["x_moe"][1] > 0
    for o, sp in enumerate(specs):
        assert int(pipe.bufs[o].done_word.item()) == 1, o
        seen, ready = int(st["t_seen"][o]), int(st["t_ready"][o])
        if o == 0:
            continue                                          # ready at the launch: instantiated
        if sp.release_word is not None:
            assert ready > seen, o                            # built only after its release
        else:
            assert ready == seen, o                           # built ahead, activated in one transition
        if sp.release_after_ns >= 0:
            assert ready >= t0 + int(sp.release_after_ns / TICK_NS), o
        if sp.depends_on_op >= 0:
            assert ready >= int(st["t_done"][sp.depends_on_op]) + int(sp.gap_ns / TICK_NS), o
        assert int(st["t_done"][o]) >= ready, o
    if not fused_combine:                                       # (with a fused combine its tiles write zeros)
        assert int(st["t_done"][3]) - int(st["t_ready"][3]) < 2000  # the empty op finished at its activation
    for b0, b1 in zip(base.bufs, pipe.bufs):
        np.testing.assert_array_equal(b1.y.view(torch.int16).cpu().numpy(), b0.y.view(torch.int16).cpu().numpy())


# Queue words of the scheduler workspace: a 256-byte header, 16 op states and
# 16 op statics of 128 bytes, then one 128-byte queue per (op, XCD) holding
# claim, size, first row tile and row-tile count.
_XQ_OFF = 256 + 16 * 128 + 16 * 128


@pytest.mark.parametrize("zipf", [0.6, 1.1, 1.6])
def test_queue_ranges_match_host_layout(dev, zipf):
    """The device's per-XCD queue ranges (cut between weight-sharing groups,
    nearest to each eighth of the row tiles) equal the host build of the same
    index functions, for both phases of a mixed launch."""
    from paper_2607_18002_amd import ops
    cfg = custom_config(2, cfg_id=402, H=512, I=512, prefill_tokens=3000, decode_tokens=300, E_global=64,
                        E_local=32, top_k=8, zipf_s=(zipf,))
    specs, lay, _ = layer_specs(cfg, 0, dev)
    pipe = _pipe(dev, specs)
    assert pipe.statuses() == (0, 0)
    ws = pipe.ffn_ws.cpu().numpy()
    for i, b in enumerate(pipe.bufs):
        bm, bn, _ = ops.moe_ffn_tile_shape(b.spec.phase, b.spec.weights.dtype)
        n1, n2 = b.spec.weights.I // (bn // 2), b.spec.weights.H // bn
        counts, offsets = b.counts.cpu().numpy(), b.offsets.cpu().numpy()
        _, _, qu, _ = ops.moe_sched_layout(counts, offsets[:-1], bm, 8, n1, n2)
        dq = ws[_XQ_OFF + i * 8 * 128: _XQ_OFF + (i + 1) * 8 * 128].view(np.int32).reshape(8, 32)
        np.testing.assert_array_equal(dq[:, 2], qu[:, 0])
        np.testing.assert_array_equal(dq[:, 3], qu[:, 1])
        np.testing.assert_array_equal(dq[:, 1], qu[:, 1] * (n1 + n2))
