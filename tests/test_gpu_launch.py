"""GPU checks of what changes the render kernel's speed but never its result:
the tile order (stripes of tiles per XCD), the early-termination path (rays
evaluated front to back in rounds, stopped rays dropped), the 16-byte block
gathers of x-neighbour corner pairs on the finest levels, the profiling
builds that time the kernel's phases, and the gather-replay microbenchmark
that measures the floor of its gather stream.

  - every tile order renders the same frame bit for bit, and every pixel;
  - the work counters are back at zero after every launch, whatever the
    kernel and grid size of the next one, and two contexts (each with its
    own counters) render on two streams at once;
  - the early-termination path renders the tile path's frame bit for bit
    (the same samples composited in the same order), at every round size,
    and evaluates fewer samples on opaque content;
  - block gathers on any set of finest levels render the same frame bit for
    bit as single-entry gathers;
  - the phase-timer build renders the same frame as the library, and its
    counters cover every tile of every launch;
  - the replay loads exactly the table entries of the oracle's corner
    indices for the frame's own sample positions (the XOR of everything it
    loads equals the XOR of those entries, which does not depend on which
    lane loaded what).
"""
import numpy as np
import pytest

import oracle
from paper_2312_11841_amd import mixrt, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


def _render(ds, **kw):
    r = mixrt.Renderer(0, sync_check=True, **kw)
    out = torch.full((ds.rays, 4), float("nan"), dtype=torch.float32, device="cuda:0")
    r.render(ds, out)
    shape = r.launch_shape(ds)
    r.sync()
    r.close()
    return out.cpu().numpy(), shape


ORDER_CFGS = [
    synth.VIEW720P_DENSE,
    synth.PAPER720P,
    synth.TINY64_DENSE.replace(name="ragged_views", H=37, W=53, views=3, K=8, gbuf="iid"),
    synth.TINY64_DENSE.replace(name="ragged_k1", H=29, W=71, views=2, K=1, gbuf="iid"),
    synth.TINY64_DENSE.replace(name="ragged_k3", H=23, W=37, views=2, K=3, gbuf="iid"),
]


@pytest.mark.parametrize("cfg", ORDER_CFGS, ids=lambda c: c.name)
def test_tile_order_never_changes_a_pixel(cfg):
    say("tile order", cfg.name)
    sc = synth.make_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    ref, (_, default_stripe) = _render(ds, tile_stripe=-1)
    assert np.all(np.isfinite(ref))
    R = 64 // cfg.K
    seen = {default_stripe}
    for stripe in (1, 2, 3, 8, 16, 37, 1 << 20, 0):
        got, (blocks, st) = _render(ds, tile_stripe=stripe)
        seen.add(st)
        assert np.array_equal(got, ref), (stripe, st)
        for b in ("two", "full"):
            got, _ = _render(ds, tile_stripe=stripe, blocks=b)
            assert np.array_equal(got, ref), (stripe, b)
    say(f"  stripes launched: {sorted(seen)} (tiles of {R} rays)")


def test_work_counters_are_ready_for_every_launch():
    """One context renders frames of different kernels and grid sizes in turn
    (a queue-kernel frame, a ragged frame, a one-sample frame on the tile
    kernel, a frame of 25 tiles on 7 blocks, so in one pool, and a frame
    whose plan takes every unit in the fixed order), twice over: the pools'
    counters, left at zero by each launch's last blocks, give every later
    launch the same frame as a fresh context's first launch."""
    cfgs = [synth.VIEW720P, ORDER_CFGS[4], synth.PAPER720P,
            synth.TINY64_DENSE.replace(name="one_pool", H=5, W=37, views=1, K=8, gbuf="iid"),
            _table3("tab3_L1_T17")]
    scenes = [mixrt.DeviceScene.from_scene(synth.make_scene(c), "cuda:0") for c in cfgs]
    refs = [_render(ds)[0] for ds in scenes]
    r = mixrt.Renderer(0, sync_check=True)
    try:
        for rep in range(2):
            for cfg, ds, ref in zip(cfgs, scenes, refs):
                plan = r.launch_plan(ds)
                say("counters", rep, cfg.name, plan)
                if cfg.name == "one_pool":
                    assert plan["blocks"] == 7
                assert plan["claims"] == (0 if cfg.name == "tab3_L1_T17" else 1)
                out = torch.full((ds.rays, 4), float("nan"), dtype=torch.float32,
                                 device="cuda:0")
                r.render(ds, out)
                r.sync()
                assert np.array_equal(out.cpu().numpy(), ref), (rep, cfg.name)
    finally:
        r.close()


def test_contexts_on_two_streams_render_at_once():
    """Two contexts, each with its own work counters, render on two streams
    at the same time (launches alternate between the streams with no wait in
    between): every frame equals a lone context's."""
    cfgs = [synth.VIEW720P, synth.PAPER720P]
    scenes = [mixrt.DeviceScene.from_scene(synth.make_scene(c), "cuda:0") for c in cfgs]
    refs = [_render(ds)[0] for ds in scenes]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    rs = [mixrt.Renderer(0, stream=st) for st in streams]
    outs = [[torch.full((ds.rays, 4), float("nan"), dtype=torch.float32, device="cuda:0")
             for _ in range(3)] for ds in scenes]
    try:
        torch.cuda.synchronize()
        for rep in range(3):
            for r, ds, o in zip(rs, scenes, outs):
                r.render(ds, o[rep])
        torch.cuda.synchronize()
        for cfg, ref, o in zip(cfgs, refs, outs):
            for rep in range(3):
                say("two streams", cfg.name, rep)
                assert np.array_equal(o[rep].cpu().numpy(), ref), (cfg.name, rep)
    finally:
        for r in rs:
            r.close()


def test_tile_order_spot_check_against_the_oracle():
    cfg = ORDER_CFGS[2]
    sc = synth.make_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    got, _ = _render(ds, tile_stripe=3)
    ref = oracle.OracleScene(sc).render_pixels(np.arange(cfg.rays), threads=oracle.max_threads())
    assert np.abs(got - ref).max() <= 2e-3


@pytest.mark.parametrize("cfg", [synth.VIEW720P, synth.PAPER720P], ids=lambda c: c.name)
def test_phase_timer_build_renders_the_same_frame(cfg):
    say("timer build", cfg.name)
    sc = synth.make_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    ref, (blocks, stripe) = _render(ds)
    r = mixrt.Renderer(0, sync_check=True, variant="timer")
    r.phase_cycles(reset=True)
    out = torch.full((ds.rays, 4), float("nan"), dtype=torch.float32, device="cuda:0")
    for _ in range(3):
        r.render(ds, out)
    ph = r.phase_cycles(reset=True)
    assert r.launch_shape(ds) == (blocks, stripe)
    r.close()
    assert np.array_equal(out.cpu().numpy(), ref)
    R = 64 // cfg.K
    say("  ", ph)
    assert ph["waves"] == 3 * blocks * 4
    assert ph["tiles"] == 3 * ds.rays // R   # whole tiles: W and H are multiples of the tile's
    assert all(ph[k] > 0 for k in ("setup", "hash", "mlp", "composite"))


def test_default_library_has_no_phase_timer():
    r = mixrt.Renderer(0)
    with pytest.raises(mixrt.MixrtError) as e:
        r.phase_cycles()
    assert e.value.status == mixrt.MIXRT_EUNSUPPORTED
    r.close()


@pytest.mark.parametrize("cfg", [synth.TINY64_DENSE.replace(name="replay_tiny", H=40, W=56),
                                 synth.VIEW720P.replace(name="replay_720p_rows", rows=48),
                                 synth.DEPLOYED720P.replace(name="replay_f4", rows=64),
                                 synth.TABLE3[0].replace(name="replay_f4_L8", rows=48),
                                 synth.TABLE3[0].replace(name="replay_f4_ragged", H=23, W=37,
                                                         views=2, K=3, gbuf="iid", delta=0.5,
                                                         log2_T=12)],
                         ids=lambda c: c.name)
def test_gather_replay_loads_exactly_the_corner_entries(cfg):
    from paper_2312_11841_amd import microbench as mb
    say("gather replay", cfg.name)
    sc = synth.make_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    r = mixrt.Renderer(0, sync_check=True)
    x, hit = r.ray_setup(ds)
    blocks, stripe = r.launch_shape(ds)
    r.sync()
    N = np.ascontiguousarray(mixrt.level_resolutions(ds.grid), np.int32)
    # the XOR over every lane's fold is the XOR over all loaded words,
    # whichever lane loaded them
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    for grid in (blocks, 2 * cus):
        for st in (stripe, 1):
            res = mb.gather_replay(x, hit, cfg.views, cfg.W, cfg.rows_kept, cfg.K, ds.table, N,
                                   st, [grid], reps=1)
            assert res["best"]["ms"] > 0
    xs = x.cpu().numpy().reshape(-1, cfg.K, 3)[hit.cpu().numpy() != 0].reshape(-1, 3)
    _, idx, _, _ = oracle.hash_encode(xs, sc.table, cfg.N_min, cfg.N_max)
    words = sc.table.view(np.uint32).reshape(cfg.L, cfg.T, -1)      # an entry's 32-bit words
    acc = np.uint32(0)
    for l in range(cfg.L):
        w = words[l][idx[:, l, :].reshape(-1)]
        acc ^= np.bitwise_xor.reduce(w.reshape(-1))
    # the tile path's order and every rounds order the render can take, with
    # the render's 16-byte block gathers on none, the library's choice, all
    # hashed levels (4- and 8-byte entries; 16-byte ones ignore it)
    plan = r.launch_plan(ds)
    n_dense = int(sum((N.astype(np.int64) + 1) ** 3 <= cfg.T))
    # one work buffer for every call: each call leaves its counters at zero
    work = torch.zeros(mb.WORK_WORDS, dtype=torch.int32, device="cuda:0")
    for block_from in sorted({cfg.L, plan["block_from"], n_dense, 0, max(cfg.L - 3, 0)}):
        for batch in (2, 4):
            # rounds of a power of two samples, as the render takes them
            for chunk in sorted({c for c in (0, 1, cfg.K // 2, cfg.K) if c & (c - 1) == 0}):
              for claims in (True, False):
                sink = torch.zeros(blocks * 256, dtype=torch.int32, device="cuda:0")
                rc = mb.lib().mixrt_mb_gather_replay(
                    x.data_ptr(), hit.data_ptr(), cfg.views, cfg.W, cfg.rows_kept, cfg.K,
                    ds.table.data_ptr(), cfg.L, cfg.log2_T, ds.table.element_size() * cfg.F,
                    N.ctypes.data, stripe, chunk, block_from, batch, 0, blocks,
                    work.data_ptr() if claims else None, sink.data_ptr(), None)
                assert rc == 0
                torch.cuda.synchronize()
                got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
                assert got == acc, (block_from, batch, chunk, claims)
    assert not work.any().item()
    r.close()


def _table3(name):
    return synth.CONFIGS[name]


BLOCK_CFGS = [
    synth.VIEW720P.replace(name="blk_720p_rows", rows=64),
    synth.VIEW720P_DENSE.replace(name="blk_dense_rows", rows=64),
    synth.OPAQUE720P.replace(name="blk_opaque_rows", rows=64),
    synth.VIEW720P.replace(name="blk_k1", K=1, rows=96),
    synth.VIEW720P.replace(name="blk_ragged", H=23, W=37, views=2, K=3, gbuf="iid",
                           delta=0.5, log2_T=12, N_max=2048),
    # 8-byte entries (fp16, F = 4): one query per pixel with the MLP, 8
    # samples per ray (the rounds path), and a ragged frame
    synth.TABLE3[0].replace(name="blk_f4_L8", rows=64),
    synth.TABLE3[0].replace(name="blk_f4_k8", K=8, delta=0.05, rows=32),
    synth.TABLE3[0].replace(name="blk_f4_ragged", H=23, W=37, views=2, K=3, gbuf="iid",
                            delta=0.5, log2_T=12),
]


@pytest.mark.parametrize("cfg", BLOCK_CFGS, ids=lambda c: c.name)
def test_block_gathers_give_the_same_frame(cfg):
    """16-byte block gathers of x-neighbour corner pairs read the same two
    entries as single gathers: every choice of levels renders the same bits,
    on the tile path and in rounds."""
    say("block gathers", cfg.name)
    sc = synth.make_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    ref = None
    seen = set()
    for chunk in (-1, 0):
        for levels in (-1, 0, 1, 3, cfg.L):
            r = mixrt.Renderer(0, sync_check=True, early_stop_chunk=chunk, block_levels=levels)
            seen.add(r.launch_plan(ds)["block_from"])
            out = torch.full((ds.rays, 4), float("nan"), dtype=torch.float32, device="cuda:0")
            r.render(ds, out)
            r.sync()
            r.close()
            got = out.cpu().numpy()
            assert np.isfinite(got).all()
            if ref is None:
                ref = got
            assert np.array_equal(got, ref), (chunk, levels)
    say(f"  first block levels launched: {sorted(seen)}")
    assert len(seen) >= 3


@pytest.mark.parametrize("cfg", [BLOCK_CFGS[1], BLOCK_CFGS[5], BLOCK_CFGS[6]],
                         ids=lambda c: c.name)
def test_block_gathers_spot_check_against_the_oracle(cfg):
    say("block gathers against the oracle", cfg.name)
    sc = synth.make_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    r = mixrt.Renderer(0, sync_check=True, block_levels=cfg.L)
    assert r.launch_plan(ds)["block_from"] < cfg.L
    got = r.render(ds).cpu().numpy()
    r.close()
    pix = np.random.default_rng(5).choice(cfg.rays, 2000, replace=False)
    ref = oracle.OracleScene(sc).render_pixels(pix, threads=oracle.max_threads())
    assert np.abs(got[pix] - ref).max() <= 2e-3


@pytest.mark.parametrize("cfg", [synth.VIEW720P, synth.VIEW720P_DENSE,
                                 synth.VIEW720P_DENSE.replace(name="d05", delta=0.05),
                                 synth.VIEW720P.replace(name="k2", K=2),
                                 synth.VIEW720P.replace(name="k3", K=3),
                                 synth.BATCH8X1080P, synth.PAPER720P],
                         ids=lambda c: c.name)
def test_default_round_size_follows_the_rule(cfg):
    """The library's default samples per round (0 = the tile path): 4 when a
    ray's samples share the voxels of half the levels and a level fits one
    XCD's L2, 2 or 1 as they share fewer, the tile path for K < 4 or K not a
    power of two and for coherent samples on levels larger than the L2."""
    want = {"view720p": 4, "view720p_dense": 1, "d05": 2, "k2": 0, "k3": 0,
            "batch8x1080p": 0, "paper720p": 0}[cfg.name]
    sc = synth.make_scene(cfg.replace(H=16, W=64, views=1))
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    r = mixrt.Renderer(0)
    assert r.launch_shape(ds, chunk=True)[2] == want
    r.close()


@pytest.mark.parametrize("cfg", [synth.VIEW720P, synth.VIEW720P_DENSE,
                                 synth.VIEW720P.replace(name="k1", K=1),
                                 synth.VIEW720P.replace(name="fine_spacing", delta=1e-4),
                                 synth.BATCH8X1080P, synth.BATCH8X1080P.replace(name="batch_k4", K=4),
                                 synth.PAPER720P, synth.DEPLOYED720P, synth.TABLE3[0],
                                 _table3("tab3_L8_T5"),
                                 _table3("tab3_L16_T17").replace(name="tab3_L16")],
                         ids=lambda c: c.name)
def test_default_gather_plan_follows_the_rule(cfg):
    """4-byte entries: block gathers on the three finest levels (five in
    rounds of one sample per ray; when a level's table exceeds one XCD's L2:
    four, and eight at K >= 8) among hashed levels finer than the sample
    spacing.  8-byte (fp16 F = 4)
    entries: on every hashed level when there are 8 or more of them in tables
    of 2^10 or more entries.  Batches of 4 hashed levels only for entries of
    8+ bytes when that covers every hashed level."""
    want = {"view720p": (13, 2), "view720p_dense": (11, 2), "k1": (13, 2),
            "fine_spacing": (16, 2), "batch8x1080p": (8, 2), "batch_k4": (12, 2),
            "paper720p": (4, 4), "deployed720p": (4, 4), "tab3_L8_T17_mlp": (0, 2),
            "tab3_L8_T5": (8, 2), "tab3_L16": (0, 2)}[cfg.name]
    sc = synth.make_scene(cfg.replace(H=16, W=64, views=1))
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    r = mixrt.Renderer(0)
    plan = r.launch_plan(ds)
    r.close()
    assert (plan["block_from"], plan["hash_batch"]) == want, plan


@pytest.mark.parametrize("cfg", [synth.VIEW720P, synth.PAPER720P, synth.BATCH8X1080P,
                                 _table3("tab3_L8_T17_mlp"), _table3("tab3_L1_T17"),
                                 _table3("tab3_L4_T17"), _table3("tab3_L8_T5")],
                         ids=lambda c: c.name)
def test_default_claims_follow_the_rule(cfg):
    """The last units are claimed from the work counters when a unit's work
    hides a claim's latency: with an MLP, or with 8 or more levels."""
    want = {"view720p": 1, "paper720p": 1, "batch8x1080p": 1, "tab3_L8_T17_mlp": 1,
            "tab3_L1_T17": 0, "tab3_L4_T17": 0, "tab3_L8_T5": 1}[cfg.name]
    sc = synth.make_scene(cfg.replace(H=16, W=64, views=1))
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    r = mixrt.Renderer(0)
    plan = r.launch_plan(ds)
    r.close()
    assert plan["claims"] == want, plan


QUEUE_CFGS = [
    synth.TINY64_DENSE.replace(name="q_tiny_dense", t_term=1e-2),
    synth.TINY64_DENSE.replace(name="q_ragged_k3", H=23, W=37, views=2, K=3, gbuf="iid",
                               t_term=1e-2),
    synth.TINY64_DENSE.replace(name="q_ragged_k7", H=19, W=21, views=3, K=7, gbuf="iid",
                               t_term=1e-3),
    synth.TINY64_DENSE.replace(name="q_k64", H=9, W=11, K=64, gbuf="iid", t_term=0.0),
    synth.TINY64_DENSE.replace(name="q_k1", H=33, W=31, views=2, K=1, gbuf="iid"),
    synth.TINY64_DENSE.replace(name="q_nomlp", widths=(16,), seed=16, t_term=1e-2),
    synth.TINY64_VEC3, synth.TINY64_U8,
    synth.OPAQUE720P, synth.TRANSLUCENT720P, synth.VIEW720P_DENSE, synth.PAPER720P,
]


@pytest.mark.parametrize("cfg", QUEUE_CFGS, ids=lambda c: c.name)
def test_early_termination_path_renders_the_same_frame(cfg):
    """Every round size renders the tile path's frame bit for bit, misses
    included (5% of each kind on the small workloads)."""
    say("early termination", cfg.name)
    sc = synth.make_scene(cfg)
    if cfg.rays < 20000:
        flat = sc.g0.reshape(-1, 4)
        rng = np.random.default_rng(cfg.seed)
        miss = rng.choice(flat.shape[0], flat.shape[0] // 20, replace=False)
        flat[miss, 0] = rng.choice([0.0, -1.0, np.nan, np.inf], miss.size)
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    ref, _ = _render(ds, early_stop_chunk=-1)
    assert np.all(np.isfinite(ref))
    for chunk in (1, 2, 4, 8, 64):
        got, _ = _render(ds, early_stop_chunk=chunk)
        assert np.array_equal(got, ref), chunk
    got, _ = _render(ds, early_stop_chunk=2, tile_stripe=-1, blocks="two")
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("cfg", [synth.OPAQUE720P, synth.TRANSLUCENT720P],
                         ids=lambda c: c.name)
def test_early_termination_against_the_oracle(cfg):
    """The frame within 2e-3 + t_term of the oracle (which never stops a
    ray) on sampled pixels, and fewer samples evaluated than the tile path
    (counted by the phase-timer build)."""
    say("early termination vs oracle", cfg.name)
    sc = synth.make_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    got, _ = _render(ds, early_stop_chunk=1)
    rng = np.random.default_rng(9)
    pix = np.unique(np.concatenate([rng.choice(cfg.rays, 3000, replace=False),
                                    np.arange(cfg.W)]))
    ref = oracle.OracleScene(sc).render_pixels(pix, threads=oracle.max_threads())
    err = np.abs(got[pix] - ref).max()
    say(f"  max |gpu - oracle| = {err:.3e}")
    assert err <= 2e-3 + cfg.t_term
    counts = {}
    for chunk in (-1, 1, 2, 4):
        r = mixrt.Renderer(0, sync_check=True, variant="timer", early_stop_chunk=chunk)
        r.phase_cycles(reset=True)
        r.render(ds)
        counts[chunk] = r.phase_cycles(reset=True)["samples"]
        r.close()
    say("  samples evaluated by round size:", counts)
    assert counts[-1] == cfg.rays * cfg.K            # every pixel hits
    assert counts[1] < counts[2] <= counts[4] < counts[-1]


def test_gather_lines_microbenchmark():
    """The L1 cost probe behind the block gathers: runs at every width and
    sharing pattern, refuses a line count that does not divide 64, and a
    gather touching 64 lines costs more than one touching 4."""
    from paper_2312_11841_amd import microbench as mb
    t = torch.zeros(16 * 1024 // 4, dtype=torch.int32, device="cuda:0")
    sink = torch.empty(256 * 256, dtype=torch.int32, device="cuda:0")
    assert mb.lib().mixrt_mb_gather_lines(t.data_ptr(), 16 * 1024, 4, 3, 1, 1, 256,
                                          sink.data_ptr(), None) != 0
    assert mb.lib().mixrt_mb_gather_lines(t.data_ptr(), 16 * 1024 + 128, 4, 4, 1, 1, 256,
                                          sink.data_ptr(), None) != 0
    few = mb.gather_lines(16 * 1024, 4, 4, True, iters=32)
    many = mb.gather_lines(16 * 1024, 4, 64, True, iters=32)
    for width in (8, 16):
        assert mb.gather_lines(2048 * 1024, width, 16, False, iters=16) > 0
    say(f"  cycles per gather: 4 lines {few:.1f}, 64 lines {many:.1f}")
    assert many > 2 * few
