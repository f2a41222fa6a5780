"""Parity sweep over seeded random workloads: every render kernel the library
builds, with samples per ray, spacing, table size, level resolutions, views,
ragged image sizes, cameras, misses, background and termination drawn at
random (tests/randcfg.py), each frame compared with the oracle pixel by
pixel through the C ABI."""
import numpy as np
import pytest

import oracle
from paper_2312_11841_amd import mixrt
from randcfg import SEEDS, random_config, random_scene

pytestmark = pytest.mark.gpu

FRAME_TOL = 2e-3


@pytest.fixture(scope="module")
def R():
    r = mixrt.Renderer(0, sync_check=True)
    yield r
    r.close()


@pytest.mark.parametrize("seed", SEEDS)
def test_random_workload_matches_oracle(R, seed):
    cfg = random_config(seed)
    print("random", seed, cfg, flush=True)
    sc = random_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    got = R.render(ds).cpu().numpy().astype(np.float64)
    R.sync()
    ref = oracle.OracleScene(sc).render_pixels(np.arange(cfg.rays), threads=oracle.max_threads())
    assert np.all(np.isfinite(got))
    # the kernel stops a ray once its transmittance is below t_term; the
    # oracle never stops, which moves a pixel by less than t_term
    err = np.abs(got - ref).max()
    print(f"  max |gpu - oracle| = {err:.3e} over {cfg.rays} px", flush=True)
    assert err <= FRAME_TOL + cfg.t_term
    # the other evaluation order (tile path against rounds of a random size)
    # and another choice of block-gathered levels render the same frame bit
    # for bit
    chunk = int(np.random.default_rng(seed).choice([-1, 1, 2, 4, 8, 16]))
    levels = int(np.random.default_rng(seed + 2).choice([-1, 0, 1, 2, cfg.L]))
    r2 = mixrt.Renderer(0, sync_check=True, early_stop_chunk=chunk, block_levels=levels,
                        tile_stripe=int(np.random.default_rng(seed + 1).integers(-1, 9)))
    got2 = r2.render(ds).cpu().numpy().astype(np.float64)
    r2.close()
    assert np.array_equal(got2, got), (chunk, levels)


@pytest.mark.parametrize("seed", list(range(3000, 3024)))
def test_random_grid_hash_encode_bit_exact(R, seed):
    """The hash stage alone on random grids: L, T, F, table dtype and level
    resolutions (dense and hashed levels, N up to 65,536) drawn at random,
    queried at random and adversarial positions; corners and table indices
    bit-exact, weights and features within the stage bars."""
    import torch
    from test_gpu_parity import _adversarial_x
    rng = np.random.default_rng(seed)
    L, F = int(rng.integers(1, 33)), int(rng.choice([2, 4]))
    f16 = bool(rng.random() < 0.5)
    log2_T = int(rng.integers(4, 21))
    while L * (1 << log2_T) * F * 4 > 64 << 20:
        log2_T -= 1
    n_min = int(rng.integers(1, 65))
    n_max = int(min(65536, n_min * np.exp(rng.uniform(0.0, np.log(4096.0)))))
    print("grid", seed, L, log2_T, F, "f16" if f16 else "f32", n_min, n_max, flush=True)
    table = rng.uniform(-1.0, 1.0, (L, 1 << log2_T, F)).astype(np.float16 if f16 else np.float32)
    N = oracle.level_resolutions(L, n_min, n_max)
    x = _adversarial_x(N, rng, 3000 + seed % 61)
    tt = torch.from_numpy(table).cuda()
    grid = mixrt.make_grid(tt, n_min, n_max)
    got = R.hash_encode(grid, torch.from_numpy(x).cuda())
    R.sync()
    corner, idx, w, feat = oracle.hash_encode(x, table, n_min, n_max)
    assert np.array_equal(got["corner"].cpu().numpy(), corner)
    assert np.array_equal(got["idx"].cpu().numpy().view(np.uint32), idx)
    assert np.abs(got["w"].cpu().numpy() - w).max() <= 1e-6
    assert np.abs(got["feat"].cpu().numpy() - feat).max() <= 1e-5
