"""The geometry stage on seeded random triangle soups (tests/randcfg.py):
small, sliver, huge, near-camera and degenerate triangles, random cameras,
image sizes and grid options; both routes (rasterise and ray cast) against
the oracle's brute-force ray casting, with the bars of tests/test_gpu_mesh.py
(exact on unambiguous pixels, valid answers on ambiguous ones)."""
import numpy as np
import pytest

from paper_2312_11841_amd import mixrt
from randcfg import MESH_SEEDS, random_soup
from test_gpu_mesh import METHODS, _check_gbuffer, gbuffer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def R():
    r = mixrt.Renderer(0, sync_check=True)
    yield r
    r.close()


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("seed", MESH_SEEDS)
def test_random_soup_gbuffer(R, seed, method):
    mesh, cams, W, H, grid_res, cpf = random_soup(seed)
    print("soup", seed, method, len(mesh.faces), "faces", W, H, len(cams), "views", grid_res, cpf,
          flush=True)
    dm = mixrt.DeviceMesh(R, mesh, grid_res=grid_res, cells_per_face=cpf)
    g0, g1 = gbuffer(R, method, dm, cams, W, H)
    R.sync()
    _check_gbuffer(mesh, cams, W, H, g0.cpu().numpy().reshape(-1, 4),
                   g1.cpu().numpy().reshape(-1, 4), np.arange(len(cams) * H * W),
                   f"soup {seed}", max_amb=0.1)
    dm.close()
