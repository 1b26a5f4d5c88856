"""The entry points only launch kernels on the caller's stream (no host
synchronisation, no allocation or memset after a first call on a device), so
they can be captured in a HIP graph.  Each graph is replayed several times,
with eager work and synchronisation between replays, and every replay must
equal the eager result bit for bit."""
import pytest

import workloads
from gpu_util import log, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def api():
    import torch

    assert torch.cuda.is_available()
    from paper_2609_32237_amd import torch_api

    return torch_api


def replay_matches(fn, out):
    import torch

    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        for _ in range(2):
            fn()  # first calls build the per-device tables
    torch.cuda.synchronize()
    ref = out.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        fn()
    torch.cuda.synchronize()
    for rep in range(4):
        out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.float32), ref.view(torch.float32)), rep
        fn()  # eager work between replays
        torch.cuda.synchronize()


def test_fft_plan_in_a_graph(api):
    import torch

    log("graph: fft rows and columns")
    x = to_dev(workloads.uniform_complex(64, 4096, 31))
    y = torch.empty_like(x)
    p = api.Plan(4096, 64, 1, 4096, 0, -1)
    replay_matches(lambda: p.execute(x, y), y)
    p.close()
    xc = x.view(4096, 64)
    yc = torch.empty_like(xc)
    pc = api.Plan(4096, 64, 64, 1, 0, 1)
    replay_matches(lambda: pc.execute(xc, yc), yc)
    pc.close()


def test_sar_chain_in_a_graph(api):
    import torch

    from paper_2609_32237_amd import _lib

    log("graph: sar chain")
    sc = workloads.sar_scene(n_az=1024, n_rg=2048, n_targets=4, len_rg=256, beta_rg=0.8, len_az=128,
                             beta_az=0.8, seed=77, min_sep=24)
    raw, hr, ha = to_dev(sc.raw), to_dev(sc.range_ref), to_dev(sc.az_ref)
    img = torch.empty_like(raw)
    ws = torch.empty(_lib.sar_workspace_bytes(1024, 2048, 0), dtype=torch.uint8, device="cuda")
    replay_matches(lambda: api.sar_form_image(raw, hr, ha, 0, out=img, workspace=ws), img)


def test_range_doppler_chain_in_a_graph(api):
    import torch

    from paper_2609_32237_amd import _lib

    log("graph: range-Doppler chain")
    sc = workloads.rd_scene_small()
    raw, ref = to_dev(sc.raw), to_dev(sc.range_ref)
    img = torch.empty_like(raw)
    ws = torch.empty(_lib.sar_rd_workspace_bytes(1024, 1024, 1), dtype=torch.uint8, device="cuda")
    replay_matches(lambda: api.sar_rd_form_image(raw, ref, sc.geometry, 1, out=img, workspace=ws), img)


def test_square_sar_chain_in_a_graph_with_new_references(api):
    """A square image's range pass computes both reference spectra in its
    first workgroups and publishes the range spectrum to its own workgroups
    through a flag in the workspace, which the azimuth pass clears.  Replays of
    one captured chain (one flag value) with the references rewritten between
    them must equal eager calls on the same inputs, bit for bit."""
    import torch

    from paper_2609_32237_amd import _lib

    log("graph: square sar chain, references rewritten between replays")
    n = 2048
    sc1 = workloads.sar_scene(n_az=n, n_rg=n, n_targets=4, len_rg=256, beta_rg=0.8, len_az=128, beta_az=0.8,
                              seed=78, min_sep=24)
    sc2 = workloads.sar_scene(n_az=n, n_rg=n, n_targets=4, len_rg=320, beta_rg=0.6, len_az=96, beta_az=0.5,
                              seed=78, min_sep=24)
    raw, hr, ha = to_dev(sc1.raw), to_dev(sc1.range_ref), to_dev(sc1.az_ref)
    refs = [(to_dev(sc1.range_ref), to_dev(sc1.az_ref)), (to_dev(sc2.range_ref), to_dev(sc2.az_ref))]
    img = torch.empty_like(raw)
    ws = torch.empty(_lib.sar_workspace_bytes(n, n, 0), dtype=torch.uint8, device="cuda")
    s = torch.cuda.Stream()
    expect = []
    for r_rg, r_az in refs:
        hr.copy_(r_rg)
        ha.copy_(r_az)
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            api.sar_form_image(raw, hr, ha, 0, out=img, workspace=ws)
        torch.cuda.synchronize()
        expect.append(img.clone())
    assert not torch.equal(expect[0], expect[1])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        api.sar_form_image(raw, hr, ha, 0, out=img, workspace=ws)
    torch.cuda.synchronize()
    for rep in range(6):
        k = rep % 2
        hr.copy_(refs[k][0])
        ha.copy_(refs[k][1])
        img.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(img.view(torch.float32), expect[k].view(torch.float32)), rep
