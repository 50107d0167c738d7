"""The allocation-free stroke encoding (sscn_encode_strokes_static) against the
workspace entry point (sscn_encode_strokes), through the C interface, on the GPU:
two calls in a row, the second with a smaller input, must give the same site
count, coordinates and features bit for bit (the same kernels on the same
inputs); a problem whose scratch exceeds the fixed size is refused before any
GPU work.
"""

import numpy as np
import pytest
import torch

from tests.gpu_harness import log
from workloads import get_config, make_paths, stroke_paths

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1409_6070_amd import sscn
    sscn.load_library()


def _dev(p):
    d = torch.device("cuda")
    return (torch.tensor(p.points, dtype=torch.int32, device=d).contiguous(),
            torch.tensor(p.stroke_begin, dtype=torch.int32, device=d).contiguous(),
            torch.tensor(p.stroke_sample, dtype=torch.int32, device=d).contiguous())


def _static(p, dtype, max_sites):
    from paper_1409_6070_amd import sscn
    pts, beg, smp = _dev(p)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    coords = torch.full((max(max_sites, 1), 3), -7, dtype=torch.int32, device="cuda")
    feats = torch.full((max(max_sites, 1), 9), -7.0, dtype=tdt, device="cuda")
    n = sscn.sscn_encode_strokes_static(p.grid, sscn.SSCN_BF16 if dtype == "bf16" else sscn.SSCN_F32,
                                        pts.data_ptr() if pts.numel() else None, int(pts.shape[0]), beg.data_ptr(),
                                        smp.data_ptr() if smp.numel() else None, int(smp.shape[0]), p.batch,
                                        coords.data_ptr(), feats.data_ptr(), max_sites, sscn._stream())
    torch.cuda.synchronize()
    return n, coords[:n].cpu().numpy(), feats[:n].float().cpu().numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_static_scratch_encoding_matches_workspace_encoding(dtype):
    from paper_1409_6070_amd.sscn import StrokeEncoder
    cfg = get_config("deepcnet4_20_paths_m9_b100")
    big = make_paths(cfg, 0)
    small = stroke_paths(np.random.default_rng(77), 7, cfg.grid, strokes=(1, 2), points=(2, 9), box=20, sigma=3.0)
    enc = StrokeEncoder(cfg.grid, cfg.batch, cfg.batch * cfg.grid * cfg.grid, dtype)
    for name, p in (("batch 100", big), ("batch 7", small)):
        log(f"[no-alloc] encode {name} {dtype}: {p.n_points} points, {p.n_strokes} strokes")
        c, f = enc.encode(*_dev(p), p.batch)
        torch.cuda.synchronize()
        want_c, want_f = c.cpu().numpy(), f.float().cpu().numpy()
        n, got_c, got_f = _static(p, dtype, enc.max_sites)
        assert n == want_c.shape[0] > 0
        np.testing.assert_array_equal(got_c, want_c)
        np.testing.assert_array_equal(got_f, want_f)


def test_static_scratch_refuses_oversized_problems():
    from paper_1409_6070_amd import sscn
    N, batch, max_sites = 192, 4000, 100000
    assert sscn.sscn_encode_workspace_bytes(N, batch, max_sites) > sscn.ENCODE_STATIC_SCRATCH_BYTES
    log("[no-alloc] oversized problem refused")
    cnt = sscn.ctypes.c_int32(0)
    st = sscn.load_library().sscn_encode_strokes_static(N, 0, None, 0, None, None, 0, batch, None, None, max_sites,
                                                        sscn.ctypes.byref(cnt), None)
    assert sscn.STATUS[st] == "SSCN_ERR_WORKSPACE"
