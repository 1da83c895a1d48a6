"""Kernel-level parity of the row GEMM (every tile shape, split-K, each epilogue)
against a float32 PyTorch reference of the same operation."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from paper_2505_20600_amd import maskstep as MS

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TILES = [(256, 256), (256, 192), (192, 192), (256, 128), (128, 128), (128, 64), (64, 128), (64, 64)]
# every deeper stage variant the library builds (tile, stages); the forced-tile
# tests above run two stages
STAGED = [((192, 192), 3), ((256, 128), 3), ((128, 128), 3), ((128, 128), 4), ((128, 64), 3), ((128, 64), 4),
          ((64, 128), 3), ((64, 128), 4), ((64, 64), 3), ((64, 64), 4)]


def _ref(A, W, b, R, epi):
    y = A.float() @ W.float().t() + b.float()
    if epi == MS.MS_EPI_BIAS_RESID:
        y = y + R.float()
    if epi == MS.MS_EPI_BIAS_GELU:
        y = F.gelu(y)
    return y


def _err(got, ref):
    return float((got.float() - ref).abs().max() / ref.abs().max())


@pytest.mark.parametrize("tile", TILES, ids=lambda t: f"{t[0]}x{t[1]}")
@pytest.mark.parametrize("epi", [MS.MS_EPI_BIAS, MS.MS_EPI_BIAS_RESID, MS.MS_EPI_BIAS_GELU],
                         ids=["bias", "resid", "gelu"])
def test_linear_tiles_match_fp32_reference(tile, epi):
    g = torch.Generator(device=DEV).manual_seed(hash((tile, epi)) % 1000)
    M, N, K = 300, 516, 320          # ragged in M and N for every tile shape
    A = torch.randn(M, K, device=DEV, generator=g).bfloat16()
    W = (torch.randn(N, K, device=DEV, generator=g) * 0.05).bfloat16()
    b = (torch.randn(N, device=DEV, generator=g) * 0.05).bfloat16()
    R = torch.randn(M, N, device=DEV, generator=g).bfloat16()
    out = torch.empty(M, N, device=DEV, dtype=torch.bfloat16)
    MS.ms_linear(A, W, b, out, resid=R, epilogue=epi, tile=tile, ksplit=1)
    torch.cuda.synchronize()
    e = _err(out, _ref(A, W, b, R, epi))
    print(f"[parity] tile {tile} epi {epi}: max-norm rel err {e:.2e}")
    assert e <= 2e-2


@pytest.fixture
def stage_override():
    """Sets MS_GEMM_STAGES for one test (the library reads it at every launch)."""
    import os
    old = os.environ.get("MS_GEMM_STAGES")
    yield lambda n: os.environ.__setitem__("MS_GEMM_STAGES", str(n))
    if old is None:
        os.environ.pop("MS_GEMM_STAGES", None)
    else:
        os.environ["MS_GEMM_STAGES"] = old


@pytest.mark.parametrize("tile,stages", STAGED, ids=lambda v: f"{v[0]}x{v[1]}" if isinstance(v, tuple) else f"s{v}")
@pytest.mark.parametrize("shape", [(300, 516, 320), (4100, 3000, 704)], ids=["ragged", "persistent"])
def test_linear_stage_variants_match_fp32_reference(tile, stages, shape, stage_override):
    """Each multi-stage main loop: ragged edges, K steps fewer and more than
    the stages, and (second shape) more tiles than resident workgroups."""
    stage_override(stages)
    g = torch.Generator(device=DEV).manual_seed(hash((tile, stages, shape)) % 1000)
    M, N, K = shape
    A = torch.randn(M, K, device=DEV, generator=g).bfloat16()
    W = (torch.randn(N, K, device=DEV, generator=g) * 0.05).bfloat16()
    b = (torch.randn(N, device=DEV, generator=g) * 0.05).bfloat16()
    R = torch.randn(M, N, device=DEV, generator=g).bfloat16()
    out = torch.empty(M, N, device=DEV, dtype=torch.bfloat16)
    MS.ms_linear(A, W, b, out, resid=R, epilogue=MS.MS_EPI_BIAS_RESID, tile=tile, ksplit=1)
    torch.cuda.synchronize()
    e = _err(out, _ref(A, W, b, R, MS.MS_EPI_BIAS_RESID))
    print(f"[parity] tile {tile} stages {stages} {shape}: max-norm rel err {e:.2e}")
    assert e <= 2e-2


@pytest.mark.parametrize("ksplit", [2, 3, 5])
def test_linear_split_k_matches_unsplit(ksplit):
    g = torch.Generator(device=DEV).manual_seed(ksplit)
    M, N, K = 200, 768, 1280
    A = torch.randn(M, K, device=DEV, generator=g).bfloat16()
    W = (torch.randn(N, K, device=DEV, generator=g) * 0.03).bfloat16()
    b = (torch.randn(N, device=DEV, generator=g) * 0.03).bfloat16()
    R = torch.randn(M, N, device=DEV, generator=g).bfloat16()
    ws = torch.empty(ksplit * M * N * 4, device=DEV, dtype=torch.uint8)
    out = torch.empty(M, N, device=DEV, dtype=torch.bfloat16)
    MS.ms_linear(A, W, b, out, resid=R, epilogue=MS.MS_EPI_BIAS_RESID, tile=(0, 0), ksplit=ksplit, workspace=ws)
    torch.cuda.synchronize()
    e = _err(out, _ref(A, W, b, R, MS.MS_EPI_BIAS_RESID))
    print(f"[parity] split-K {ksplit}: max-norm rel err {e:.2e}")
    assert e <= 2e-2


def test_linear_large_planned_shape():
    """A c5-sized projection (planner picks the big tiles)."""
    g = torch.Generator(device=DEV).manual_seed(7)
    M, N, K = 3000, 3072, 3072
    A = torch.randn(M, K, device=DEV, generator=g).bfloat16()
    W = (torch.randn(N, K, device=DEV, generator=g) * 0.02).bfloat16()
    b = (torch.randn(N, device=DEV, generator=g) * 0.02).bfloat16()
    out = torch.empty(M, N, device=DEV, dtype=torch.bfloat16)
    MS.ms_linear(A, W, b, out)
    torch.cuda.synchronize()
    e = _err(out, _ref(A, W, b, None, MS.MS_EPI_BIAS))
    print(f"[parity] planned large GEMM: max-norm rel err {e:.2e}")
    assert e <= 2e-2


def test_linear_fp32_matches_reference():
    g = torch.Generator(device=DEV).manual_seed(3)
    M, N, K = 130, 260, 96
    A = torch.randn(M, K, device=DEV, generator=g)
    W = torch.randn(N, K, device=DEV, generator=g) * 0.1
    b = torch.randn(N, device=DEV, generator=g) * 0.1
    out = torch.empty(M, N, device=DEV)
    MS.ms_linear(A, W, b, out, epilogue=MS.MS_EPI_BIAS_GELU)
    torch.cuda.synchronize()
    ref = F.gelu(A.double() @ W.double().t() + b.double())
    e = float((out.double() - ref).abs().max() / ref.abs().max())
    print(f"[parity] fp32 GEMM: max-norm rel err {e:.2e}")
    assert e <= 1e-4


def test_linear_rejects_bad_arguments():
    A = torch.zeros(8, 64, device=DEV, dtype=torch.bfloat16)
    W = torch.zeros(8, 64, device=DEV, dtype=torch.bfloat16)
    b = torch.zeros(8, device=DEV, dtype=torch.bfloat16)
    out = torch.empty(8, 8, device=DEV, dtype=torch.bfloat16)
    with pytest.raises(MS.MaskStepError):
        MS.ms_linear(A, W, b, out, tile=(96, 64))
    with pytest.raises(MS.MaskStepError):
        MS.ms_linear(A, W, b, out, epilogue=MS.MS_EPI_BIAS_RESID)   # no residual given
    with pytest.raises(MS.MaskStepError):
        MS.ms_linear(A, W, b, out, ksplit=2)                          # no workspace


@pytest.mark.parametrize("tile,M,N", [((64, 64), 4096, 2112), ((128, 64), 3000, 2048), ((256, 256), 4608, 4352),
                                      ((128, 64), 8192, 2048), ((256, 256), 16384, 8448)],
                         ids=["64x64", "128x64", "256x256", "128x64-8-per-CU", "256x256-8-per-CU"])
@pytest.mark.parametrize("epi", [MS.MS_EPI_BIAS, MS.MS_EPI_BIAS_RESID, MS.MS_EPI_BIAS_GELU],
                         ids=["bias", "resid", "gelu"])
def test_linear_more_tiles_than_resident_workgroups(tile, M, N, epi):
    """More tiles than the CUs hold at once: each workgroup loops over several tiles,
    loading the next tile's first stages during the current tile's epilogue. With 8
    or more tiles per CU the GELU output is restaged through LDS too."""
    g = torch.Generator(device=DEV).manual_seed(hash((tile, epi, M)) % 1000)
    K = 192
    A = torch.randn(M, K, device=DEV, generator=g).bfloat16()
    W = (torch.randn(N, K, device=DEV, generator=g) * 0.05).bfloat16()
    b = (torch.randn(N, device=DEV, generator=g) * 0.05).bfloat16()
    R = torch.randn(M, N, device=DEV, generator=g).bfloat16()
    out = torch.empty(M, N, device=DEV, dtype=torch.bfloat16)
    MS.ms_linear(A, W, b, out, resid=R, epilogue=epi, tile=tile, ksplit=1)
    torch.cuda.synchronize()
    e = _err(out, _ref(A, W, b, R, epi))
    print(f"[parity] persistent tile {tile} {M}x{N} epi {epi}: max-norm rel err {e:.2e}")
    assert e <= 2e-2


def test_diagnostic_probes_report_plausible_rates():
    """The probes behind bench.py --ceilings: matrix-core rate below the 2.5 PFLOP/s
    nominal dense peak and a clock near the 2.4 GHz nominal, LDS and operand-stream
    rates positive, the direct-to-LDS stream at least as fast as through VGPRs."""
    r = MS.probe_ceilings()
    print("[probe]", r)
    for k, v in r.items():
        assert v > 0, k
    for k in ("mfma_16x16x32_bf16_2wave_tflops", "mfma_32x32x16_bf16_2wave_tflops"):
        assert 500 < r[k] < 2600, k
    assert 1.0 < r["mfma_16x16x32_bf16_2wave_clock_ghz"] < 3.0
    assert r["operand_stream_to_lds_tbs"] >= 0.9 * r["operand_stream_to_vgprs_tbs"]
    # a failed call's message does not outlive a later successful probe
    import ctypes as C
    lib = MS.load()
    tb = C.c_double()
    assert lib.mask_probe_lds(None) == MS.MS_EINVAL and lib.mask_last_error()
    assert lib.mask_probe_lds(C.byref(tb)) == MS.MS_OK and lib.mask_last_error() == b""
