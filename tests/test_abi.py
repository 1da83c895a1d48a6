"""C-ABI checks that need no GPU: the library loads, exports every function the
headers declare, and rejects bad arguments before touching a device."""
import ctypes as C
import os
import re

import pytest

from paper_2505_20600_amd import maskstep as MS
from paper_2505_20600_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if not fn.endswith(".h"):
            continue
        src = open(os.path.join(ROOT, "include", fn)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        for m in re.finditer(r"^[A-Za-z_][\w \*]*?\b([a-z_][a-z0-9_]*)\s*\(", src, flags=re.M):
            if m.group(1) not in ("if", "while", "for", "return", "sizeof"):
                names.add(m.group(1))
    return names


def test_library_exports_every_declared_function():
    lib = MS.load()
    declared = _declared_functions()
    assert {"mask_step_init", "mask_block_forward", "mask_stack_forward", "cache_prefetch_layer"} <= declared
    for name in declared:
        assert hasattr(lib, name), name
    assert set(MS.EXPORTED) == declared


def test_abi_version():
    assert MS.load().mask_abi_version() == 7


def test_kv_block_of_4_gib_is_rejected():
    """The bf16 attention's 32-bit buffer offsets: T x 2 x d x 2 bytes must stay below 2^32."""
    ok = W.ModelShape("k", 1, 4096, 32, 4, 512, 511, dtype="bf16")      # 4 * 261632 * 4096 < 2^32
    bad = W.ModelShape("k", 1, 4096, 32, 4, 512, 512, dtype="bf16")     # = 2^32
    assert MS.mask_workspace_bytes(MS.model_desc(ok), 1) > 0
    with pytest.raises(MS.MaskStepError) as e:
        MS.mask_workspace_bytes(MS.model_desc(bad), 1)
    assert "4 GiB" in str(e.value)


def test_static_scratch_rejects_before_any_device_work():
    lib = MS.load()
    big = W.CONFIGS["c3"]
    desc = MS.model_desc(big)
    assert MS.mask_workspace_bytes(desc, 1) > MS.STATIC_SCRATCH_BYTES
    h = C.c_void_p()
    assert lib.mask_step_init_static(C.byref(h), C.byref(desc), 1, 16, None) == MS.MS_EWORKSPACE
    assert b"static scratch" in lib.mask_last_error()
    assert lib.mask_step_init_static(None, C.byref(desc), 1, 16, None) == MS.MS_EINVAL
    assert lib.mask_step_init_static(C.byref(h), C.byref(desc), 0, 16, None) == MS.MS_ESHAPE


def _desc(**kw):
    d = MS.model_desc(W.CONFIGS["c2"])
    for k, v in kw.items():
        setattr(d, k, v)
    return d


def test_workspace_bytes_scales_with_batch_and_rejects_bad_shapes():
    lib = MS.load()
    n1 = MS.mask_workspace_bytes(_desc(max_batch=4), 1)
    n4 = MS.mask_workspace_bytes(_desc(max_batch=4), 4)
    # per request: five [T][d] bf16 activation buffers + [T][4d]; the split buffers are shared
    T, d = 4096, 768
    per_request = T * d * 2 * 5 + T * 4 * d * 2
    assert n1 >= per_request
    assert n4 - n1 >= 3 * per_request
    bad = [
        dict(d_model=100), dict(n_heads=5), dict(d_model=768, n_heads=4),   # head_dim 192
        dict(dtype=7), dict(n_layers=0), dict(grid_h=0), dict(max_batch=0), dict(max_batch=65),
        dict(mlp_mult=0), dict(dual_stream=3), dict(n_text=-1), dict(ln_eps=float("nan")),
    ]
    for kw in bad:
        assert lib.mask_workspace_bytes(C.byref(_desc(**kw)), 1) == 0, kw
        assert lib.mask_last_error()
    assert lib.mask_workspace_bytes(C.byref(_desc(max_batch=2)), 3) == 0
    assert lib.mask_workspace_bytes(None, 1) == 0


def test_fp32_limits():
    lib = MS.load()
    d = MS.model_desc(W.CONFIGS["c1"])
    assert lib.mask_workspace_bytes(C.byref(d), 1) > 0
    d.n_heads = 2  # head_dim 128 in fp32: not supported
    assert lib.mask_workspace_bytes(C.byref(d), 1) == 0


def test_step_init_validates_before_any_device_work():
    lib = MS.load()
    desc = _desc()
    h = C.c_void_p()
    ws = 1 << 12
    cases = [
        ((None, C.byref(desc), 1, 16, 16, ws, None), MS.MS_EINVAL),
        ((C.byref(h), None, 1, 16, 16, ws, None), MS.MS_EINVAL),
        ((C.byref(h), C.byref(desc), 0, 16, 16, ws, None), MS.MS_ESHAPE),
        ((C.byref(h), C.byref(desc), 1, None, 16, ws, None), MS.MS_EINVAL),
        ((C.byref(h), C.byref(desc), 1, 16, None, ws, None), MS.MS_EINVAL),
        ((C.byref(h), C.byref(desc), 1, 16, 24, ws, None), MS.MS_EALIGN),
        ((C.byref(h), C.byref(desc), 1, 16, 16, ws, None), MS.MS_EWORKSPACE),
    ]
    for args, want in cases:
        assert lib.mask_step_init(*args) == want, (args, lib.mask_last_error())
        assert h.value is None


def test_probes_validate_before_any_device_work():
    """The diagnostic probes reject bad arguments with MS_EINVAL and a message,
    before any HIP call (so this runs without a GPU)."""
    lib = MS.load()
    tf, ghz, us, tb = C.c_double(), C.c_double(), C.c_double(), C.c_double()
    for args in ((2, 1, C.byref(tf), C.byref(ghz)), (0, 0, C.byref(tf), None), (0, 5, C.byref(tf), None),
                 (1, 1, None, C.byref(ghz))):
        assert lib.mask_probe_mfma(*args) == MS.MS_EINVAL
        assert lib.mask_last_error()
    assert lib.mask_probe_lds(None) == MS.MS_EINVAL
    assert lib.mask_probe_operand_stream(1, None, C.byref(tb)) == MS.MS_EINVAL
    assert lib.mask_probe_operand_stream(0, C.byref(us), None) == MS.MS_EINVAL


def test_linear_validates_before_any_device_work():
    """The row GEMM's shape checks come before any pointer or device use; the
    bf16 kernels address a tile's rows with 32-bit offsets, so K stops below 2^23."""
    lib = MS.load()
    def call(dtype, M, N, K, epi=MS.MS_EPI_BIAS, tile=(0, 0)):
        return lib.ms_linear(dtype, M, N, K, None, None, None, None, None, epi, tile[0], tile[1], 0, None, 0, None)
    assert call(MS.MS_BF16, 16, 6, 64) == MS.MS_ESHAPE            # N not a multiple of 4
    assert call(MS.MS_BF16, 16, 8, 96) == MS.MS_ESHAPE            # K not a multiple of 64
    assert call(MS.MS_BF16, 16, 8, 1 << 23) == MS.MS_ESHAPE
    assert "2^23" in lib.mask_last_error().decode()
    assert call(MS.MS_BF16, 16, 8, (1 << 23) - 64, epi=7) == MS.MS_EINVAL
    assert call(MS.MS_BF16, 16, 8, 64) == MS.MS_EINVAL            # NULL operands
    assert call(7, 16, 8, 64) == MS.MS_EDTYPE


def test_calls_without_a_step_context_fail_cleanly():
    lib = MS.load()
    assert lib.mask_gather_rows(None, 16, 16, None) == MS.MS_ESTATE
    assert lib.mask_block_forward(None, 0, None, 16, 16, None) == MS.MS_ESTATE
    assert lib.mask_scatter_rows(None, 16, 16, 16, None) == MS.MS_ESTATE
    assert lib.cache_prefetch_layer(None, 0, 16, 16, None, None, None) == MS.MS_ESTATE
    assert lib.mask_stack_forward(None, None, 16, 16, None, 16, None, None) == MS.MS_ESTATE
    info = MS.StepInfo()
    assert lib.mask_step_get_info(None, C.byref(info)) == MS.MS_EINVAL
    lib.mask_step_destroy(None)  # no-op


def test_planner_matches_the_oracle_planner():
    """mask_plan_dense_prefix (host-only) against Alg. 1's recurrences evaluated in the oracle."""
    import numpy as np
    import oracle
    g = np.random.default_rng(5)
    for _ in range(300):
        n = int(g.integers(1, 30))
        L, cw = float(g.uniform(0.05, 5)), float(g.uniform(0.01, 2))
        cwo = cw + float(g.uniform(0, 6))
        k, lat = MS.mask_plan_dense_prefix(n, L, cw, cwo)
        k_ref, lat_ref = oracle.best_dense_prefix(n, L, cw, cwo)
        assert k == k_ref
        assert abs(lat - lat_ref) <= 1e-9 * max(1.0, lat_ref)
    with pytest.raises(MS.MaskStepError):
        MS.mask_plan_dense_prefix(0, 1.0, 1.0, 1.0)
    with pytest.raises(MS.MaskStepError):
        MS.mask_plan_dense_prefix(4, -1.0, 1.0, 1.0)


def test_error_message_is_per_call():
    lib = MS.load()
    assert lib.mask_workspace_bytes(C.byref(_desc(d_model=100)), 1) == 0
    assert b"d_model" in lib.mask_last_error()
    assert lib.mask_workspace_bytes(C.byref(_desc()), 1) > 0
    assert lib.mask_last_error() == b""
