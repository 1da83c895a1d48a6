"""Thin ctypes binding of ``libmaskstep.so`` (the C ABI in ``include/maskstep.h``).

Argument marshalling only: every step of the path runs in the library's HIP
kernels. Torch tensors are passed by device pointer, streams by their HIP
handle. Loading fails loudly when the library has not been built; there is no
fallback of any kind.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

import torch  # loads torch's HIP runtime first, so the library binds to the same one

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmaskstep.so")

MS_OK, MS_EINVAL, MS_ESHAPE, MS_EDTYPE, MS_EALIGN, MS_ENOTPINNED, MS_EWORKSPACE, MS_ESTATE, MS_EHIP = range(9)
MS_FP32, MS_BF16 = 0, 1
MS_KV_DEVICE, MS_KV_HOST_PINNED, MS_Y_DEVICE, MS_Y_HOST_PINNED = 0, 1, 2, 3

STATUS_NAMES = {0: "MS_OK", 1: "MS_EINVAL", 2: "MS_ESHAPE", 3: "MS_EDTYPE", 4: "MS_EALIGN",
                5: "MS_ENOTPINNED", 6: "MS_EWORKSPACE", 7: "MS_ESTATE", 8: "MS_EHIP"}


class ModelDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("mlp_mult", C.c_int32), ("grid_h", C.c_int32), ("grid_w", C.c_int32),
                ("n_text", C.c_int32), ("dual_stream", C.c_int32), ("max_batch", C.c_int32),
                ("dtype", C.c_int32), ("ln_eps", C.c_float)]


WEIGHT_FIELDS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                 "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2")


class LayerWeights(C.Structure):
    _fields_ = [(k, C.c_void_p) for k in WEIGHT_FIELDS]


class KVSource(C.Structure):
    _fields_ = [("kind", C.c_int32), ("layer", C.POINTER(C.c_void_p)), ("n_slots", C.c_int32),
                ("slots", C.POINTER(C.c_void_p)), ("request_layer", C.POINTER(C.c_void_p)), ("flags", C.c_int32)]


MS_KV_LOADS_AHEAD = 1


class CostModel(C.Structure):
    """ms_cost_model: per-block Comp(F) = comp_ms0 + comp_ms_per_gflop * F / 1e9 and
    Load(B) = load_ms0 + load_ms_per_mb * B / 1e6 (Sec. 4.3)."""
    _fields_ = [("comp_ms0", C.c_double), ("comp_ms_per_gflop", C.c_double), ("load_ms0", C.c_double),
                ("load_ms_per_mb", C.c_double), ("cache_bytes_per_token", C.c_double)]


class StepInfo(C.Structure):
    _fields_ = [("batch", C.c_int32), ("rows", C.c_int32), ("n_segments", C.c_int32),
                ("n_qtiles", C.c_int32), ("text_rows", C.c_int32), ("dense_prefix", C.c_int32),
                ("copy_spans", C.c_int32), ("copy_rows", C.c_int64), ("copy_spans_y", C.c_int32),
                ("copy_rows_y", C.c_int64)]


class MaskStepError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


_lib = None


def load() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2505_20600_amd.build.build()")
        lib = C.CDLL(LIB_PATH)
        vp, i32, sz = C.c_void_p, C.c_int32, C.c_size_t
        sig = {
            "mask_abi_version": (i32, []),
            "mask_last_error": (C.c_char_p, []),
            "mask_workspace_bytes": (sz, [C.POINTER(ModelDesc), i32]),
            "mask_step_init": (i32, [C.POINTER(vp), C.POINTER(ModelDesc), i32, vp, vp, sz, vp]),
            "mask_step_init_static": (i32, [C.POINTER(vp), C.POINTER(ModelDesc), i32, vp, vp]),
            "mask_step_get_info": (i32, [vp, C.POINTER(StepInfo)]),
            "mask_step_index": (i32, [vp, C.POINTER(vp), C.POINTER(vp), C.POINTER(vp)]),
            "mask_gather_rows": (i32, [vp, vp, vp, vp]),
            "mask_block_forward": (i32, [vp, i32, C.POINTER(LayerWeights), vp, vp, vp]),
            "mask_scatter_rows": (i32, [vp, vp, vp, vp, vp]),
            "cache_prefetch_layer": (i32, [vp, i32, vp, vp, vp, vp, vp]),
            "cache_prefetch_inputs": (i32, [vp, i32, vp, vp, vp, vp, vp]),
            "mask_recompute_kv": (i32, [vp, i32, C.POINTER(LayerWeights), vp, vp, vp]),
            "mask_stack_forward": (i32, [vp, C.POINTER(LayerWeights), vp, vp, C.POINTER(KVSource),
                                         vp, vp, vp]),
            "mask_step_destroy": (None, [vp]),
            "mask_step_set_dense_prefix": (i32, [vp, i32, vp]),
            "mask_plan_dense_prefix": (i32, [i32, C.c_double, C.c_double, C.c_double, C.POINTER(i32),
                                             C.POINTER(C.c_double)]),
            "mask_profiler_start": (i32, [C.c_uint32, i32]),
            "ms_linear": (i32, [i32, i32, i32, i32, vp, vp, vp, vp, vp, i32, i32, i32, i32, vp, sz, vp]),
            "mask_profiler_stop": (i32, [C.POINTER(C.c_double), C.POINTER(C.c_int64), C.POINTER(C.c_int64)]),
            "mask_profiler_intervals": (i32, [C.POINTER(C.c_int32), C.POINTER(C.c_double), C.POINTER(C.c_double),
                                              i32, C.POINTER(C.c_int32)]),
            "mask_plan_copies": (i32, [vp, i32, i32, C.c_double, C.POINTER(i32), i32, C.POINTER(i32)]),
            "mask_probe_mfma": (i32, [i32, i32, C.POINTER(C.c_double), C.POINTER(C.c_double)]),
            "mask_probe_lds": (i32, [C.POINTER(C.c_double)]),
            "mask_probe_operand_stream": (i32, [i32, C.POINTER(C.c_double), C.POINTER(C.c_double)]),
            "mask_fit_linear": (i32, [C.POINTER(C.c_double), C.POINTER(C.c_double), i32, C.POINTER(C.c_double),
                                      C.POINTER(C.c_double), C.POINTER(C.c_double)]),
            "mask_batch_cost": (i32, [C.POINTER(ModelDesc), C.POINTER(CostModel), C.POINTER(i32), i32,
                                      C.POINTER(C.c_double), C.POINTER(i32), C.POINTER(C.c_double)]),
            "mask_route_request": (i32, [C.POINTER(ModelDesc), C.POINTER(CostModel), C.POINTER(i32),
                                         C.POINTER(i32), i32, i32, i32, C.POINTER(i32), C.POINTER(C.c_double)]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


STATIC_SCRATCH_BYTES = 128 << 20   # MS_STATIC_SCRATCH_BYTES

EXPORTED = ("mask_abi_version", "mask_last_error", "mask_workspace_bytes", "mask_step_init",
            "mask_step_init_static",
            "mask_step_get_info", "mask_step_index", "mask_gather_rows", "mask_block_forward",
            "mask_scatter_rows", "cache_prefetch_layer", "cache_prefetch_inputs", "mask_recompute_kv",
            "mask_stack_forward", "mask_step_destroy",
            "mask_step_set_dense_prefix", "mask_plan_dense_prefix",
            "mask_profiler_start", "mask_profiler_stop", "mask_profiler_intervals", "ms_linear",
            "mask_fit_linear", "mask_batch_cost", "mask_route_request", "mask_plan_copies",
            "mask_probe_mfma", "mask_probe_lds", "mask_probe_operand_stream")

MS_EPI_BIAS, MS_EPI_BIAS_RESID, MS_EPI_BIAS_GELU = 0, 1, 2


def ms_linear(A, W, bias, out, *, resid=None, epilogue=MS_EPI_BIAS, tile=(0, 0), ksplit=0,
              workspace=None, stream=None):
    """out = epilogue(A W^T + bias (+ resid)) through the library's GEMM kernels."""
    M, K = A.shape
    N = W.shape[0]
    dt = MS_BF16 if A.dtype == torch.bfloat16 else MS_FP32
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(load().ms_linear(dt, M, N, K, _ptr(A), _ptr(W), _ptr(bias), _ptr(resid), _ptr(out), epilogue,
                            tile[0], tile[1], ksplit, _ptr(workspace), ws_bytes, _stream(stream)))

KERNEL_CLASSES = ("compact", "gather", "layernorm", "gemm_qkv", "attention", "gemm_out", "gemm_up",
                  "gemm_down", "scatter", "copy", "attn_combine", "gemm_reduce")


def profiler_start(classes=KERNEL_CLASSES, capacity: int = 65536):
    mask = 0
    for c in classes:
        mask |= 1 << KERNEL_CLASSES.index(c)
    _check(load().mask_profiler_start(mask, capacity))


def profiler_stop() -> dict:
    """{class: (total_ms, launches)} of the launches recorded since profiler_start()."""
    n = len(KERNEL_CLASSES)
    ms = (C.c_double * n)()
    cnt = (C.c_int64 * n)()
    dropped = C.c_int64()
    _check(load().mask_profiler_stop(ms, cnt, C.byref(dropped)))
    out = {c: (ms[i], cnt[i]) for i, c in enumerate(KERNEL_CLASSES) if cnt[i]}
    out["_dropped"] = dropped.value
    return out


def profiler_intervals() -> list:
    """[(class, start_ms, end_ms)] of the launches of the last profiler_start()..profiler_stop()
    run, on one timeline across streams (ms from the first recorded start)."""
    lib = load()
    n = C.c_int32()
    _check(lib.mask_profiler_intervals(None, None, None, 0, C.byref(n)))
    k = n.value
    cls, t0, t1 = (C.c_int32 * max(k, 1))(), (C.c_double * max(k, 1))(), (C.c_double * max(k, 1))()
    _check(lib.mask_profiler_intervals(cls, t0, t1, k, C.byref(n)))
    return [(KERNEL_CLASSES[cls[i]], t0[i], t1[i]) for i in range(min(k, n.value))]


def _check(status: int):
    if status != MS_OK:
        raise MaskStepError(status, load().mask_last_error().decode())


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _event(e) -> int | None:
    """Raw hipEvent_t of a torch.cuda.Event (or an int handle). torch creates its events
    on first use; passing one that does not exist yet would silently drop the ordering."""
    if e is None:
        return None
    if isinstance(e, int):
        return e
    h = e.cuda_event
    if not h:
        raise ValueError("torch.cuda.Event has no HIP event yet: record it once before passing it")
    return h


def _stream(s) -> int | None:
    if s is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def mask_plan_dense_prefix(n_layers: int, load_ms: float, cached_ms: float, full_ms: float):
    """(k, modelled latency) of the best dense prefix under Alg. 1's latency model."""
    k = C.c_int32()
    lat = C.c_double()
    _check(load().mask_plan_dense_prefix(n_layers, load_ms, cached_ms, full_ms, C.byref(k), C.byref(lat)))
    return k.value, lat.value


def mask_plan_copies(mask, grid_h: int, grid_w: int, copy_cost_rows: float):
    """Copies (n0, w, h) of one request's cache-load plan: rows n0 + j * grid_w + [0, w), j < h."""
    m = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8).reshape(-1))
    if m.size != grid_h * grid_w:
        raise ValueError(f"mask has {m.size} entries, the grid {grid_h} x {grid_w}")
    n = C.c_int32()
    st = load().mask_plan_copies(m.ctypes.data, grid_h, grid_w, copy_cost_rows, None, 0, C.byref(n))
    if st not in (MS_OK, MS_ESHAPE) or (st == MS_ESHAPE and n.value == 0):
        _check(st)
    out = (C.c_int32 * max(1, 3 * n.value))()
    _check(load().mask_plan_copies(m.ctypes.data, grid_h, grid_w, copy_cost_rows, out, n.value, C.byref(n)))
    return [(out[3 * i], out[3 * i + 1], out[3 * i + 2]) for i in range(n.value)]


def probe_ceilings():
    """The diagnostic probes (matrix-core issue rate and clock, LDS reads, operand stream) on cuda:0."""
    lib = load()
    out = {}
    for kind, name in ((0, "16x16x32"), (1, "32x32x16")):
        for wps in (1, 2):
            tf, ghz = C.c_double(), C.c_double()
            _check(lib.mask_probe_mfma(kind, wps, C.byref(tf), C.byref(ghz)))
            out[f"mfma_{name}_bf16_{wps}wave_tflops"] = round(tf.value, 1)
            out[f"mfma_{name}_bf16_{wps}wave_clock_ghz"] = round(ghz.value, 3)
    tb = C.c_double()
    _check(lib.mask_probe_lds(C.byref(tb)))
    out["lds_read_tbs"] = round(tb.value, 1)
    for to_lds, name in ((1, "to_lds"), (0, "to_vgprs")):
        us, tbs = C.c_double(), C.c_double()
        _check(lib.mask_probe_operand_stream(to_lds, C.byref(us), C.byref(tbs)))
        out[f"operand_stream_{name}_us_per_64kb_step"] = round(us.value, 3)
        out[f"operand_stream_{name}_tbs"] = round(tbs.value, 2)
    return out


def mask_fit_linear(x, y):
    """(intercept, slope, r2) of the least-squares line y ~ intercept + slope * x."""
    n = len(x)
    xa = (C.c_double * max(1, n))(*[float(v) for v in x])
    ya = (C.c_double * max(1, len(y)))(*[float(v) for v in y])
    if len(y) != n:
        raise MaskStepError(MS_EINVAL, "x and y differ in length")
    a, b, r2 = C.c_double(), C.c_double(), C.c_double()
    _check(load().mask_fit_linear(xa, ya, n, C.byref(a), C.byref(b), C.byref(r2)))
    return a.value, b.value, r2.value


def mask_batch_cost(desc: ModelDesc, model: CostModel, masked):
    """((L, C_w, C_wo), dense prefix, latency) of one batch (masked image tokens per request)."""
    n = len(masked)
    arr = (C.c_int32 * max(1, n))(*[int(v) for v in masked])
    costs = (C.c_double * 3)()
    k, lat = C.c_int32(), C.c_double()
    _check(load().mask_batch_cost(C.byref(desc), C.byref(model), arr, n, costs, C.byref(k), C.byref(lat)))
    return (costs[0], costs[1], costs[2]), k.value, lat.value


def mask_route_request(desc: ModelDesc, model: CostModel, workers, max_batch: int, request_masked: int):
    """(worker index or -1, cost) of Alg. 2 for one request; ``workers`` = running batches."""
    flat = [int(v) for w in workers for v in w]
    run = (C.c_int32 * max(1, len(flat)))(*flat)
    sizes = (C.c_int32 * max(1, len(workers)))(*[len(w) for w in workers])
    w, cost = C.c_int32(), C.c_double()
    _check(load().mask_route_request(C.byref(desc), C.byref(model), run, sizes, len(workers), max_batch,
                                     int(request_masked), C.byref(w), C.byref(cost)))
    return w.value, cost.value


def model_desc(shape, max_batch: int | None = None) -> ModelDesc:
    """ModelDesc from an object with the ModelShape fields."""
    return ModelDesc(shape.n_layers, shape.d_model, shape.n_heads, shape.mlp_mult, shape.grid_h,
                     shape.grid_w, shape.n_text, 1 if shape.dual_stream else 0,
                     max_batch if max_batch is not None else max(1, shape.batch),
                     MS_BF16 if shape.dtype == "bf16" else MS_FP32, shape.ln_eps)


def mask_workspace_bytes(desc: ModelDesc, batch: int) -> int:
    n = load().mask_workspace_bytes(C.byref(desc), batch)
    if n == 0:
        raise MaskStepError(MS_ESHAPE, load().mask_last_error().decode())
    return n


def layer_weights_struct(w: dict) -> LayerWeights:
    return LayerWeights(*[_ptr(w[k]) for k in WEIGHT_FIELDS])


def weights_array(layers) -> C.Array:
    """[L] (or [L][2] image, text) weight dicts of device tensors -> a C array of structs.
    The array keeps the tensors alive: the structs hold only their addresses."""
    flat = []
    for w in layers:
        if isinstance(w, (tuple, list)):
            flat.extend(w)
        else:
            flat.append(w)
    arr = (LayerWeights * len(flat))(*[layer_weights_struct(w) for w in flat])
    arr._tensors = flat
    return arr


class MaskStep:
    """One step context (mask set): wraps mask_step_init ... mask_step_destroy."""

    def __init__(self, desc: ModelDesc, batch: int, d_mask: torch.Tensor, workspace: torch.Tensor | None,
                 stream=None):
        """``workspace`` None: mask_step_init_static (the library's static scratch)."""
        self._lib = load()
        self.desc = desc
        self.batch = batch
        self.workspace = workspace
        self.mask = d_mask
        h = C.c_void_p()
        if workspace is None:
            _check(self._lib.mask_step_init_static(C.byref(h), C.byref(desc), batch, _ptr(d_mask), _stream(stream)))
        else:
            _check(self._lib.mask_step_init(C.byref(h), C.byref(desc), batch, _ptr(d_mask), _ptr(workspace),
                                            workspace.numel() * workspace.element_size(), _stream(stream)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            self._lib.mask_step_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def info(self) -> StepInfo:
        info = StepInfo()
        _check(self._lib.mask_step_get_info(self.handle, C.byref(info)))
        return info

    def index_views(self):
        """(rows [M], inv [B*T], seg_start [n_seg+1]) as int32 views into the workspace."""
        if self.workspace is None:
            raise ValueError("a step on the static scratch has no workspace tensor to view")
        r, i, s = C.c_void_p(), C.c_void_p(), C.c_void_p()
        _check(self._lib.mask_step_index(self.handle, C.byref(r), C.byref(i), C.byref(s)))
        info = self.info()
        T = self.desc.n_text + self.desc.grid_h * self.desc.grid_w
        base = self.workspace.data_ptr()
        ws8 = self.workspace.view(torch.uint8)

        def view(p, n):
            off = p - base
            return ws8[off:off + 4 * n].view(torch.int32)

        return view(r.value, info.rows), view(i.value, self.batch * T), view(s.value, info.n_segments + 1)

    def gather_rows(self, x, xm=None, stream=None):
        _check(self._lib.mask_gather_rows(self.handle, _ptr(x), _ptr(xm), _stream(stream)))

    def block_forward(self, layer: int, weights, xm, kv, stream=None):
        arr = weights_array([weights])
        _check(self._lib.mask_block_forward(self.handle, layer, arr, _ptr(xm), _ptr(kv), _stream(stream)))

    def scatter_rows(self, xm, ycache, y, stream=None):
        _check(self._lib.mask_scatter_rows(self.handle, _ptr(xm), _ptr(ycache), _ptr(y), _stream(stream)))

    def prefetch_layer(self, layer: int, h_kv, d_slot, copy_stream, wait_event=None, signal_event=None):
        """cache_prefetch_layer; events are torch.cuda.Event objects (already created, e.g.
        recorded once) or raw hipEvent_t handles."""
        _check(self._lib.cache_prefetch_layer(self.handle, layer, _ptr(h_kv), _ptr(d_slot),
                                              _stream(copy_stream), _event(wait_event), _event(signal_event)))

    def prefetch_inputs(self, layer: int, h_yin, d_slot, copy_stream, wait_event=None, signal_event=None):
        _check(self._lib.cache_prefetch_inputs(self.handle, layer, _ptr(h_yin), _ptr(d_slot),
                                               _stream(copy_stream), _event(wait_event), _event(signal_event)))

    def recompute_kv(self, layer: int, weights, y_in, kv, stream=None):
        """K/V of the unmasked image tokens from their cached block input (Y caching);
        ``weights`` as for block_forward."""
        arr = weights_array([weights])
        _check(self._lib.mask_recompute_kv(self.handle, layer, arr, _ptr(y_in), _ptr(kv), _stream(stream)))

    def set_dense_prefix(self, k: int, stream=None):
        _check(self._lib.mask_step_set_dense_prefix(self.handle, k, _stream(stream)))

    def stack_forward(self, weights_c, x, ycache, kv_layers, y, *, pinned: bool = False, slots=(),
                      stream=None, copy_stream=None, inputs: bool = False, per_request=None,
                      loads_ahead: bool = False):
        """``weights_c`` from weights_array(); ``kv_layers``: [L] tensors (device or pinned host),
        per-layer K/V [B][T|N][2][d], or with ``inputs`` the cached block inputs [B][N][d]
        (Y caching); ``slots``: device buffers the pinned layers stream through. With
        ``pinned``, ``per_request`` may replace ``kv_layers``: [L][B] pinned per-request
        buffers (or None for requests that recompute nothing). ``loads_ahead``: MS_KV_LOADS_AHEAD
        (nothing else touches the slots between consecutive calls through them)."""
        if per_request is not None:
            L = len(per_request)
            ptrs = (C.c_void_p * 1)()
            req = (C.c_void_p * max(1, sum(len(r) for r in per_request)))(
                *[_ptr(t) for r in per_request for t in r])
            req_p = C.cast(req, C.POINTER(C.c_void_p))
            layer_p = C.POINTER(C.c_void_p)()
        else:
            L = len(kv_layers)
            ptrs = (C.c_void_p * L)(*[_ptr(t) for t in kv_layers])
            req_p = C.POINTER(C.c_void_p)()
            layer_p = C.cast(ptrs, C.POINTER(C.c_void_p))
        sl = (C.c_void_p * max(1, len(slots)))(*[_ptr(t) for t in slots])
        kind = (MS_Y_HOST_PINNED if pinned else MS_Y_DEVICE) if inputs else \
               (MS_KV_HOST_PINNED if pinned else MS_KV_DEVICE)
        src = KVSource(kind, layer_p, len(slots) if pinned else 0, C.cast(sl, C.POINTER(C.c_void_p)), req_p,
                       MS_KV_LOADS_AHEAD if loads_ahead else 0)
        cs = _stream(stream)
        ps = _stream(copy_stream) if copy_stream is not None else cs
        _check(self._lib.mask_stack_forward(self.handle, weights_c, _ptr(x), _ptr(ycache), C.byref(src),
                                            _ptr(y), cs, ps))
