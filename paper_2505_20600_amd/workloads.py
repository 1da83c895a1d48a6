"""Seeded synthetic workloads: model shapes, weights, hidden states, caches, masks.

This module is shared by the CPU oracle's tests and the GPU path's tests and
benchmark. It holds none of the method's arithmetic: it only draws seeded
random numbers and shapes them. Values that must be bf16 are produced by
torch's float32 -> bfloat16 conversion (round to nearest even), so both sides
receive identical, exactly representable inputs.

Every generator uses ``numpy.random.default_rng(SeedSequence([cfg, stream,
index]))`` with the streams:

    0  weights            (index = layer; dual-stream text weights use index + 1000)
    1  template hidden    (index = request)
    2  edited masked rows (index = request)
    3  masks              (index = request, or a caller-chosen mask id)
    4  mask-ratio draws   (index = draw)
    5  synthetic caches   (index = layer)

The paper's production traces are not available; the mask generators
(axis-aligned rectangle, union of random ellipses with an exact token count,
Gaussian-blurred random blobs) stand in for them, and their ratio
distributions follow the mask-ratio statistics the paper reports in its
workload characterisation (Sec. 2.2, means 0.11 / 0.19 / 0.35).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

# ---------------------------------------------------------------------------
# Model / workload shapes
# ---------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Shape of a pre-LN transformer block stack (Sec. 3.1: token-wise ops + attention).

    Tokens are the raster-order flattening of a ``grid_h x grid_w`` latent
    (Sec. 2.1), optionally preceded by ``n_text`` always-recomputed text
    tokens that use their own weight set (``dual_stream``).
    """

    name: str
    n_layers: int
    d_model: int
    n_heads: int
    mlp_mult: int
    grid_h: int
    grid_w: int
    n_text: int = 0
    dual_stream: bool = False
    dtype: str = "bf16"          # "fp32" or "bf16"
    batch: int = 1
    ln_eps: float = 1e-5

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    @property
    def n_image(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def n_tokens(self) -> int:
        return self.n_text + self.n_image

    def replace(self, **kw) -> "ModelShape":
        return dataclasses.replace(self, **kw)


# The five workloads: single fp32 block; 12-block d=768 stack; 28-block
# d=1152 stack streamed from pinned host memory; a heterogeneous batch of 8
# on the same stack; a 19-block d=3072 dual-stream stack with 512 text tokens.
CONFIGS = {
    "c1": ModelShape("c1_block_d256_fp32", 1, 256, 4, 4, 32, 32, dtype="fp32"),
    "c2": ModelShape("c2_stack12_d768_bf16", 12, 768, 12, 4, 64, 64),
    "c3": ModelShape("c3_stack28_d1152_bf16_streamed", 28, 1152, 16, 4, 64, 64),
    "c4": ModelShape("c4_stack28_d1152_bf16_batch8", 28, 1152, 16, 4, 64, 64, batch=8),
    "c5": ModelShape("c5_mmdit19_d3072_bf16_batch4", 19, 3072, 24, 4, 64, 64,
                     n_text=512, dual_stream=True, batch=4),
}
CONFIG_IDS = {"c1": 1, "c2": 2, "c3": 3, "c4": 4, "c5": 5}

C3_RATIOS = (0.05, 0.10, 0.25, 0.50, 1.00)


def rng(cfg: int, stream: int, index: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(cfg), int(stream), int(index)]))


def to_bf16_values(a: np.ndarray) -> np.ndarray:
    """float32 array whose values are the bf16 (RNE) conversions of ``a``."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _maybe_bf16(a: np.ndarray, dtype: str) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    return to_bf16_values(a) if dtype == "bf16" else a


# ---------------------------------------------------------------------------
# Weights and hidden states
# ---------------------------------------------------------------------------

LAYER_KEYS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
              "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2")


def layer_weights(shape: ModelShape, cfg: int, layer: int, *, random_ln: bool = False,
                  text: bool = False, std: float = 0.02) -> dict:
    """One layer's parameters, Linear weights stored ``[out][in]``.

    Weights and biases ~ N(0, std). LayerNorm gamma/beta are 1/0 unless
    ``random_ln`` (then 1 + N(0, 0.1) and N(0, 0.1), to exercise the affine path).
    """
    d, f = shape.d_model, shape.mlp_mult * shape.d_model
    g = rng(cfg, 0, layer + (1000 if text else 0))
    w = {
        "w_qkv": g.normal(0, std, (3 * d, d)),
        "b_qkv": g.normal(0, std, (3 * d,)),
        "w_o": g.normal(0, std, (d, d)),
        "b_o": g.normal(0, std, (d,)),
        "w_1": g.normal(0, std, (f, d)),
        "b_1": g.normal(0, std, (f,)),
        "w_2": g.normal(0, std, (d, f)),
        "b_2": g.normal(0, std, (d,)),
    }
    if random_ln:
        w["ln1_g"] = 1.0 + g.normal(0, 0.1, (d,))
        w["ln1_b"] = g.normal(0, 0.1, (d,))
        w["ln2_g"] = 1.0 + g.normal(0, 0.1, (d,))
        w["ln2_b"] = g.normal(0, 0.1, (d,))
    else:
        w["ln1_g"] = np.ones(d)
        w["ln1_b"] = np.zeros(d)
        w["ln2_g"] = np.ones(d)
        w["ln2_b"] = np.zeros(d)
    return {k: _maybe_bf16(w[k], shape.dtype) for k in LAYER_KEYS}


def stack_weights(shape: ModelShape, cfg: int, *, random_ln: bool = False,
                  std: float = 0.02) -> list:
    """Per layer: a dict (single stream) or a pair ``(image, text)`` (dual stream)."""
    out = []
    for l in range(shape.n_layers):
        wi = layer_weights(shape, cfg, l, random_ln=random_ln, std=std)
        if shape.dual_stream:
            wt = layer_weights(shape, cfg, l, random_ln=random_ln, text=True, std=std)
            out.append((wi, wt))
        else:
            out.append(wi)
    return out


def template_hidden(shape: ModelShape, cfg: int) -> np.ndarray:
    """``X_template [B][T][d]`` ~ N(0, 1)."""
    B, T, d = shape.batch, shape.n_tokens, shape.d_model
    x = np.empty((B, T, d), np.float32)
    for b in range(B):
        x[b] = rng(cfg, 1, b).standard_normal((T, d))
    return _maybe_bf16(x, shape.dtype)


def edited_hidden(shape: ModelShape, cfg: int, x_template: np.ndarray,
                  mask: np.ndarray) -> np.ndarray:
    """The template with the masked image rows (and all text rows) redrawn ~ N(0, 1)."""
    x = np.array(x_template, dtype=np.float32, copy=True)
    B, T, d = x.shape
    nt = shape.n_text
    for b in range(B):
        g = rng(cfg, 2, b)
        fresh = _maybe_bf16(g.standard_normal((T, d)), shape.dtype)
        sel = np.zeros(T, bool)
        sel[:nt] = True
        sel[nt:] = mask[b] != 0
        x[b, sel] = fresh[sel]
    return x


def synthetic_kv_cache(shape: ModelShape, cfg: int, layer: int, std: float = 0.5,
                       image_only: bool = False) -> np.ndarray:
    """A random stand-in for one layer's cached K/V, ``[B][T][2][d]`` (or ``[B][N][2][d]``).

    The masked computation is defined for any cache contents; a random cache
    is used where a dense run of the oracle would be too slow.
    """
    B, d = shape.batch, shape.d_model
    rows = shape.n_image if image_only else shape.n_tokens
    g = rng(cfg, 5, layer)
    return _maybe_bf16(g.normal(0, std, (B, rows, 2, d)), shape.dtype)


def synthetic_y_cache(shape: ModelShape, cfg: int) -> np.ndarray:
    B, T, d = shape.batch, shape.n_tokens, shape.d_model
    g = rng(cfg, 5, 100000)
    return _maybe_bf16(g.standard_normal((B, T, d)), shape.dtype)


# ---------------------------------------------------------------------------
# Masks on the token grid (uint8, nonzero = masked)
# ---------------------------------------------------------------------------


def rect_mask(grid_h: int, grid_w: int, ratio: float, g: np.random.Generator) -> np.ndarray:
    """Axis-aligned rectangle of h x w cells with h*w closest to ratio*N (ties: most square)."""
    target = ratio * grid_h * grid_w
    best = None
    for h in range(1, grid_h + 1):
        for w in range(1, grid_w + 1):
            key = (abs(h * w - target), abs(h - w), h)
            if best is None or key < best[0]:
                best = (key, h, w)
    _, h, w = best
    if h > w:  # prefer the wider orientation, h <= w
        h, w = w, h
    r0 = int(g.integers(0, grid_h - h + 1))
    c0 = int(g.integers(0, grid_w - w + 1))
    m = np.zeros((grid_h, grid_w), np.uint8)
    m[r0:r0 + h, c0:c0 + w] = 1
    return m.reshape(-1)


def _select_exact(score: np.ndarray, count: int, lowest: bool) -> np.ndarray:
    n = score.size
    order = np.lexsort((np.arange(n), score if lowest else -score))
    m = np.zeros(n, np.uint8)
    m[order[:count]] = 1
    return m


def ellipse_mask(grid_h: int, grid_w: int, ratio: float, g: np.random.Generator,
                 k: int | None = None) -> np.ndarray:
    """Union of k (1..4) random ellipses, scaled jointly so exactly round(ratio*N) cells are masked."""
    n = grid_h * grid_w
    count = int(round(ratio * n))
    if k is None:
        k = int(g.integers(1, 5))
    yy, xx = np.meshgrid(np.arange(grid_h) + 0.5, np.arange(grid_w) + 0.5, indexing="ij")
    score = np.full((grid_h, grid_w), np.inf)
    for _ in range(k):
        cy, cx = g.uniform(0, grid_h), g.uniform(0, grid_w)
        aspect = g.uniform(0.5, 2.0)
        size = g.uniform(0.5, 1.5)
        theta = g.uniform(0, math.pi)
        a, b = size * math.sqrt(aspect), size / math.sqrt(aspect)
        dy, dx = yy - cy, xx - cx
        u = dx * math.cos(theta) + dy * math.sin(theta)
        v = -dx * math.sin(theta) + dy * math.cos(theta)
        score = np.minimum(score, np.sqrt((u / a) ** 2 + (v / b) ** 2))
    return _select_exact(score.reshape(-1), count, lowest=True)


def _gauss_blur_1d(a: np.ndarray, sigma: float, axis: int) -> np.ndarray:
    r = int(math.ceil(3 * sigma))
    t = np.arange(-r, r + 1)
    k = np.exp(-0.5 * (t / sigma) ** 2)
    k /= k.sum()
    return np.apply_along_axis(lambda v: np.convolve(v, k, mode="same"), axis, a)


def blob_mask(grid_h: int, grid_w: int, ratio: float, g: np.random.Generator) -> np.ndarray:
    """Gaussian-blurred N(0,1) field (sigma = grid_w/12, zero padding); the round(ratio*N) highest cells."""
    n = grid_h * grid_w
    count = int(round(ratio * n))
    field = g.standard_normal((grid_h, grid_w))
    sigma = grid_w / 12.0
    field = _gauss_blur_1d(_gauss_blur_1d(field, sigma, 0), sigma, 1)
    return _select_exact(field.reshape(-1), count, lowest=False)


def ratio_draw(cfg_key: str, index: int) -> float:
    """The mask ratio distribution of each workload."""
    g = rng(CONFIG_IDS[cfg_key], 4, index)
    if cfg_key == "c1":
        return 0.2
    if cfg_key == "c2":
        return float(g.uniform(0.05, 0.60))
    if cfg_key == "c3":
        return C3_RATIOS[index % len(C3_RATIOS)]
    if cfg_key == "c4":
        return float(math.exp(g.uniform(math.log(0.03), math.log(0.80))))
    if cfg_key == "c5":
        return float(g.uniform(0.10, 0.40))
    raise KeyError(cfg_key)


def workload_mask(cfg_key: str, shape: ModelShape, mask_id: int = 0,
                  ratio: float | None = None) -> np.ndarray:
    """``uint8 [B][N]`` masks of workload ``cfg_key`` (mask set ``mask_id``)."""
    cfg = CONFIG_IDS[cfg_key]
    B, H, W = shape.batch, shape.grid_h, shape.grid_w
    out = np.zeros((B, H * W), np.uint8)
    for b in range(B):
        g = rng(cfg, 3, mask_id * 64 + b)
        r = ratio if ratio is not None else ratio_draw(cfg_key, mask_id * 64 + b)
        if r >= 1.0:
            out[b] = 1
        elif cfg_key == "c1":
            out[b] = rect_mask(H, W, r, g)
        elif cfg_key in ("c2", "c3"):
            out[b] = ellipse_mask(H, W, r, g)
        else:
            out[b] = blob_mask(H, W, r, g)
    return out
