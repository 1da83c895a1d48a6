"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Index work (compaction, gather, scatter, untouched cache rows) is compared bit
for bit; floating point within max relative error 1e-4 (fp32) and 2e-2 (bf16)
in the max norm, and element-wise within the bound for the number of blocks
between the shared input and the compared tensor (tests/parity_gate). bf16
references round the softmax weights to bf16 (the oracle's ``round_p``), as
the matrix units do.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_20600_amd import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the gpu-marked tests must run on an MI355X")


@pytest.fixture(autouse=True)
def _gpu():
    _require_gpu()
    yield


def _random_mask(shape, ratio, seed):
    g = np.random.default_rng(seed)
    m = np.zeros((shape.batch, shape.n_image), np.uint8)
    for b in range(shape.batch):
        r = ratio[b] if isinstance(ratio, (list, tuple)) else ratio
        k = int(round(r * shape.n_image))
        m[b, g.choice(shape.n_image, k, replace=False)] = 1
    return m


def _inputs(shape, cfg, *, dense_cache=False, random_ln=True, std=0.02):
    ws = W.stack_weights(shape, cfg, random_ln=random_ln, std=std)
    xt = W.template_hidden(shape, cfg)
    if dense_cache:
        yc, kv = oracle.dense_stack(xt, ws, shape)   # bf16 configs: already bf16 values
    else:
        kv = np.stack([W.synthetic_kv_cache(shape, cfg, l) for l in range(shape.n_layers)])
        yc = W.synthetic_y_cache(shape, cfg)
    return ws, xt, kv, yc


# ------------------------------------------------------------------ compaction

COMPACT_SHAPES = [
    W.ModelShape("g8", 1, 64, 1, 4, 8, 8, dtype="bf16", batch=1),
    W.ModelShape("g8b3", 1, 64, 1, 4, 8, 8, dtype="bf16", batch=3),
    W.ModelShape("g8txt", 1, 64, 1, 4, 8, 8, n_text=5, dual_stream=True, dtype="bf16", batch=2),
    W.ModelShape("g8txt1", 1, 64, 1, 4, 8, 8, n_text=3, dual_stream=False, dtype="bf16", batch=2),
    W.ModelShape("g64", 1, 64, 1, 4, 64, 64, dtype="bf16", batch=8),
    W.ModelShape("g64txt", 1, 64, 1, 4, 64, 64, n_text=512, dual_stream=True, dtype="bf16", batch=4),
    W.ModelShape("g70", 1, 64, 1, 4, 70, 70, dtype="bf16", batch=1),   # N=4900 > one scan chunk
]


def _edge_masks(shape):
    B, N = shape.batch, shape.n_image
    out = [np.zeros((B, N), np.uint8), np.ones((B, N), np.uint8)]
    m = np.zeros((B, N), np.uint8); m[:, 0] = 1; out.append(m)
    m = np.zeros((B, N), np.uint8); m[:, -1] = 1; out.append(m)
    m = np.zeros((B, N), np.uint8); m[0, :] = 7; out.append(m)          # request 0 full, others empty
    m = (np.arange(N)[None, :].repeat(B, 0) % 2).astype(np.uint8) * 200; out.append(m)  # checkerboard-ish
    return out


@pytest.mark.parametrize("shape", COMPACT_SHAPES, ids=lambda s: s.name)
def test_compaction_bit_exact(shape):
    masks = _edge_masks(shape) + [_random_mask(shape, r, s) for s, r in enumerate((0.03, 0.31, 0.77))]
    for i, mask in enumerate(masks):
        step = G.new_step(shape, mask)
        ref = oracle.compact(mask, shape.n_text, shape.dual_stream)
        rows, inv, seg = step.index_views()
        torch.cuda.synchronize()
        info = step.info()
        assert info.rows == ref["M"], i
        np.testing.assert_array_equal(rows.cpu().numpy(), ref["rows"], err_msg=f"mask {i}")
        np.testing.assert_array_equal(inv.cpu().numpy(), ref["inv"], err_msg=f"mask {i}")
        np.testing.assert_array_equal(seg.cpu().numpy(), ref["seg_start"], err_msg=f"mask {i}")
        sizes = np.diff(ref["seg_start"])
        assert info.n_qtiles == int(np.sum((sizes + 63) // 64))
        step.close()


def test_gather_and_scatter_bit_exact():
    shape = W.ModelShape("gs", 1, 128, 2, 4, 16, 16, n_text=8, dtype="bf16", batch=3)
    mask = _random_mask(shape, (0.1, 0.5, 0.0), 3)
    ref = oracle.compact(mask, shape.n_text, False)
    g = np.random.default_rng(4)
    x = W.to_bf16_values(g.standard_normal((shape.batch, shape.n_tokens, shape.d_model)))
    yc = W.to_bf16_values(g.standard_normal(x.shape))
    step = G.new_step(shape, mask)
    d_x, d_yc = G.to_dev(x, shape), G.to_dev(yc, shape)
    xm = torch.empty((ref["M"], shape.d_model), dtype=torch.bfloat16, device=G.DEV)
    step.gather_rows(d_x, xm)
    flat = x.reshape(-1, shape.d_model)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(G.to_np(xm), flat[ref["rows"]])
    xm.mul_(-1)
    y = torch.empty_like(d_yc)
    step.scatter_rows(xm, d_yc, y)
    want = yc.reshape(-1, shape.d_model).copy()
    want[ref["rows"]] = -flat[ref["rows"]]
    torch.cuda.synchronize()
    np.testing.assert_array_equal(G.to_np(y).reshape(-1, shape.d_model), want)
    step.scatter_rows(xm, d_yc, d_yc)  # aliased: in place
    torch.cuda.synchronize()
    np.testing.assert_array_equal(G.to_np(d_yc).reshape(-1, shape.d_model), want)


# ------------------------------------------------------------------ one block, staged

def test_block_fresh_kv_rows_match_oracle():
    """LN1 + QKV GEMM + K/V scatter epilogue: fresh K/V rows and untouched cached rows."""
    shape = W.ModelShape("blk", 1, 256, 4, 4, 16, 16, dtype="bf16")
    ws, xt, kv, yc = _inputs(shape, 21, std=0.05)
    mask = _random_mask(shape, 0.3, 5)
    y, kv_gpu, _ = G.run_stack(shape, mask, xt, kv, yc, ws)
    y_ref, kv_ref = oracle.masked_stack(xt, mask, kv, yc, ws, shape, return_kv=True, round_p=True)
    toks = oracle.masked_tokens(mask[0], 0)
    keep = np.setdiff1d(np.arange(shape.n_tokens), toks)
    np.testing.assert_array_equal(kv_gpu[0][0, keep], kv[0][0, keep])
    G.assert_close(kv_gpu[0][0, toks], kv_ref[0, 0, toks], "bf16", "fresh K/V", blocks=1)
    G.assert_close(y[0, toks], y_ref[0, toks], "bf16", "block output", blocks=1, inp=xt[0, toks])
    np.testing.assert_array_equal(y[0, keep], yc[0, keep])


# ------------------------------------------------------------------ workload-shaped parity

def test_c1_fp32_block_matches_oracle():
    """Single fp32 block d=256, 4 heads, 32x32 grid, 12x17 rectangle, cache from a dense run."""
    shape = W.CONFIGS["c1"]
    ws, xt, kv, yc = _inputs(shape, 1, dense_cache=True, random_ln=False)
    mask = W.workload_mask("c1", shape)
    assert int(mask.sum()) == 204
    x = W.edited_hidden(shape, 1, xt, mask)
    y, kv_gpu, _ = G.run_stack(shape, mask, x, kv, yc, ws)
    y_ref, kv_ref = oracle.masked_stack(x, mask, kv, yc, ws, shape, return_kv=True)
    G.assert_close(y, y_ref, "fp32", "c1 output", blocks=1, inp=x)
    G.assert_close(kv_gpu[0], kv_ref[0], "fp32", "c1 working K/V", blocks=1)
    keep = mask[0] == 0
    # the cached rows pass through the device's float32 copy of the cache unchanged
    np.testing.assert_array_equal(y[0, keep], yc[0, keep].astype(np.float32))


def test_c1_own_cache_reproduces_dense():
    """Cache = this input's own dense K/V: masked rows equal the dense rows (and so does the rest)."""
    shape = W.CONFIGS["c1"]
    ws, xt, kv, yc = _inputs(shape, 1, dense_cache=True, random_ln=True)
    mask = W.workload_mask("c1", shape)
    y, _, _ = G.run_stack(shape, mask, xt, kv, yc, ws)
    G.assert_close(y, yc, "fp32", "c1 own-cache", blocks=1, inp=xt)


SMALL_BF16 = [
    # ragged key tiles (T = 144), head_dim 72 padded to 96
    W.ModelShape("hd72_T144", 2, 576, 8, 4, 12, 12, dtype="bf16"),
    # head_dim 64, several key tiles, multi-layer
    W.ModelShape("hd64_T256_L3", 3, 256, 4, 4, 16, 16, dtype="bf16"),
    # head_dim 128, batch 3, varlen
    W.ModelShape("hd128_b3", 2, 256, 2, 4, 12, 16, dtype="bf16", batch=3),
    # dual weight streams with text rows always recomputed
    W.ModelShape("dual_txt40_b2", 2, 256, 2, 4, 10, 10, n_text=40, dual_stream=True, dtype="bf16", batch=2),
    # 2 x 96 text rows: the text / image boundary on a multiple of every tile height
    W.ModelShape("dual_txt96_b2", 2, 256, 2, 4, 10, 10, n_text=96, dual_stream=True, dtype="bf16", batch=2),
]


@pytest.mark.parametrize("shape", SMALL_BF16, ids=lambda s: s.name)
@pytest.mark.parametrize("ratio", [0.07, 0.45, 1.0])
def test_small_bf16_stack_matches_oracle(shape, ratio):
    ws, xt, kv, yc = _inputs(shape, 30 + shape.n_layers, std=0.03)
    mask = _random_mask(shape, [ratio * (1 - 0.3 * b) for b in range(shape.batch)], 7)
    x = W.edited_hidden(shape, 30, xt, mask)
    y, kv_gpu, _ = G.run_stack(shape, mask, x, kv, yc, ws)
    y_ref, kv_ref = oracle.masked_stack(x, mask, kv, yc, ws, shape, return_kv=True, round_p=True)
    G.assert_close(y, y_ref, "bf16", f"{shape.name} output", blocks=shape.n_layers, inp=x)
    for l in range(shape.n_layers):
        G.assert_close(kv_gpu[l], kv_ref[l], "bf16", f"{shape.name} K/V layer {l}", blocks=l + 1)
    for b in range(shape.batch):
        keep = np.concatenate([np.zeros(shape.n_text, bool), mask[b] == 0])
        np.testing.assert_array_equal(y[b, keep], yc[b, keep])
        np.testing.assert_array_equal(kv_gpu[0][b, keep], kv[0][b, keep])


# The widest bf16 model the library accepts (d_model 4096, 32 heads of 128), and the
# largest batch with two weight streams: 64 requests, 2 x 64 packed segments, the
# most one step holds (masks of 0 to 100% by turns, so whole-request skips too).
LIMIT_SHAPES = [
    W.ModelShape("limit_d4096", 1, 4096, 32, 4, 4, 8, dtype="bf16"),
    W.ModelShape("limit_b64_dual", 1, 256, 2, 4, 4, 4, n_text=4, dual_stream=True, dtype="bf16", batch=64),
]


@pytest.mark.parametrize("shape", LIMIT_SHAPES, ids=lambda s: s.name)
def test_step_at_the_accepted_limits_matches_oracle(shape):
    ws, xt, kv, yc = _inputs(shape, 90)
    ratio = [(b % 5) / 4 for b in range(shape.batch)] if shape.batch > 1 else 0.5
    mask = _random_mask(shape, ratio, 23)
    x = W.edited_hidden(shape, 90, xt, mask)
    y, kv_gpu, _ = G.run_stack(shape, mask, x, kv, yc, ws)
    y_ref, kv_ref = oracle.masked_stack(x, mask, kv, yc, ws, shape, return_kv=True, round_p=True)
    G.assert_close(y, y_ref, "bf16", f"{shape.name} output", blocks=1, inp=x)
    G.assert_close(kv_gpu[0], kv_ref[0], "bf16", f"{shape.name} K/V", blocks=1)
    for b in range(shape.batch):
        keep = np.concatenate([np.zeros(shape.n_text, bool), mask[b] == 0])
        np.testing.assert_array_equal(y[b, keep], yc[b, keep])


def test_single_masked_token_per_request_matches_oracle():
    """One recomputed row per request: a query tile of one valid row over every key."""
    shape = W.ModelShape("one_token_b3", 2, 256, 4, 4, 12, 16, dtype="bf16", batch=3)
    ws, xt, kv, yc = _inputs(shape, 91, std=0.03)
    mask = _random_mask(shape, 1.0 / shape.n_image, 29)
    assert (mask.sum(1) == 1).all()
    x = W.edited_hidden(shape, 91, xt, mask)
    y, kv_gpu, _ = G.run_stack(shape, mask, x, kv, yc, ws)
    y_ref, kv_ref = oracle.masked_stack(x, mask, kv, yc, ws, shape, return_kv=True, round_p=True)
    G.assert_close(y, y_ref, "bf16", "one token output", blocks=shape.n_layers, inp=x)
    for l in range(shape.n_layers):
        G.assert_close(kv_gpu[l], kv_ref[l], "bf16", f"one token K/V layer {l}", blocks=l + 1)


FUSE_SHAPES = [
    # d = 576 at a few hundred rows: both residual projections split K
    W.ModelShape("fuse_dual_d576", 3, 576, 8, 4, 10, 12, n_text=24, dual_stream=True, dtype="bf16", batch=2),
    # float32 never splits K: LayerNorm runs per row range after each projection
    W.ModelShape("fuse_f32_d256", 3, 256, 4, 4, 10, 10, dtype="fp32", batch=2),
]


@pytest.mark.parametrize("shape", FUSE_SHAPES, ids=lambda s: s.name)
def test_split_k_sum_fused_with_layernorm_is_bit_exact(shape, monkeypatch):
    """A split-K residual projection with its following LayerNorm in one kernel gives the
    same bits as the split-K sum and a LayerNorm launch, across blocks (LayerNorm 1 of the
    next block), with two weight sets, a dense prefix and Y caching."""
    ws, xt, kv, yc = _inputs(shape, 80, std=0.03)
    mask = _random_mask(shape, [0.3, 0.1], 17)
    x = W.edited_hidden(shape, 80, xt, mask)
    dt = "bf16" if shape.dtype == "bf16" else "fp32"
    G.assert_close(G.run_stack(shape, mask, x, kv, yc, ws)[0],
                   oracle.masked_stack(x, mask, kv, yc, ws, shape, round_p=True), dt, f"{shape.name} fused",
                   blocks=shape.n_layers, inp=x)
    yin = np.stack([np.asarray(yc)[:, shape.n_text:]] * shape.n_layers)
    runs = [dict(), dict(dense_prefix=1), dict(pinned=True), dict(inputs=True, pinned=True)]
    for kw in runs:
        outs = []
        for flag in ("0", "1"):
            monkeypatch.setenv("MS_NO_LN_FUSE", flag)
            cache = yin if kw.get("inputs") else kv
            outs.append(G.run_stack(shape, mask, x, cache, yc, ws, **kw)[0])
        np.testing.assert_array_equal(outs[0], outs[1], err_msg=f"{shape.name} {kw}")


def test_all_ones_mask_with_poisoned_cache_equals_dense():
    shape = W.ModelShape("ones", 2, 256, 4, 4, 12, 12, dtype="bf16", batch=2)
    ws, xt, _, _ = _inputs(shape, 40, std=0.03)
    y_ref, _ = oracle.dense_stack(xt, ws, shape, round_p=True)
    ones = np.ones((shape.batch, shape.n_image), np.uint8)
    kv = np.zeros((shape.n_layers, shape.batch, shape.n_tokens, 2, shape.d_model))
    y, _, _ = G.run_stack(shape, ones, xt, kv, None, ws, poison_cache=True)
    assert np.all(np.isfinite(y))
    G.assert_close(y, y_ref, "bf16", "all-ones", blocks=shape.n_layers, inp=xt)


@pytest.mark.parametrize("aliased", [False, True])
def test_empty_mask_returns_cache_bit_exact(aliased):
    shape = W.ModelShape("empty", 2, 256, 4, 4, 12, 12, dtype="bf16", batch=2)
    ws, xt, kv, yc = _inputs(shape, 41)
    zero = np.zeros((shape.batch, shape.n_image), np.uint8)
    y, kv_gpu, step = G.run_stack(shape, zero, xt, kv, yc, ws, aliased=aliased)
    assert step.info().rows == 0
    np.testing.assert_array_equal(y, yc)
    np.testing.assert_array_equal(kv_gpu[1], kv[1])


def test_batch_equals_single_requests(monkeypatch):
    """Requests are independent: bit-exact with one key range per query tile (the key-range
    split count depends on the whole batch's row count), within tolerance with the default split."""
    shape = W.ModelShape("sep", 2, 256, 4, 4, 12, 12, dtype="bf16", batch=3)
    ws, xt, kv, yc = _inputs(shape, 42, std=0.03)
    mask = _random_mask(shape, [0.2, 0.6, 0.05], 9)
    one = shape.replace(batch=1)
    for target in ("1", None):
        if target:
            monkeypatch.setenv("MS_ATTN_SPLIT_TARGET", target)
        else:
            monkeypatch.delenv("MS_ATTN_SPLIT_TARGET", raising=False)
        yb, _, _ = G.run_stack(shape, mask, xt, kv, yc, ws)
        for b in range(3):
            y1, _, _ = G.run_stack(one, mask[b:b + 1], xt[b:b + 1], kv[:, b:b + 1], yc[b:b + 1], ws)
            if target:
                np.testing.assert_array_equal(y1[0], yb[b])
            else:
                G.assert_close(y1[0], yb[b], "bf16", f"request {b} alone vs in the batch", blocks=shape.n_layers,
                               inp=xt[b])


# ------------------------------------------------------------------ streamed cache

STREAM_SHAPE = W.ModelShape("stream", 5, 256, 2, 4, 16, 16, n_text=0, dtype="bf16", batch=2)
STREAM_DUAL = W.ModelShape("stream_dual", 3, 256, 2, 4, 8, 16, n_text=16, dual_stream=True, dtype="bf16",
                           batch=2)


@pytest.mark.parametrize("shape", [STREAM_SHAPE, STREAM_DUAL], ids=lambda s: s.name)
def test_streamed_cache_matches_resident_and_serialized(shape):
    ws, xt, kv, yc = _inputs(shape, 50, std=0.03)
    mask = np.stack([W.ellipse_mask(shape.grid_h, shape.grid_w, r, W.rng(3, 3, b)) for b, r in
                     enumerate((0.25, 0.1))])
    x = W.edited_hidden(shape, 50, xt, mask)
    y_res, _, _ = G.run_stack(shape, mask, x, kv, yc, ws)
    y_pipe, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True)
    y_ser, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True, serialize=True)
    np.testing.assert_array_equal(y_pipe, y_res)
    np.testing.assert_array_equal(y_ser, y_res)
    y_ref = oracle.masked_stack(x, mask, kv, yc, ws, shape, round_p=True)
    G.assert_close(y_res, y_ref, "bf16", f"{shape.name} streamed", blocks=shape.n_layers, inp=x)


def test_streamed_repeated_steps_are_identical():
    """Back-to-back steps on the same slots (copy stream racing the previous step)."""
    shape = STREAM_SHAPE
    ws, xt, kv, yc = _inputs(shape, 51, std=0.03)
    mask = _random_mask(shape, 0.15, 11)
    dw = G.dev_weights(ws, shape)
    wc = G.MS.weights_array(dw)
    step = G.new_step(shape, mask)
    host = []
    for l in range(shape.n_layers):
        t = torch.empty((shape.batch, shape.n_image, 2, shape.d_model), dtype=torch.bfloat16, pin_memory=True)
        t.copy_(torch.as_tensor(np.ascontiguousarray(kv[l], np.float32)).to(torch.bfloat16))
        host.append(t)
    slots = [torch.empty((shape.batch, shape.n_tokens, 2, shape.d_model), dtype=torch.bfloat16,
                         device=G.DEV) for _ in range(3)]
    d_x, d_yc = G.to_dev(xt, shape), G.to_dev(yc, shape)
    copy = torch.cuda.Stream()
    outs = []
    for _ in range(4):
        y = torch.empty_like(d_yc)
        step.stack_forward(wc, d_x, d_yc, host, y, pinned=True, slots=slots, copy_stream=copy)
        outs.append(y)
    torch.cuda.synchronize()
    for y in outs[1:]:
        assert torch.equal(y, outs[0])


# ------------------------------------------------------------------ attention key-range split

@pytest.mark.parametrize("hd_shape", [
    W.ModelShape("split_hd64", 1, 256, 4, 4, 16, 20, dtype="bf16", batch=2),
    W.ModelShape("split_hd72", 1, 576, 8, 4, 12, 20, dtype="bf16"),
    W.ModelShape("split_hd128", 1, 256, 2, 4, 20, 16, dtype="bf16"),
], ids=lambda s: s.name)
def test_attention_split_and_unsplit_match_oracle(hd_shape, monkeypatch):
    """The key range of a query tile is split over workgroups (log-sum-exp combine) or not."""
    shape = hd_shape
    ws, xt, kv, yc = _inputs(shape, 60, std=0.03)
    mask = _random_mask(shape, 0.4, 13)
    x = W.edited_hidden(shape, 60, xt, mask)
    y_ref = oracle.masked_stack(x, mask, kv, yc, ws, shape, round_p=True)
    outs = []
    for target in ("1", "100000"):
        monkeypatch.setenv("MS_ATTN_SPLIT_TARGET", target)
        y, _, _ = G.run_stack(shape, mask, x, kv, yc, ws)
        G.assert_close(y, y_ref, "bf16", f"{shape.name} split target {target}", blocks=1, inp=x)
        outs.append(y)
    G.assert_close(outs[1], outs[0], "bf16", "split vs unsplit", blocks=1, inp=x)


# ------------------------------------------------------------------ dense prefix (bubble-free pipeline)

PREFIX_SHAPE = W.ModelShape("prefix", 4, 256, 2, 4, 16, 16, dtype="bf16", batch=2)
PREFIX_DUAL = W.ModelShape("prefix_dual", 3, 256, 2, 4, 8, 16, n_text=16, dual_stream=True, dtype="bf16",
                           batch=2)


@pytest.mark.parametrize("shape", [PREFIX_SHAPE, PREFIX_DUAL], ids=lambda s: s.name)
def test_dense_prefix_matches_oracle_and_streaming_is_exact(shape):
    """Blocks [0, k) over every token, the rest cached: resident, streamed through 1, 2 or
    n_layers slots, pipelined or serialized — identical bits, and the oracle within tolerance."""
    ws, xt, kv, yc = _inputs(shape, 70, std=0.03)
    mask = np.stack([W.ellipse_mask(shape.grid_h, shape.grid_w, r, W.rng(7, 3, b)) for b, r in
                     enumerate((0.3, 0.12))])
    x = W.edited_hidden(shape, 70, xt, mask)
    for k in (1, 2, shape.n_layers):
        y_ref = oracle.masked_stack(x, mask, kv, yc, ws, shape, dense_prefix=k, round_p=True)
        y_res, _, step = G.run_stack(shape, mask, x, kv, yc, ws, dense_prefix=k)
        assert step.info().dense_prefix == k
        G.assert_close(y_res, y_ref, "bf16", f"{shape.name} dense prefix {k}", blocks=shape.n_layers, inp=x)
        for n_slots in (1, 2, shape.n_layers):
            y_pipe, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True, n_slots=n_slots, dense_prefix=k)
            np.testing.assert_array_equal(y_pipe, y_res, err_msg=f"k={k} slots={n_slots}")
        y_ser, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True, serialize=True, dense_prefix=k)
        np.testing.assert_array_equal(y_ser, y_res)
    # the prefix reads no cache of its blocks: poisoning them changes nothing
    poisoned = kv.copy()
    poisoned[:2] = np.nan
    y_a, _, _ = G.run_stack(shape, mask, x, poisoned, yc, ws, dense_prefix=2)
    y_b, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, dense_prefix=2)
    np.testing.assert_array_equal(y_a, y_b)


def test_dense_prefix_own_cache_reproduces_dense():
    shape = PREFIX_SHAPE.replace(batch=1)
    ws = W.stack_weights(shape, 71, random_ln=True, std=0.03)
    xt = W.template_hidden(shape, 71)
    y_dense, kv_dense = oracle.dense_stack(xt, ws, shape, round_p=True)
    mask = np.stack([W.ellipse_mask(16, 16, 0.25, W.rng(7, 3, 9))])
    y, _, _ = G.run_stack(shape, mask, xt, kv_dense, y_dense, ws, pinned=True, n_slots=4, dense_prefix=2)
    G.assert_close(y, y_dense, "bf16", "own cache with a dense prefix", blocks=shape.n_layers, inp=xt)


# ------------------------------------------------------------------ Y caching (Sec. 3.1, Fig. 5 bottom)

Y_SHAPE = W.ModelShape("ycache", 4, 256, 2, 4, 16, 16, dtype="bf16", batch=2)
Y_DUAL = W.ModelShape("ycache_dual", 3, 256, 2, 4, 8, 16, n_text=16, dual_stream=True, dtype="bf16", batch=2)


def _y_inputs(shape, cfg):
    ws = W.stack_weights(shape, cfg, random_ln=True, std=0.03)
    xt = W.template_hidden(shape, cfg)
    yin = oracle.dense_inputs(xt, ws, shape, round_p=True)   # the template's cached block inputs
    yc, _ = oracle.dense_stack(xt, ws, shape, round_p=True)
    return ws, xt, yin, yc


@pytest.mark.parametrize("shape", [Y_SHAPE, Y_DUAL], ids=lambda s: s.name)
def test_y_cache_matches_oracle_resident_and_streamed(shape):
    ws, xt, yin, yc = _y_inputs(shape, 60)
    mask = np.stack([W.ellipse_mask(shape.grid_h, shape.grid_w, r, W.rng(3, 6, b)) for b, r in
                     enumerate((0.3, 0.1))])
    x = W.edited_hidden(shape, 60, xt, mask)
    ref = oracle.masked_stack_y(x, mask, yin, yc, ws, shape, round_p=True)
    y_res, _, _ = G.run_stack(shape, mask, x, yin, yc, ws, inputs=True)
    G.assert_close(y_res, ref, "bf16", f"{shape.name} Y cache resident", blocks=shape.n_layers, inp=x)
    for serialize in (False, True):
        y_pin, _, _ = G.run_stack(shape, mask, x, yin, yc, ws, inputs=True, pinned=True, serialize=serialize)
        np.testing.assert_array_equal(y_pin, y_res)
    # unmasked rows of the output are the cached final state, bit for bit
    yc_b = G.to_np(G.to_dev(yc, shape))
    for b in range(shape.batch):
        keep = np.concatenate([np.zeros(shape.n_text, bool), mask[b] == 0])
        np.testing.assert_array_equal(y_res[b, keep], yc_b[b, keep])


def test_y_cache_reads_no_recomputed_row_and_no_prefix_cache():
    shape = Y_SHAPE
    ws, xt, yin, yc = _y_inputs(shape, 61)
    mask = _random_mask(shape, 0.25, 12)
    x = W.edited_hidden(shape, 61, xt, mask)
    for k in (0, 2):
        ref, _, _ = G.run_stack(shape, mask, x, yin, yc, ws, inputs=True, dense_prefix=k)
        poisoned = yin.copy()
        poisoned[:k] = np.nan
        for b in range(shape.batch):
            poisoned[:, b, mask[b] != 0] = np.nan
        y, _, _ = G.run_stack(shape, mask, x, poisoned, yc, ws, inputs=True, dense_prefix=k, pinned=True)
        np.testing.assert_array_equal(y, ref)
        G.assert_close(ref, oracle.masked_stack_y(x, mask, yin, yc, ws, shape, dense_prefix=k, round_p=True),
                       "bf16", f"Y cache, dense prefix {k}", blocks=shape.n_layers, inp=x)


def test_y_cache_own_cache_is_dense_and_all_masked_reads_nothing():
    shape = Y_DUAL
    ws, xt, yin, yc = _y_inputs(shape, 62)
    mask = _random_mask(shape, 0.3, 13)
    y_dense = yc                                         # own cache: the current input is the template
    y, _, _ = G.run_stack(shape, mask, xt, yin, yc, ws, inputs=True)
    G.assert_close(y, y_dense, "bf16", "Y own cache vs dense", blocks=shape.n_layers, inp=xt)
    ones = np.ones_like(mask)
    y1, _, _ = G.run_stack(shape, ones, xt, np.full_like(yin, np.nan), None, ws, inputs=True)
    G.assert_close(y1, y_dense, "bf16", "all masked, Y cache never read", blocks=shape.n_layers, inp=xt)


# ------------------------------------------------------------------ slot reuse (use after recycle)

@pytest.mark.parametrize("shape", [STREAM_SHAPE, STREAM_DUAL], ids=lambda s: s.name)
@pytest.mark.parametrize("inputs", [False, True], ids=["kv", "y"])
def test_poisoned_slots_change_nothing(shape, inputs, monkeypatch):
    """MS_POISON fills each streamed slot with NaN right after its block: with fewer slots
    than cached layers (each slot reloaded by later layers), a dense prefix and the
    serialized form, the output is bit-identical to the unpoisoned run, so no block
    reads a row that its own load or its fresh K/V did not write."""
    ws, xt, kv, yc = _inputs(shape, 52, std=0.03)
    mask = _random_mask(shape, [0.3, 0.1], 19)
    x = W.edited_hidden(shape, 52, xt, mask)
    cache = np.stack([np.asarray(yc)[:, shape.n_text:]] * shape.n_layers) if inputs else kv
    for kw in (dict(n_slots=2), dict(n_slots=1), dict(n_slots=2, dense_prefix=1), dict(n_slots=2, serialize=True)):
        monkeypatch.delenv("MS_POISON", raising=False)
        y0, _, _ = G.run_stack(shape, mask, x, cache, yc, ws, pinned=True, inputs=inputs, **kw)
        monkeypatch.setenv("MS_POISON", "1")
        y1, _, _ = G.run_stack(shape, mask, x, cache, yc, ws, pinned=True, inputs=inputs, **kw)
        assert np.all(np.isfinite(y1)), kw
        np.testing.assert_array_equal(y1, y0, err_msg=str(kw))
