"""Pins of the vision-block oracle (oracle/vit.py): the whole block against the
Qwen2.5-VL vision block of `transformers` (random weights, windows as cu_seqlens), the
2-D rotary embedding against its rotary module, window ids in closed form, and the
partial-recompute invariants."""
import numpy as np
import pytest
import torch

import fcdata
from oracle import vit as ov

SH = fcdata.TINY_VIT
OSH = ov.VitShape(d=SH.d, heads=SH.heads, hd=SH.hd, ffn=SH.ffn)


def test_patch_positions_token_major():
    pos = ov.patch_positions(2, 3, 2)
    # token (0, 1): patches (0, 2), (0, 3), (1, 2), (1, 3)
    np.testing.assert_array_equal(pos[4:8], [[0, 2], [0, 3], [1, 2], [1, 3]])
    assert pos.shape == (24, 2) and pos[:, 0].max() == 3 and pos[:, 1].max() == 5


def test_window_ids_closed_form():
    w = ov.window_ids(8, 8, 2, 4)            # 8 x 8 tokens, windows of 4 x 4 tokens
    tok = w[::4]
    assert set(tok) == {0, 1, 2, 3}
    assert tok[0] == 0 and tok[4] == 1 and tok[32] == 2 and tok[63] == 3
    assert (np.bincount(tok) == 16).all()
    assert not ov.window_ids(8, 8, 2, 0).any()
    # a ragged grid: 6 x 6 tokens, windows of 4: ceil(6/4) = 2 windows per row
    t = ov.window_ids(6, 6, 1, 4)
    assert t[5] == 1 and t[4 * 6] == 2 and t[35] == 3


def test_vision_rope_matches_transformers():
    from transformers.models.qwen2_5_vl.modeling_qwen2_5_vl import Qwen2_5_VisionRotaryEmbedding
    pos = ov.patch_positions(4, 5, 2)
    cos, sin = ov.vision_rope(pos, 80, 10000.0)
    rot = Qwen2_5_VisionRotaryEmbedding(40)
    freqs = rot(torch.arange(16)).float()                 # [max, 20]
    f = torch.cat([freqs[torch.from_numpy(pos[:, 0])], freqs[torch.from_numpy(pos[:, 1])]], dim=1)
    emb = torch.cat([f, f], dim=-1)
    np.testing.assert_allclose(cos, emb.cos().numpy(), atol=2e-6)
    np.testing.assert_allclose(sin, emb.sin().numpy(), atol=2e-6)


def transformers_block(wt, d, heads, ffn):
    from transformers.models.qwen2_5_vl.modeling_qwen2_5_vl import (Qwen2_5_VLVisionBlock,
                                                                    Qwen2_5_VLVisionConfig)
    cfg = Qwen2_5_VLVisionConfig(hidden_size=d, num_heads=heads, intermediate_size=ffn,
                                 hidden_act="silu")
    cfg._attn_implementation = "eager"
    blk = Qwen2_5_VLVisionBlock(cfg, attn_implementation="eager").float().eval()
    t = {k: torch.from_numpy(fcdata.bf16_to_f32(v)) for k, v in wt.items()}
    with torch.no_grad():
        blk.norm1.weight.copy_(t["g1"])
        blk.norm2.weight.copy_(t["g2"])
        blk.attn.qkv.weight.copy_(t["w_qkv"])
        blk.attn.qkv.bias.copy_(t["b_qkv"])
        blk.attn.proj.weight.copy_(t["w_o"])
        blk.attn.proj.bias.copy_(t["b_o"])
        blk.mlp.gate_proj.weight.copy_(t["w_gate"])
        blk.mlp.gate_proj.bias.copy_(t["b_gate"])
        blk.mlp.up_proj.weight.copy_(t["w_up"])
        blk.mlp.up_proj.bias.copy_(t["b_up"])
        blk.mlp.down_proj.weight.copy_(t["w_down"])
        blk.mlp.down_proj.bias.copy_(t["b_down"])
    return blk


@pytest.mark.parametrize("window_tokens", [2, 0])
def test_block_matches_transformers(window_tokens):
    """The whole block on a 4 x 6 token grid (2 x 2 merge, 96 patches), windowed and full,
    against transformers' block run on the patches in window order with cu_seqlens."""
    gh, gw, m = 4, 6, 2
    wt = fcdata.vit_weights(3, SH)
    rng = np.random.default_rng(4)
    x = fcdata.bf16_round(rng.standard_normal((gh * gw * 4, SH.d), dtype=np.float32))
    y, _, _ = ov.vit_block_full(x, wt, OSH, gh, gw, m, window_tokens)
    win = ov.window_ids(gh, gw, m, window_tokens)
    order = np.argsort(win, kind="stable")
    counts = np.bincount(win)
    cu = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    cos, sin = ov.vision_rope(ov.patch_positions(gh, gw, m), SH.hd, 10000.0)
    blk = transformers_block(wt, SH.d, SH.heads, SH.ffn)
    with torch.no_grad():
        out = blk(torch.from_numpy(fcdata.bf16_to_f32(x)[order]), cu_seqlens=cu,
                  position_embeddings=(torch.from_numpy(cos[order]), torch.from_numpy(sin[order])))
    ref = np.empty_like(y)
    ref[order] = out.numpy()
    np.testing.assert_allclose(y, ref, rtol=2e-4, atol=2e-4)


def test_partial_full_recompute_equals_block():
    gh, gw, m = 4, 4, 2
    wt = fcdata.vit_weights(5, SH)
    rng = np.random.default_rng(6)
    x = fcdata.bf16_round(rng.standard_normal((gh * gw * 4, SH.d), dtype=np.float32))
    y0, k0, v0 = ov.vit_block_full(x, wt, OSH, gh, gw, m, 2)
    junk = fcdata.bf16_round(rng.standard_normal(k0.shape, dtype=np.float32))
    y, k, v = ov.vit_block_partial(x, np.arange(gh * gw), junk, junk,
                                   fcdata.bf16_round(np.zeros_like(y0)), wt, OSH, gh, gw, m, 2)
    np.testing.assert_allclose(y, y0, rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(k, k0, rtol=1e-6, atol=1e-6)


def test_partial_with_exact_cache_matches_block_rows():
    """With caches holding the current frame's own k, v (what the block computes), the
    recomputed rows equal the whole block's rows; other rows keep the cache's outputs."""
    gh, gw, m = 4, 4, 2
    wt = fcdata.vit_weights(7, SH)
    rng = np.random.default_rng(8)
    x = fcdata.bf16_round(rng.standard_normal((gh * gw * 4, SH.d), dtype=np.float32))
    y0, k0, v0 = ov.vit_block_full(x, wt, OSH, gh, gw, m, 2)
    ycache = fcdata.bf16_round(rng.standard_normal(y0.shape, dtype=np.float32))
    rec = np.array([1, 5, 6, 14])
    y, k, v = ov.vit_block_partial(x, rec, k0, v0, ycache, wt, OSH, gh, gw, m, 2)
    rows = (rec[:, None] * 4 + np.arange(4)).ravel()
    np.testing.assert_allclose(y[rows], y0[rows], rtol=1e-5, atol=1e-5)
    keep = np.setdiff1d(np.arange(y.shape[0]), rows)
    np.testing.assert_array_equal(y[keep], fcdata.bf16_to_f32(ycache)[keep])


def test_partial_nothing_recomputed_changes_nothing():
    gh, gw, m = 2, 2, 2
    wt = fcdata.vit_weights(9, SH)
    rng = np.random.default_rng(10)
    k = fcdata.bf16_round(rng.standard_normal((16, SH.heads, SH.hd), dtype=np.float32))
    yc = fcdata.bf16_round(rng.standard_normal((16, SH.d), dtype=np.float32))
    y, k2, _ = ov.vit_block_partial(yc, np.array([], np.int64), k, k, yc, wt, OSH, gh, gw, m, 0)
    np.testing.assert_array_equal(y, fcdata.bf16_to_f32(yc))
    np.testing.assert_array_equal(k2, fcdata.bf16_to_f32(k))


def test_vit_cache_update_moves_whole_tokens():
    """A reused token takes all m x m patch rows of its source token, read from the
    previous frame's rows even when the source itself is overwritten in the same step."""
    gw, m = 3, 2
    n = 2 * gw * 4
    k = np.arange(n * 2, dtype=np.float32).reshape(n, 1, 2)
    y = -np.arange(n * 3, dtype=np.float32).reshape(n, 3)
    reuse = np.zeros(6, np.uint8)
    reuse[[0, 1]] = 1                                    # tokens 0, 1 take tokens 1, 2
    kc, vc, yc = ov.vit_cache_update(k, k, y, np.zeros_like(y), (0, 1), reuse, gw, m)
    np.testing.assert_array_equal(kc[0:4], k[4:8])
    np.testing.assert_array_equal(kc[4:8], k[8:12])      # from the old rows of token 2
    np.testing.assert_array_equal(yc[0:4], y[4:8])
    np.testing.assert_array_equal(kc[8:], k[8:])
    assert not yc[8:].any()


MSH = fcdata.TINY_MERGER
OMSH = ov.MergerShape(d=MSH.d, m=MSH.m, d_out=MSH.d_out)


def test_gelu_closed_forms():
    """GELU(0) = 0; GELU(x) - GELU(-x) = x (Phi(x) + Phi(-x) = 1); GELU(1) = Phi(1) with
    Phi(1) = 0.841344746068543 (normal table)."""
    x = np.linspace(-4, 4, 33).astype(np.float32)
    g = ov.gelu(x)
    assert ov.gelu(np.float32(0.0)) == 0.0
    np.testing.assert_allclose(g - ov.gelu(-x), x, atol=1e-6)
    np.testing.assert_allclose(ov.gelu(np.float32(1.0)), 0.841344746068543, rtol=1e-7)


def test_merger_matches_transformers():
    """The merger of a few tokens against transformers' Qwen2.5-VL patch merger on the
    same (bf16-valued) weights and inputs."""
    from transformers.models.qwen2_5_vl.modeling_qwen2_5_vl import Qwen2_5_VLPatchMerger
    wt = fcdata.merger_weights(40, MSH)
    rng = np.random.default_rng(41)
    n_tok = 12
    y = fcdata.bf16_round(rng.standard_normal((n_tok * 4, MSH.d), dtype=np.float32))
    toks = np.array([0, 3, 4, 11], np.int64)
    got = ov.merger_rows(y, toks, wt, OMSH)
    mod = Qwen2_5_VLPatchMerger(MSH.d_out, MSH.d, spatial_merge_size=2).float().eval()
    t = {k: torch.from_numpy(fcdata.bf16_to_f32(v)) for k, v in wt.items()}
    with torch.no_grad():
        mod.ln_q.weight.copy_(t["g"])
        mod.mlp[0].weight.copy_(t["w1"])
        mod.mlp[0].bias.copy_(t["b1"])
        mod.mlp[2].weight.copy_(t["w2"])
        mod.mlp[2].bias.copy_(t["b2"])
        want = mod(torch.from_numpy(fcdata.bf16_to_f32(y))).numpy()[toks]
    np.testing.assert_allclose(got, want, rtol=2e-5, atol=2e-5)


def test_merger_tokens_are_independent():
    """A token's output depends only on its own m^2 patch rows: changing another token's
    rows leaves it bit-identical, and the patch order inside the token matters."""
    wt = fcdata.merger_weights(42, MSH)
    rng = np.random.default_rng(43)
    y = fcdata.bf16_round(rng.standard_normal((8 * 4, MSH.d), dtype=np.float32))
    a = ov.merger_rows(y, [2], wt, OMSH)
    y2 = y.copy()
    y2[:8] = fcdata.bf16_round(rng.standard_normal((8, MSH.d), dtype=np.float32))
    np.testing.assert_array_equal(ov.merger_rows(y2, [2], wt, OMSH), a)
    y3 = y.copy()
    y3[8:12] = y[[9, 8, 11, 10]]
    assert not np.allclose(ov.merger_rows(y3, [2], wt, OMSH), a)
