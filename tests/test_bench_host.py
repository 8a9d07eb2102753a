"""Host-side logic of bench.py (no GPU): how kernel groups are named from
their algorithmic work, and how counter summaries are matched to a group.
A group that takes another kernel's counters would report a wrong `traffic`
figure in the benchmark line."""
import bench
import synth


def _names(cfg):
    return {(c, w): n for c, n, _, w in bench.kernel_shapes(cfg)}


def test_kernel_shapes_name_every_group_once():
    for name in ("dit_xl2", "pixart", "hunyuan"):
        shapes = bench.kernel_shapes(synth.CONFIGS[name])
        keys = [(c, w) for c, _, _, w in shapes]
        assert len(keys) == len(set(keys)), name      # (class, work) identifies a launch


def test_dit_xl2_runs_the_fused_qkv_attention():
    cfg = synth.CONFIGS["dit_xl2"]
    names = _names(cfg)
    B, T, D, H, hd = cfg.batch, cfg.tokens, cfg.hidden, cfg.heads, cfg.head_dim
    work = 2.0 * B * T * 3 * D * D + 4.0 * B * H * T * T * hd
    assert names[("attention", work)].startswith("QKV projection + self-attention")
    assert not any(n == "QKV projection" for n in names.values())
    # PixArt's 4096 tokens exceed the fused kernel's 256: separate QKV GEMM and attention.
    px = _names(synth.CONFIGS["pixart"])
    assert "QKV projection" in px.values() and "self-attention" in px.values()


def test_counter_tags_match_class_as_well_as_flops():
    cfg = synth.CONFIGS["dit_xl2"]
    B, T, D, F = cfg.batch, cfg.tokens, cfg.hidden, cfg.mlp
    flops = 2.0 * B * T * F * D                           # MLP up and down: the same FLOPs
    up = bench.counter_tag(cfg, {"class": "gemm_gelu", "work": flops})
    down = bench.counter_tag(cfg, {"class": "gemm_down", "work": flops})
    assert up[0] == "gemm_fc1_dit_xl2" and down[0] == "gemm_fc2_dit_xl2"
    assert bench.counter_tag(cfg, {"class": "gemm_gated", "work": flops}) == (None, None)


def test_grid_fits_tells_pixart_self_from_cross_attention():
    cfg = synth.CONFIGS["pixart"]
    B, H, T, hd = cfg.batch, cfg.heads, cfg.tokens, cfg.head_dim
    self_att = {"shape": [B, H, T, T, hd]}
    cross_att = {"shape": [B, H, T, cfg.ctx_tokens, hd]}
    streaming = "void bc::attention_dma_kernel<72, 4, 8, 2, true, true, false>(bc::AttnArgs)"
    resident = "void bc::attention_dma_kernel<72, 2, 8, 4, false, false, false>(bc::AttnArgs)"
    g_stream = -(-T // (16 * 4 * 8)) * H * B * 64 * 8
    g_res = -(-T // (16 * 2 * 8)) * H * B * 64 * 8
    assert bench.grid_fits(streaming, g_stream, self_att)
    assert not bench.grid_fits(streaming, g_stream, cross_att)
    assert bench.grid_fits(resident, g_res, cross_att)
    assert not bench.grid_fits(resident, g_res, self_att)


def test_grid_fits_gemm_tiles():
    g = {"shape": [4096, 1152, 4608]}
    kernel = "void bc::gemm_wide_kernel<2, 128, 144, 4, 4, 4, 64, 1, 1>(bc::GemmArgs)"
    assert bench.grid_fits(kernel, 32 * 8 * 64 * 16, g)
    assert not bench.grid_fits(kernel, 32 * 8 * 64 * 12, g)
