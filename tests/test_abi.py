"""The C-ABI library loads and exports every symbol include/incvit.h declares;
host-only queries (no GPU) validate configs and report sizes."""
import os
import re

import pytest

from paper_2607_12287_amd import incvit, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "incvit.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(incvit_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    L = incvit.lib()
    declared = header_functions()
    assert declared == sorted(incvit.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def test_sizes_match_canonical_layout():
    for m in (synth.TINY, synth.SO400M, synth.VIT_L, synth.small_model(dtype="bf16")):
        cfg = incvit.make_config(m, 4)
        eb = 2 if m.dtype == "bf16" else 4
        assert incvit.incvit_canonical_weights_bytes(cfg) == synth.canonical_weight_count(m) * eb
        assert incvit.incvit_packed_weights_bytes(cfg) >= incvit.incvit_canonical_weights_bytes(cfg) // 2


@pytest.mark.parametrize("field,value,status", [
    ("patch", 5, incvit.INCVIT_ERR_SHAPE),            # 32 is not a multiple of 5
    ("heads", 3, incvit.INCVIT_ERR_SHAPE),            # 64 % 3
    ("dim", 48, incvit.INCVIT_ERR_UNSUPPORTED),       # dim % 32
    ("dtype", 7, incvit.INCVIT_ERR_UNSUPPORTED),
    ("max_streams", 0, incvit.INCVIT_ERR_UNSUPPORTED),
    ("ln_eps", float("nan"), incvit.INCVIT_ERR_SHAPE),
    ("score", 7, incvit.INCVIT_ERR_ARG),
])
def test_invalid_configs_are_rejected_before_any_device_work(field, value, status):
    cfg = incvit.make_config(synth.small_model(dtype="bf16"), 2)
    setattr(cfg, field, value)
    assert incvit.incvit_canonical_weights_bytes(cfg) == 0
    assert incvit.incvit_last_error(None) != ""
    # packing with an invalid config fails synchronously with the right code
    assert incvit.incvit_pack_weights(cfg, 256, 256, 0) == status


@pytest.mark.parametrize("fields", [
    # 64 streams of 4096 tokens with a 16384-wide fp32 MLP: the hidden rows alone are 16 GiB
    dict(img_h=256, img_w=256, patch=4, dim=2048, heads=16, mlp_dim=16384, dtype=0, max_streams=64),
    # 1000 channels of 64x64 patches: one stream's patches are 64 MiB but W_pe is 32 GiB
    dict(img_h=256, img_w=256, channels=1000, patch=64, dim=2048, heads=16, mlp_dim=64, dtype=0, max_streams=1),
])
def test_buffers_beyond_32_bit_offsets_are_rejected(fields):
    cfg = incvit.make_config(synth.small_model(dtype="bf16"), 2)
    for k, v in fields.items():
        setattr(cfg, k, v)
    assert incvit.incvit_canonical_weights_bytes(cfg) == 0
    assert "4 GiB" in incvit.incvit_last_error(None)
    assert incvit.incvit_pack_weights(cfg, 256, 256, 0) == incvit.INCVIT_ERR_UNSUPPORTED
    # the same shapes with one stream and a narrow MLP are accepted
    if fields.get("channels", 3) == 3:
        cfg.max_streams, cfg.mlp_dim = 1, 512
        assert incvit.incvit_canonical_weights_bytes(cfg) > 0


def test_overlapping_caches_are_rejected_before_any_device_work():
    # a handle needs no device memory of its own; every pointer below is only
    # checked on the host (the call fails before anything is enqueued)
    cfg = incvit.make_config(synth.small_model(dtype="bf16"), 4)
    st, h = incvit.incvit_create(cfg, 1 << 20)
    assert st == incvit.INCVIT_OK
    try:
        cb = incvit.incvit_cache_bytes(h)
        base, ws, patches = 1 << 32, 1 << 30, 1 << 31
        for ptrs in ([base, base], [base, base + cb - 256], [base + cb // 512 * 256, base]):
            assert incvit.incvit_full_encode(h, len(ptrs), patches, ptrs, ws) == incvit.INCVIT_ERR_ARG
            assert "overlap" in incvit.incvit_last_error(h)
    finally:
        incvit.lib().incvit_destroy(h)


def test_null_arguments_are_rejected():
    cfg = incvit.make_config(synth.small_model(dtype="bf16"), 2)
    assert incvit.incvit_pack_weights(cfg, 0, 256, 0) == incvit.INCVIT_ERR_ARG
    st, h = incvit.incvit_create(cfg, 0)
    assert st == incvit.INCVIT_ERR_ARG and not h.value
    assert incvit.lib().incvit_full_encode(None, 1, None, None, None, None) == incvit.INCVIT_ERR_ARG


def test_noalloc_step_beyond_the_static_scratch_is_rejected_on_the_host():
    """incvit_step_noalloc refuses a call whose workspace exceeds its static
    scratch before touching the device (eight ViT-L streams need 72 MiB)."""
    m = synth.VIT_L
    st, h = incvit.incvit_create(incvit.make_config(m, 8), 1 << 20)
    assert st == incvit.INCVIT_OK
    try:
        assert incvit.incvit_workspace_bytes(h, 8) > incvit.NOALLOC_SCRATCH_BYTES
        assert incvit.incvit_workspace_bytes(h, 4) <= incvit.NOALLOC_SCRATCH_BYTES
        caches = [(1 << 40) + i * (1 << 30) for i in range(8)]
        st = incvit.incvit_step_noalloc(h, 8, 1 << 36, caches, 0.98, [256] * 8, 1 << 37, 1 << 38, 0, 0)
        assert st == incvit.INCVIT_ERR_ARG
        assert "static scratch" in incvit.incvit_last_error(h)
        assert incvit.incvit_step_noalloc(h, 9, 1 << 36, caches, 0.98, [256] * 9, 1 << 37, 1 << 38, 0, 0) \
            == incvit.INCVIT_ERR_ARG
    finally:
        incvit.lib().incvit_destroy(h)


@pytest.mark.parametrize("field,value", [
    ("cols", (3, 0, 0, 0)), ("cols", (0, 0, 0, 8)), ("cols", (-1, 0, 0, 0)),
    ("attn_qtiles", 3), ("attn_qtiles", -1), ("row_groups", 9), ("attn_waves", 6),
    ("fc2_mode", 3), ("tiled", 2),
])
def test_invalid_tunings_are_rejected(field, value):
    """incvit_set_tuning validates every field on the host (no device work)."""
    cfg = incvit.make_config(synth.small_model(dtype="bf16"), 2)
    st, h = incvit.incvit_create(cfg, 1 << 20)
    assert st == incvit.INCVIT_OK
    try:
        assert incvit.incvit_set_tuning(h, **{field: value}) == incvit.INCVIT_ERR_ARG
        assert field.split("_")[0] in incvit.incvit_last_error(h)
        # valid settings and the defaults are accepted
        assert incvit.incvit_set_tuning(h, cols=(1, 2, 4, 0), attn_qtiles=2, row_groups=8, attn_waves=4,
                                        fc2_mode=1, tiled=1) == incvit.INCVIT_OK
        assert incvit.lib().incvit_set_tuning(h, None) == incvit.INCVIT_OK
    finally:
        incvit.lib().incvit_destroy(h)
