"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and its host-side arithmetic and validation behave as
documented (errors that are detected before any HIP call)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2606_00422_amd import upr
from synth import blob_size

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "upr.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(upr_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = upr.load()
    names = declared_functions()
    assert set(names) == set(upr.EXPORTS)
    for name in names:
        assert hasattr(lib, name), name


def test_weights_count_matches_blob_layout():
    for d, H, L, F in [(64, 2, 1, 256), (256, 4, 2, 1024), (512, 8, 4, 2048)]:
        cfg = upr.make_config(d, H, L, F, "bf16")
        assert upr.upr_weights_count(cfg) == blob_size(d, L, F)


def test_cache_bytes_and_index():
    cfg = upr.make_config(128, 2, 3, 256, "bf16")
    cap = 77
    assert upr.upr_kv_cache_bytes(cfg, cap) == 3 * 2 * 2 * cap * 64 * 2
    rng = np.random.default_rng(0)
    for _ in range(300):
        l, kv, h = int(rng.integers(3)), int(rng.integers(2)), int(rng.integers(2))
        r, e = int(rng.integers(cap)), int(rng.integers(64))
        assert upr.upr_kv_cache_index(cfg, cap, l, kv, h, r, e) == oracle.cache_index(2, 64, cap, l, kv, h, r, e)
    assert upr.upr_kv_cache_index(cfg, cap, 3, 0, 0, 0, 0) == -1
    assert upr.upr_kv_cache_index(cfg, cap, 0, 2, 0, 0, 0) == -1
    assert upr.upr_kv_cache_index(cfg, cap, 0, 0, 0, cap, 0) == -1
    assert upr.upr_kv_cache_index(cfg, cap, 0, 0, 0, 0, 64) == -1


@pytest.mark.parametrize("kw,status", [
    (dict(d_model=96, n_heads=3, head_dim=32), upr.UPR_ERR_CONFIG),    # d not a multiple of 64
    (dict(head_dim=48, n_heads=2, d_model=96), upr.UPR_ERR_CONFIG),
    (dict(d_model=128, n_heads=4, head_dim=64), upr.UPR_ERR_CONFIG),   # 4*64 != 128
    (dict(n_layers=0), upr.UPR_ERR_CONFIG),
    (dict(d_ff=100), upr.UPR_ERR_CONFIG),
    (dict(dtype=7), upr.UPR_ERR_DTYPE),
    (dict(ln_eps=0.0), upr.UPR_ERR_CONFIG),
    (dict(dtype=upr.UPR_BF16_MXFP8), upr.UPR_ERR_CONFIG),                   # d 128: not % 256
    (dict(dtype=upr.UPR_BF16_MXFP8, d_model=256, n_heads=4, d_ff=320), upr.UPR_ERR_CONFIG),  # F % 128
])
def test_model_create_rejects_bad_configs(kw, status):
    base = dict(d_model=128, n_heads=2, head_dim=64, n_layers=1, d_ff=256, dtype=upr.UPR_BF16,
                ln_eps=1e-5)
    base.update(kw)
    cfg = upr.upr_config(**base)
    assert upr.upr_weights_count(cfg) == -1
    with pytest.raises(upr.UprError) as ei:
        upr.upr_model_create(cfg, np.zeros(10, np.float32))
    assert ei.value.status == status
    assert upr.upr_last_error() != ""


def test_model_create_rejects_wrong_blob_size():
    cfg = upr.make_config(128, 2, 1, 256, "bf16")
    n = upr.upr_weights_count(cfg)
    with pytest.raises(upr.UprError) as ei:
        upr.upr_model_create(cfg, np.zeros(n - 1, np.float32))
    assert ei.value.status == upr.UPR_ERR_WEIGHTS


def test_null_model_is_rejected_before_any_launch():
    lib = upr.load()
    offs = np.array([0, 4], np.int32)
    seg = upr.segments(offs)
    cache = upr.upr_kv_cache(0, 4)
    st = lib.upr_encode_user(None, None, ctypes.byref(seg), ctypes.byref(cache), None, 0, None)
    assert st == upr.UPR_ERR_NULL
    st = lib.upr_rank_candidates(None, ctypes.byref(cache), ctypes.byref(seg), None,
                                 ctypes.byref(seg), None, None, 0, None)
    assert st == upr.UPR_ERR_NULL
    assert upr.upr_rank_workspace_bytes(0, seg, seg) == 0
    assert upr.upr_status_string(upr.UPR_ERR_OFFSETS) == "malformed segment offsets"


def test_host_mx_encoding_matches_the_oracle_bit_for_bit():
    """upr_mx_quantize_host (host logic: the fp8 variant's weight encoding)
    against oracle.mx_quantize on float32 values, including saturating block
    tops, subnormal-range values, zeros and negative zeros."""
    import oracle
    rng = np.random.default_rng(31)
    x = (rng.standard_normal((64, 256)) * np.exp2(rng.integers(-30, 30, (64, 1)))).astype(np.float32)
    x[0] = 0.0
    x[1, :32] = -0.0
    x[2, 5] = 1e-42                      # subnormal float32 block maximum
    x[3, :32] = rng.uniform(-1, 1, 32).astype(np.float32) * np.float32(2.0 ** -140)
    x[4, 7] = 3.0e38
    codes, scales = upr.upr_mx_quantize_host(x)
    oc, os_ = oracle.mx_quantize(x.astype(np.float64))
    np.testing.assert_array_equal(codes, oc)
    np.testing.assert_array_equal(scales, os_)


def test_mx_calls_validate_before_any_launch():
    for k in (0, 33, -32):
        with pytest.raises(upr.UprError) as ei:
            upr.upr_mx_quantize_host(np.zeros((2, max(k, 1)), np.float32)[:, :0] if k <= 0 else
                                     np.zeros((2, k), np.float32))
        assert ei.value.status == upr.UPR_ERR_LIMIT
    lib = upr.load()
    assert lib.upr_mx_quantize(None, 9, 1, 32, None, None, None) == upr.UPR_ERR_DTYPE
    assert lib.upr_mx_quantize(None, upr.UPR_MX_IN_F32, 4, 48, None, None, None) == upr.UPR_ERR_LIMIT
    assert lib.upr_mx_quantize(None, upr.UPR_MX_IN_F32, 4, 64, None, None, None) == upr.UPR_ERR_NULL
    assert lib.upr_mx_quantize(None, upr.UPR_MX_IN_F32, 0, 64, None, None, None) == upr.UPR_OK
    assert lib.upr_mx_linear(None, None, None, None, None, 4, 16, 96, None, None) == upr.UPR_ERR_LIMIT
    assert lib.upr_mx_linear(None, None, None, None, None, 4, 12, 128, None, None) == upr.UPR_ERR_LIMIT
    assert lib.upr_mx_linear(None, None, None, None, None, 4, 16, 128, None, None) == upr.UPR_ERR_NULL
    assert lib.upr_mx_linear(None, None, None, None, None, 0, 16, 128, None, None) == upr.UPR_OK


def test_kv_pool_validation_before_any_hip_call(tmp_path):
    """Pool calls that must fail before touching the GPU: bad shapes, sizes
    beyond the documented limit, malformed handles and files, NULL pools."""
    lib = upr.load()
    cfg = upr.make_config(512, 8, 4, 2048, "bf16")
    out = ctypes.c_void_p()
    bad = upr.make_config(96, 3, 1, 256, "bf16")
    assert lib.upr_kv_pool_create(ctypes.byref(bad), 2, 16, ctypes.byref(out)) == upr.UPR_ERR_CONFIG
    assert lib.upr_kv_pool_create(ctypes.byref(cfg), 0, 16, ctypes.byref(out)) == upr.UPR_ERR_LIMIT
    assert lib.upr_kv_pool_create(ctypes.byref(cfg), 2, 0, ctypes.byref(out)) == upr.UPR_ERR_LIMIT
    # 4 layers x 2 x 8 heads x 64 x 2 bytes = 8 KiB per row: 2^18 rows is 2 GiB
    assert lib.upr_kv_pool_create(ctypes.byref(cfg), 1, 1 << 18, ctypes.byref(out)) == upr.UPR_ERR_LIMIT
    assert lib.upr_kv_pool_create(ctypes.byref(cfg), 3, 100_000, ctypes.byref(out)) == upr.UPR_ERR_LIMIT
    assert out.value is None
    h = upr.upr_kv_pool_handle()
    h.magic, h.slots, h.capacity_rows, h.cfg = 0x1234, 1, 16, cfg
    assert lib.upr_kv_pool_open(ctypes.byref(h), ctypes.byref(out)) == upr.UPR_ERR_CONFIG
    h.magic, h.bytes = upr.UPR_KV_POOL_MAGIC, 12345              # size inconsistent with the shape
    assert lib.upr_kv_pool_open(ctypes.byref(h), ctypes.byref(out)) == upr.UPR_ERR_CONFIG
    assert lib.upr_kv_pool_open_file(os.fsencode(str(tmp_path / "missing")), ctypes.byref(out)) == upr.UPR_ERR_LIMIT
    short = tmp_path / "short"
    short.write_bytes(b"UPRP")
    assert lib.upr_kv_pool_open_file(os.fsencode(str(short)), ctypes.byref(out)) == upr.UPR_ERR_CONFIG
    assert out.value is None
    assert lib.upr_kv_pool_next_slot(None) == -1
    c = upr.upr_kv_cache()
    assert lib.upr_kv_pool_slot(None, 0, ctypes.byref(c)) == upr.UPR_ERR_NULL
    assert lib.upr_kv_pool_info(None, None, None, None) == upr.UPR_ERR_NULL
    lib.upr_kv_pool_destroy(None)
