"""C-ABI surface: the library loads, exports every function include/*.h
declares, and rejects bad configurations without touching a GPU (CPU only)."""
import os
import re

import pytest

import synth
from paper_2606_12154_amd import hh

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if h.endswith(".h"):
            text = open(os.path.join(ROOT, "include", h)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(hh_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_header_declares_the_binding_names():
    assert declared_functions() == sorted(hh.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = hh.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_workspace_sizes():
    tiny = hh.hh_workspace_size(hh.make_config(synth.TINY, 4, 256))
    assert 10_000_000 < tiny < 100_000_000
    big = hh.hh_workspace_size(hh.make_config(synth.ONE_B, 1, 8704, 8192))
    # bf16 weights + fp16 MFMA copy (2 x 2.47 GB) + fp16 KV (32 KiB/token) + scratch
    assert 2 * 2_471_632_896 + 8704 * 32768 < big < 7_000_000_000


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 128, hh.HH_ERR_UNSUPPORTED),
    ("page_size", 32, hh.HH_ERR_UNSUPPORTED),
    ("n_kv_heads", 3, hh.HH_ERR_UNSUPPORTED),
    ("d_model", 200, hh.HH_ERR_UNSUPPORTED),
    ("ffn_dim", 690, hh.HH_ERR_UNSUPPORTED),
    ("dtype", 7, hh.HH_ERR_UNSUPPORTED),
    ("max_streams", 0, hh.HH_ERR_UNSUPPORTED),
    ("max_context", 131073, hh.HH_ERR_UNSUPPORTED),
    ("weight_format", 2, hh.HH_ERR_UNSUPPORTED),
    ("weight_format", hh.HH_WF_Q4G32, hh.HH_ERR_UNSUPPORTED),  # the tiny model is fp32
])
def test_unsupported_configs(field, value, status):
    cfg = hh.make_config(synth.TINY, 2, 128)
    setattr(cfg, field, value)
    with pytest.raises(hh.HHError) as e:
        hh.hh_workspace_size(cfg)
    assert e.value.status == status


def test_query_group_must_be_power_of_two():
    cfg = hh.make_config(synth.TINY, 2, 128)
    cfg.n_heads, cfg.n_kv_heads, cfg.d_model = 12, 4, 768  # 3 query heads per kv head
    with pytest.raises(hh.HHError) as e:
        hh.hh_workspace_size(cfg)
    assert e.value.status == hh.HH_ERR_UNSUPPORTED


def test_create_rejects_null_arena_and_small_arena():
    cfg = hh.make_config(synth.TINY, 2, 128)
    with pytest.raises(hh.HHError) as e:
        hh.hh_create(cfg, 0, 1 << 30, 1)
    assert e.value.status == hh.HH_ERR_INVALID_ARG
    with pytest.raises(hh.HHError) as e:
        hh.hh_create(cfg, 1 << 20, 16, 1)
    assert e.value.status == hh.HH_ERR_OOM


def test_q4_workspace_adds_the_stored_rows():
    base = hh.hh_workspace_size(hh.make_config(synth.ONE_B, 1, 1024))
    q4 = hh.hh_workspace_size(hh.make_config(synth.ONE_B, 1, 1024, weight_format=hh.HH_WF_Q4G32))
    # 4.5 bits per weight of every streamed matrix (the head included, the
    # embedding table not), each region rounded up to 256 bytes.
    sh = synth.ONE_B
    rows = sh.vocab + sh.n_layers * (sh.q_dim + 2 * sh.kv_dim + sh.d_model + 2 * sh.ffn_dim + sh.ffn_dim)
    expect = rows * (sh.d_model // 2 + sh.d_model // 16)
    assert expect <= q4 - base <= expect + 256 * (1 + 4 * sh.n_layers)


def test_q4_quantize_rejects_bad_arguments():
    with pytest.raises(hh.HHError) as e:
        hh.hh_q4g32_quantize(1 << 20, 4, 48, 1 << 21, 0)   # K not a multiple of 32
    assert e.value.status == hh.HH_ERR_INVALID_ARG
    with pytest.raises(hh.HHError) as e:
        hh.hh_q4g32_quantize(0, 4, 64, 1 << 21, 0)
    assert e.value.status == hh.HH_ERR_INVALID_ARG


def test_read_probe_rejects_bad_arguments():
    import numpy as np
    host = np.zeros(64, dtype=np.uint8)
    for ptr, n in [(host.ctypes.data, 64), (0, 64), (host.ctypes.data, 15)]:
        with pytest.raises(hh.HHError) as e:
            hh.hh_read_probe(ptr, n, 0)
        assert e.value.status == hh.HH_ERR_INVALID_ARG
