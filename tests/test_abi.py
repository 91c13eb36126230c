"""CPU-only checks of the C-ABI: the library loads, exports every function that
include/lsv.h declares, and rejects bad arguments on the host before any HIP call."""
import ctypes
import os
import re

import pytest

from paper_2608_08721_amd import lsv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared():
    src = open(os.path.join(ROOT, "include", "lsv.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lsv_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lsv.LIB_PATH):
        from paper_2608_08721_amd import build
        build.build()
    return lsv.load()


def test_exports_every_declared_symbol(lib):
    names = declared()
    assert len(names) >= 13
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(lsv.EXPORTED) == names


def test_status_strings(lib):
    assert lsv.lsv_status_string(0) == "ok"
    assert "capacity" in lsv.lsv_status_string(lsv.LSV_ERR_CAPACITY)
    assert lsv.lsv_abi_version() == 3


def test_timing_hook_validation(lib):
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_set_timing_events, 9, [], 0, 0)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_set_timing_events, 2, [0] * 2, 257, 0)
    lsv.lsv_set_timing_events(2, [], 0)


def tiny_cfg(**kw):
    c = dict(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=4, head_dim=64, d_ff=688, vocab=1024,
             dtype=lsv.LSV_DTYPE_F32, rms_eps=1e-5, reserved0=0.0, rope_base=10000.0)
    c.update(kw)
    return lsv.ModelConfig(**c)


def test_size_queries_are_host_only(lib):
    cfg = tiny_cfg()
    assert lsv.lsv_packed_model_bytes(cfg) > 0
    assert lsv.lsv_kv_cache_bytes(cfg, 2, 128) == 2 * 2 * 2 * 4 * 128 * 64 * 4
    assert lsv.lsv_kv_cache_bytes(cfg, 2, 100) == 0  # capacity must be a multiple of LSV_KV_ALIGN
    assert lsv.lsv_verify_workspace_bytes(cfg, 1, 17, 145) > 0
    assert lsv.lsv_verify_workspace_bytes(cfg, 1, 264, 145) > 0
    assert lsv.lsv_verify_workspace_bytes(cfg, 1, lsv.LSV_MAX_ROWS + 1, 145) == 0
    assert lsv.lsv_packed_model_bytes(tiny_cfg(head_dim=96)) == 0
    assert lsv.lsv_packed_model_bytes(tiny_cfg(n_kv_heads=3)) == 0
    assert lsv.lsv_accept_workspace_bytes(1, 17, 128256) > 0
    # every packed matrix stays below 4 GiB: at d_model 8192 in bf16 an LM head fragment row is 256 KiB
    wide = dict(d_model=8192, n_q_heads=64, n_kv_heads=8, head_dim=128, d_ff=28672, dtype=lsv.LSV_DTYPE_BF16)
    assert lsv.lsv_packed_model_bytes(tiny_cfg(vocab=16383 * 16, **wide)) > 0
    assert lsv.lsv_packed_model_bytes(tiny_cfg(vocab=16384 * 16, **wide)) == 0
    assert "4 GiB" in lsv.lsv_last_error()


def test_attention_split_plan_in_the_workspace_size(lib):
    """The attention partials take n_splits x max_rows x n_q x (head_dim + 2) floats of the
    workspace, so its size shows the host's split plan.  Eight sequences over eight kv heads:
    a 128-chunk bound fits one round of four splits of 32 chunks, a 129-chunk bound would walk 33
    per split, more than twice the 16-chunk cap, and takes the packed grid's three rounds of
    splits (12 of 11 chunks).  Four sequences (one round of eight splits either way) keep the
    same plan, and so the same workspace."""
    cfg = tiny_cfg(n_layers=1, d_model=1024, n_q_heads=8, n_kv_heads=8, head_dim=128, d_ff=2816, vocab=4096,
                   dtype=lsv.LSV_DTYPE_BF16)
    per_split = 64 * 8 * (128 + 2) * 4  # max_rows 64, 8 query heads
    ws = lambda batch, ctx: lsv.lsv_verify_workspace_bytes(cfg, batch, 64, ctx)
    assert ws(8, 129 * 64) - ws(8, 128 * 64) == (12 - 4) * per_split
    assert ws(4, 129 * 64) == ws(4, 128 * 64)


def expect(code, fn, *args):
    with pytest.raises(lsv.LsvError) as e:
        fn(*args)
    assert e.value.code == code, str(e.value)
    return str(e.value)


def test_host_validation(lib):
    cfg = tiny_cfg()
    S = 0  # stream handle; never reached
    # selector
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_length, 7, 1, 4, 1, 1, 1, 4, 2.0, 2, 0, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_length, 0, 1, 65, 1, 1, 1, 4, 2.0, 2, 0, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_length, 0, 1, 4, 1, 1, 1, 5, 2.0, 2, 0, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_length, 0, 1, 4, 1, None, 1, 4, 2.0, 2, 0, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_length, 2, 1, 4, 1, None, 1, 4, 0.0, 2, 0, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_length, 2, 1, 4, 1, None, 1, 4, 2.0, 0, 0, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_length, 1, 1, 4, 1, 1, 1, 4, 2.0, 2, 4, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_length, 1, 65, 4, 1, 1, 1, 4, 2.0, 2, 0, 1, None, 1, None, S)
    # joint selection: batch, G, d_max, flags, required pointers
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_joint, 65, 4, 1, 1, 4, 0, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_joint, 2, 65, 1, 1, 4, 0, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_joint, 2, 4, 1, 1, 5, 0, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_joint, 2, 4, 1, 1, 4, 2, 1, None, None, None, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_select_joint, 2, 4, 1, None, 4, 0, 1, None, None, None, S)
    # baseline length policy: batch, bounds, required pointers, row offsets past LSV_MAX_BATCH
    g4 = [1, 1, 1, None, 1, 16, 1, None, None, S]
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_next_length_g4, *([0] + g4[1:]))
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_next_length_g4, *(g4[:4] + [0] + g4[5:]))
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_next_length_g4, *(g4[:4] + [17] + g4[5:]))
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_next_length_g4, *(g4[:5] + [lsv.LSV_MAX_SEQ_ROWS] + g4[6:]))
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_next_length_g4, *(g4[:2] + [None] + g4[3:]))
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_next_length_g4, *(g4[:6] + [None] + g4[7:]))
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_next_length_g4, *([65] + g4[1:7] + [1] + g4[8:]))
    # accept
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_accept, 3, 1, 10, 1, 1, 2, 2, 1, None, 0.0, 0, 0, 1, 1, None, None, 1,
           1 << 20, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_accept, 1, 1, 10, 1, 1, 2, 2, 1, 1, 0.0, 0, 0, 1, 1, None, None, 1,
           1 << 20, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_accept, 1, 1, 10, 1, 1, 2, 2, 1, None, 1.0, 0, 0, 1, 1, None, None, 1,
           1 << 20, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_accept, 0, 1, 10, 1, 1, 2, 65, 1, None, 0.0, 0, 0, 1, 1, None, None, 1,
           1 << 20, S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_accept, 0, 1, 10, 1, 1, 2, 2, 1, None, 0.0, 0, 0, 1, 1, None, None, 1,
           16, S)
    # verify
    args = [cfg, 1, 1, 128, 1, 1, 1, 1, 17, 128, 1, None, 1, 1 << 30, S]
    msg = expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_verify_block, *(args[:9] + [129] + args[10:]))
    assert "max_ctx" in msg
    msg = expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_verify_block, *(args[:3] + [100] + args[4:9] + [100] + args[10:]))
    assert "multiple" in msg
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_verify_block, *(args[:8] + [lsv.LSV_MAX_ROWS + 1] + args[9:]))
    msg = expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_verify_block, *(args[:3] + [1 << 23] + args[4:]))
    assert "2 GiB" in msg  # 2^23 positions x kv heads x 64 dims x 4 bytes: block offsets would not fit 32 bits
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_verify_block, *(args[:4] + [0] + args[5:]))
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_verify_block, *(args[:13] + [16] + args[14:]))
    expect(lsv.LSV_ERR_UNSUPPORTED, lsv.lsv_verify_block, *([tiny_cfg(head_dim=96)] + args[1:]))
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_verify_block, *([tiny_cfg(reserved0=1.0)] + args[1:]))
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_verify_block, *(args[:1] + [None] + args[2:]))
    # pack
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_pack_layer, cfg, 2, *([1] * 10), S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_workspace_clear, 1, 17, S)


def test_accept_noalloc_host_checks(lib):
    """The allocation-free acceptance validates like lsv_accept and refuses, before any HIP call,
    a call whose scratch would not fit the library's fixed array (LSV_ACCEPT_NOALLOC_BYTES)."""
    S = 0
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_accept_noalloc, 3, 1, 10, 1, 1, 2, 2, 1, None, 0.0, 0, 0, 1, 1, None, None,
           S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_accept_noalloc, 1, 1, 10, 1, 1, 2, 2, 1, None, 1.0, 0, 0, 1, 1, None, None,
           S)
    expect(lsv.LSV_ERR_INVALID_ARG, lsv.lsv_accept_noalloc, 0, 1, 10, None, 1, 2, 2, 1, None, 0.0, 0, 0, 1, 1, None,
           None, S)
    # 512 rows of a 300K vocabulary: 74 chunk partials per row need more than the fixed scratch
    assert lsv.lsv_accept_workspace_bytes(8, lsv.LSV_MAX_ROWS, 300000) > lsv.LSV_ACCEPT_NOALLOC_BYTES
    msg = expect(lsv.LSV_ERR_UNSUPPORTED, lsv.lsv_accept_noalloc, 0, 8, 300000, 1, 1, lsv.LSV_MAX_ROWS, 64, 1, None,
                 0.0, 0, 0, 1, 1, None, None, S)
    assert "scratch" in msg
    # the largest configurations of the workloads fit: 8 x 33 rows of 128256, 4 x 17 rows of 152064
    assert lsv.lsv_accept_workspace_bytes(8, 264, 128256) <= lsv.LSV_ACCEPT_NOALLOC_BYTES
    assert lsv.lsv_accept_workspace_bytes(4, 68, 152064) <= lsv.LSV_ACCEPT_NOALLOC_BYTES
