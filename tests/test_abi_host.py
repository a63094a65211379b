"""Host-side checks of the C ABI (no GPU work is launched).

The library loads, exports every function include/moe.h declares, and
rejects bad arguments with the documented status codes before enqueuing
anything.
"""
import ctypes
import os
import re

import pytest

import paper_2606_10493_amd as moe

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "moe.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s+(moe_[a-z0-9_]+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_documented_entry_points():
    names = _declared_functions()
    for n in ("moe_quant_act", "moe_pack_weight", "moe_permute", "moe_expert_ffn", "moe_combine", "moe_ffn_streamed",
              "moe_status_string", "moe_permute_workspace", "moe_expert_ffn_workspace"):
        assert n in names


def test_library_exports_every_declared_function():
    lib = ctypes.CDLL(moe.LIB_PATH)
    missing = [n for n in _declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    # the binding declares a signature for every exported entry point too
    assert set(_declared_functions()) <= set(moe.EXPORTED_SYMBOLS)


def test_status_strings():
    assert moe.moe_status_string(moe.MOE_OK) == "MOE_OK"
    assert moe.moe_status_string(moe.MOE_ERR_WORKSPACE) == "MOE_ERR_WORKSPACE"
    assert moe.moe_status_string(-99) == "MOE_ERR_UNKNOWN"


def test_argument_errors_return_before_any_launch():
    lib = moe.lib
    P = ctypes.c_void_p
    fake = P(0x1000)
    assert lib.moe_quant_act(fake, 4, 100, fake, fake, None) == moe.MOE_ERR_UNSUPPORTED_SHAPE
    assert lib.moe_quant_act(None, 4, 128, fake, fake, None) == moe.MOE_ERR_INVALID_ARG
    assert lib.moe_quant_act(None, 0, 128, None, None, None) == moe.MOE_OK      # empty: no-op
    assert lib.moe_quant_weight(fake, 1, 100, 128, fake, fake, None) == moe.MOE_ERR_UNSUPPORTED_SHAPE
    assert lib.moe_pack_weight(fake, 1, 24, 128, P(0x2000), None) == moe.MOE_ERR_UNSUPPORTED_SHAPE
    assert lib.moe_pack_weight(fake, 1, 16, 100, P(0x2000), None) == moe.MOE_ERR_UNSUPPORTED_SHAPE
    assert lib.moe_pack_weight(fake, 1, 16, 128, fake, None) == moe.MOE_ERR_INVALID_ARG      # in place
    assert lib.moe_pack_weight(None, 1, 16, 128, fake, None) == moe.MOE_ERR_INVALID_ARG
    assert lib.moe_pack_weight(None, 0, 16, 128, None, None) == moe.MOE_OK                   # empty: no-op
    assert lib.moe_permute(fake, 4, 9, 8, fake, fake, fake, None, None, 0, None) == moe.MOE_ERR_INVALID_ARG
    assert lib.moe_permute(fake, 4, 2, 2000, fake, fake, fake, None, None, 0, None) == moe.MOE_ERR_INVALID_ARG
    # more than one chunk of tokens needs the workspace
    assert lib.moe_permute(fake, 1000, 2, 8, fake, fake, fake, None, None, 0, None) == moe.MOE_ERR_WORKSPACE
    assert lib.moe_combine(fake, fake, fake, 3, 2, 100, fake, None) == moe.MOE_ERR_UNSUPPORTED_SHAPE
    d = moe.MoeDims(7168, 2048, 256, 8)
    args = [fake] * 10
    assert lib.moe_expert_ffn(moe.MoeDims(7000, 2048, 256, 8), 1, 0, *args, fake, None, 0, None) == \
        moe.MOE_ERR_UNSUPPORTED_SHAPE
    assert lib.moe_expert_ffn(moe.MoeDims(7168, 2048, 4, 8), 1, 0, *args, fake, None, 0, None) == \
        moe.MOE_ERR_INVALID_ARG
    assert lib.moe_expert_ffn(d, 65, moe.MOE_REGIME_DECODE, *args, fake, None, 0, None) == moe.MOE_ERR_INVALID_ARG
    assert lib.moe_expert_ffn(d, 1, 7, *args, fake, None, 0, None) == moe.MOE_ERR_INVALID_ARG
    assert lib.moe_expert_ffn(d, 1, 0, *args, fake, None, 0, None) == moe.MOE_ERR_WORKSPACE
    assert "workspace" in moe.moe_last_error()
    assert lib.moe_ffn_streamed(d, 4, 0, *([fake] * 11), None, fake, None, fake, 1 << 40, None, None) == \
        moe.MOE_ERR_INVALID_ARG   # chunk_tokens = 0
    assert lib.moe_ffn_streamed(d, 4, 2, *([fake] * 11), None, fake, None, fake, 1 << 40, None, None) == \
        moe.MOE_ERR_INVALID_ARG   # no stream context


def test_workspace_sizes():
    d = moe.MoeDims(7168, 2048, 256, 8)
    assert moe.moe_permute_workspace(1, 8, 256) > 0
    assert moe.moe_permute_workspace(8192, 8, 256) >= 2 * 32 * 257 * 4
    dec = moe.moe_expert_ffn_workspace(d, 4, moe.MOE_REGIME_DECODE)
    assert dec >= 4 * 8 * 2048 * 5          # qh + fp32 h
    pre = moe.moe_expert_ffn_workspace(d, 8192, moe.MOE_REGIME_PREFILL)
    assert pre >= 8192 * 8 * 2048
    assert moe.moe_ring_bytes(d, 256) == 256 * 3 * 7168 * 2048
    assert moe.moe_ring_scale_bytes(d, 2) == 2 * 3 * 56 * 16 * 4
    assert moe.moe_ffn_streamed_workspace(d, 32768, 4096) >= 32768 * 8 * 7168 * 4


@pytest.mark.parametrize("bad", [0, -1, 5000])
def test_stream_context_rejects_bad_slot_counts(bad):
    with pytest.raises(moe.MoEError):
        moe.StreamContext(bad)
