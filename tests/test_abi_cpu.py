"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
rejects malformed requests before touching any device state."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2608_01150_amd import api
from tests import _descs

FAKE = 0x10000  # never dereferenced: every call below fails validation first

# Calls here pass FAKE device pointers and rely on validation rejecting them
# before anything is enqueued.  On a machine with a GPU a mistake in a case
# would launch a kernel on them, so the module runs only where none is
# visible (its checks need no device).
pytestmark = pytest.mark.skipif(torch.cuda.device_count() > 0,
                                reason="fake-pointer validation tests run only without a visible GPU")


def test_exports_every_declared_symbol():
    names = api.header_symbols()
    assert {"zl_attn_fwd", "zl_attn_bwd", "zl_lse_merge", "zl_plan_dump", "zl_workspace_size",
            "zl_last_error", "zl_abi_version", "zl_shutdown", "zl_profile_enable", "zl_profile_read",
            "zl_profile_reset", "zl_attn_fwd_step", "zl_ulysses_pack_qkv", "zl_ulysses_unpack_qkv",
            "zl_ulysses_pack_out", "zl_ulysses_unpack_out", "zl_fill_pack", "zl_attn_bwd_step",
            "zl_attn_fwd_ex", "zl_lse_merge_ex"} <= set(names)
    for n in names:
        assert hasattr(api._lib, n), n


def test_abi_version():
    assert api.abi_version() == 1


def _fwd(d, H=2, hd=64, dt=api.ZL_BF16, scale=0.125, nslots=None, ptrs=(FAKE,) * 7):
    return api._fwd(d.ptr(), H, hd, dt, scale, *ptrs, d.num_slots if nslots is None else nslots, None)


def _ok_desc(**over):
    base = _descs.mixed_small()
    base.update(over)
    return api.SegDesc.of(base)


@pytest.mark.parametrize("over,needle", [
    (dict(cu_seqlens_q=(1, 200, 200, 277, 427, 460)), "cu_seqlens_q[0]"),
    (dict(cu_seqlens_q=(0, 200, 190, 277, 427, 460)), "decreases"),
    (dict(cu_seqlens_k=(0, 200, 200, 276, 577, 577, 706, 770)), "WHOLE segment 2"),
    (dict(kind=(0, 0, 0, 1, 2)), "unknown kind"),
    (dict(kv_count=(1, 1, 1, 0, 1)), "kv_count"),
    (dict(kv_count=(1, 1, 2, 3, 1)), "exactly one range"),
    (dict(kv_first=(0, 1, 2, 3, 7)), "outside"),
    (dict(block_index=(0, 0, 0, 2, 0, 3, 0)), "block_index 3"),
    (dict(block_index=(0, 0, 0, 2, 2, 1, 0)), "same slot"),
    (dict(k_offset=(0, 0, 0, 0, 250, 250, 500)), "overlap"),
    (dict(q_offset=(0, 0, 5, 0, 500)), "q_offset differs"),
    (dict(q_offset=(0, 0, 0, -1, 500)), "q_offset -1 outside"),
    (dict(k_offset=(0, 0, -3, 0, 250, 300, 500)), "k_offset -3 outside"),
])
def test_invalid_descriptors_are_rejected(over, needle):
    d = _ok_desc(**over)
    # the host-only schedule dump must reject the descriptor before the entry point sees it
    with pytest.raises(api.ZlError):
        api.plan_dump(d, 2, 64, torch.bfloat16, api.ZL_OP_FWD)
    assert _fwd(d) == api.ZL_ERR_INVALID_ARG
    assert needle in api.last_error()


def test_invalid_scalars_and_pointers():
    d = _ok_desc()
    assert _fwd(d, H=0) == api.ZL_ERR_INVALID_ARG
    assert _fwd(d, H=16385) == api.ZL_ERR_UNSUPPORTED  # ZL_MAX_HEADS + 1
    assert "exceeds 16384" in api.last_error()
    assert _fwd(d, hd=96) == api.ZL_ERR_UNSUPPORTED
    assert _fwd(d, scale=0.0) == api.ZL_ERR_INVALID_ARG
    assert _fwd(d, scale=float("nan")) == api.ZL_ERR_INVALID_ARG
    assert _fwd(d, dt=7) == api.ZL_ERR_INVALID_ARG
    assert _fwd(d, nslots=2) == api.ZL_ERR_INVALID_ARG
    assert _fwd(d, ptrs=(FAKE + 8,) + (FAKE,) * 6) == api.ZL_ERR_INVALID_ARG   # misaligned q
    assert "16-byte" in api.last_error()
    assert _fwd(d, ptrs=(FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE)) == api.ZL_ERR_INVALID_ARG  # no out
    assert _fwd(d, ptrs=(FAKE,) * 5 + (None, FAKE)) == api.ZL_ERR_INVALID_ARG  # no o_part
    assert api._fwd(None, 2, 64, 0, 0.1, *((FAKE,) * 7), 3, None) == api.ZL_ERR_INVALID_ARG


def test_backward_rules():
    d = _ok_desc()
    args = [FAKE] * 9
    # fp32 backward is not built
    st = api._bwd(d.ptr(), 2, 64, api.ZL_FP32, 0.1, *args, 0, FAKE, 1 << 40, None)
    assert st == api.ZL_ERR_UNSUPPORTED
    # unknown flags
    assert api._bwd(d.ptr(), 2, 64, api.ZL_BF16, 0.1, *args, 1, FAKE, 1 << 40, None) == api.ZL_ERR_INVALID_ARG
    # workspace too small
    need = api.workspace_size(d, 2, 64, torch.bfloat16, api.ZL_OP_BWD)
    assert need == 2 * ((460 * 2 * 4 + 255) // 256 * 256)
    st = api._bwd(d.ptr(), 2, 64, api.ZL_BF16, 0.1, *args, 0, FAKE, need - 1, None)
    assert st == api.ZL_ERR_WORKSPACE
    # shared K/V ranges are forward-only
    shared = api.SegDesc.of(_descs.desc((0, 4, 8), (1, 1), (0, 0), (2, 2), (0, 4, 8), (0, 1), 2))
    st = api._bwd(shared.ptr(), 2, 64, api.ZL_BF16, 0.1, *args, 0, FAKE, 1 << 40, None)
    assert st == api.ZL_ERR_INVALID_ARG and "at most one segment" in api.last_error()


def test_workspace_size_forward_is_zero():
    assert api.workspace_size(_ok_desc(), 3, 128, torch.bfloat16, api.ZL_OP_FWD) == 0


def test_last_error_cleared_by_success():
    d = _ok_desc()
    _fwd(d, H=0)
    assert api.last_error()
    api.workspace_size(d, 2, 64, torch.bfloat16, api.ZL_OP_FWD)
    assert api.last_error() == ""


def _step(d, flags=api.ZL_STEP_FIRST | api.ZL_STEP_LAST, ptrs=(FAKE,) * 7, H=2, hd=64):
    return api._fwd_step(d.ptr(), H, hd, api.ZL_BF16, 0.125, *ptrs, flags, None)


def _step_desc(**over):
    """mixed_small with the 150-query shard reduced to its first block (one ring step)."""
    base = _descs.desc(cu_q=(0, 200, 200, 277, 427, 460), kind=(0, 0, 0, 1, 1), kv_first=(0, 1, 2, 3, 4),
                       kv_count=(1, 1, 1, 1, 1), cu_k=(0, 200, 200, 277, 577, 641), block_index=(0, 0, 0, 0, 0),
                       num_slots=1)
    base.update(over)
    return api.SegDesc.of(base)


def test_ring_step_rules():
    # a SHARD segment must bring exactly one block per step
    assert _step(_ok_desc()) == api.ZL_ERR_INVALID_ARG and "exactly one range" in api.last_error()
    # unknown flags
    assert _step(_step_desc(), flags=4) == api.ZL_ERR_INVALID_ARG and "flags" in api.last_error()
    # without ZL_STEP_FIRST|ZL_STEP_LAST the SHARD rows need the accumulator
    ptrs = (FAKE,) * 5 + (None, None)
    for flags in (0, api.ZL_STEP_FIRST, api.ZL_STEP_LAST):
        assert _step(_step_desc(), flags=flags, ptrs=ptrs) == api.ZL_ERR_INVALID_ARG
        assert "o_acc" in api.last_error()
    # the last step needs out / lse even with no WHOLE rows
    only_shard = _descs.desc(cu_q=(0, 33), kind=(1,), kv_first=(0,), kv_count=(1,), cu_k=(0, 64), block_index=(0,),
                             num_slots=1)
    assert _step(api.SegDesc.of(only_shard), flags=api.ZL_STEP_LAST,
                 ptrs=(FAKE, FAKE, FAKE, None, None, FAKE, FAKE)) == api.ZL_ERR_INVALID_ARG
    # misaligned accumulator
    assert _step(_step_desc(), flags=0, ptrs=(FAKE,) * 5 + (FAKE + 4, FAKE)) == api.ZL_ERR_INVALID_ARG
    assert "16-byte" in api.last_error()


def _bstep(d, flags, acc=FAKE, ptrs=(FAKE,) * 9, dt=api.ZL_BF16):
    # no workspace: every call below must fail validation before any device work
    return api._bwd_step(d.ptr(), 2, 64, dt, 0.125, *ptrs, acc, flags, None, 0, None)


def test_bwd_step_rules():
    full = api.ZL_STEP_FIRST | api.ZL_STEP_LAST
    # a SHARD segment must bring exactly one block per step
    assert _bstep(_ok_desc(), full) == api.ZL_ERR_INVALID_ARG and "exactly one range" in api.last_error()
    # unknown flags, bf16 only
    assert _bstep(_step_desc(), 4) == api.ZL_ERR_INVALID_ARG and "flags" in api.last_error()
    assert _bstep(_step_desc(), full, dt=api.ZL_FP32) == api.ZL_ERR_UNSUPPORTED
    # without FIRST|LAST the SHARD rows need the dQ accumulator
    for flags in (0, api.ZL_STEP_FIRST, api.ZL_STEP_LAST):
        assert _bstep(_step_desc(), flags, acc=None) == api.ZL_ERR_INVALID_ARG and "dq_acc" in api.last_error()
    assert _bstep(_step_desc(), 0, acc=FAKE + 4) == api.ZL_ERR_INVALID_ARG and "16-byte" in api.last_error()
    # otherwise valid: the workspace is checked last
    assert _bstep(_step_desc(), full, acc=None) == api.ZL_ERR_WORKSPACE
    assert _bstep(_step_desc(), 0) == api.ZL_ERR_WORKSPACE
    # the plain backward still rejects any flag
    assert api._bwd(_step_desc().ptr(), 2, 64, api.ZL_BF16, 0.125, *(FAKE,) * 9, 1, None, 0,
                    None) == api.ZL_ERR_INVALID_ARG


def test_ulysses_rules():
    q = FAKE
    # group must divide the heads, bf16 only, head_dim 64/128
    assert api._u_pack_qkv(3, 8, 8, 128, api.ZL_BF16, q, q, q, q, None) == api.ZL_ERR_INVALID_ARG
    assert "multiple" in api.last_error()
    assert api._u_pack_qkv(0, 8, 8, 128, api.ZL_BF16, q, q, q, q, None) == api.ZL_ERR_INVALID_ARG
    assert api._u_pack_qkv(2, 8, 8, 128, api.ZL_FP32, q, q, q, q, None) == api.ZL_ERR_UNSUPPORTED
    assert api._u_pack_qkv(2, 8, 8, 96, api.ZL_BF16, q, q, q, q, None) == api.ZL_ERR_UNSUPPORTED
    assert api._u_pack_qkv(2, 8, 8, 128, api.ZL_BF16, q, None, q, q, None) == api.ZL_ERR_INVALID_ARG
    assert api._u_unpack_out(2, 8, 8, 128, api.ZL_BF16, q + 8, q, None) == api.ZL_ERR_INVALID_ARG
    assert "16-byte" in api.last_error()
    # cu_rank rules
    bad = np.array([[0, 3, 2], [0, 1, 4]], np.int32)
    assert api._u_unpack_qkv(2, 2, bad.ctypes.data_as(api._i32p), 8, 128, api.ZL_BF16, q, q, q, q,
                             None) == api.ZL_ERR_INVALID_ARG and "decreases" in api.last_error()
    bad = np.array([[1, 3, 4], [0, 1, 4]], np.int32)
    assert api._u_pack_out(2, 2, bad.ctypes.data_as(api._i32p), 8, 128, api.ZL_BF16, q, q,
                           None) == api.ZL_ERR_INVALID_ARG and "start at 0" in api.last_error()
    good = np.array([[0, 3, 4], [0, 1, 4]], np.int32)
    assert api._u_pack_out(2, 2, good.ctypes.data_as(api._i32p), 8, 128, api.ZL_BF16, None, q,
                           None) == api.ZL_ERR_INVALID_ARG
    # empty work is a no-op that needs no device
    assert api._u_pack_qkv(2, 0, 8, 128, api.ZL_BF16, None, None, None, None, None) == api.ZL_OK
    empty = np.zeros((2, 3), np.int32)
    assert api._u_unpack_qkv(2, 2, empty.ctypes.data_as(api._i32p), 8, 128, api.ZL_BF16, None, None, None, None,
                             None) == api.ZL_OK


def test_partial_dtype_rules():
    """zl_attn_fwd_ex / zl_lse_merge_ex reject an unknown partial dtype, and bf16 partials of an fp32
    forward, before looking at anything else."""
    d = _ok_desc()
    ptrs = (FAKE,) * 5
    st = api._fwd_ex(d.ptr(), 2, 64, api.ZL_BF16, 0.125, *ptrs, FAKE, 7, FAKE, d.num_slots, None)
    assert st == api.ZL_ERR_INVALID_ARG and "partial dtype" in api.last_error()
    st = api._fwd_ex(d.ptr(), 2, 64, api.ZL_FP32, 0.125, *ptrs, FAKE, api.ZL_BF16, FAKE, d.num_slots, None)
    assert st == api.ZL_ERR_UNSUPPORTED and "bf16 partials" in api.last_error()
    st = api._merge_ex(d.ptr(), 2, 64, api.ZL_BF16, FAKE, 9, FAKE, d.num_slots, FAKE, FAKE, None)
    assert st == api.ZL_ERR_INVALID_ARG and "partial dtype" in api.last_error()
