"""The Python binding checks tensor extents, dtypes and device before it hands
raw pointers to the library, whose kernels trust the descriptor: a tensor
that is too small must fail here, not read out of bounds on the GPU.  These
tests use CPU tensors, so every call below stops in the binding (a shape or
dtype error, or, with correct shapes, the one-GPU check) and never reaches a
library entry point."""
import pytest
import torch

from paper_2608_01150_amd import api
from tests import _descs

BF, F32 = torch.bfloat16, torch.float32


def _desc():
    return api.SegDesc.of(_descs.mixed_small())  # Tq 460, Tk 770, 3 slots, SHARD rows end at 460


def _t(*shape, dtype=BF):
    return torch.zeros(shape, dtype=dtype)


def _raises(fn, needle):
    with pytest.raises(api.ZlError) as e:
        fn()
    assert e.value.status == api.ZL_ERR_INVALID_ARG
    assert needle in str(e.value), str(e.value)


def test_forward_checks_extents_dtypes_and_device():
    d = _desc()
    q, k, v = _t(460, 2, 64), _t(770, 2, 64), _t(770, 2, 64)
    _raises(lambda: api.attn_fwd(d, q, _t(769, 2, 64), v, 0.125), "k has shape")
    _raises(lambda: api.attn_fwd(d, _t(459, 2, 64), k, v, 0.125), "q has shape")
    _raises(lambda: api.attn_fwd(d, q, k, _t(770, 2, 64, dtype=F32), 0.125), "v has dtype")
    _raises(lambda: api.attn_fwd(d, q, k, v, 0.125, lse=_t(460, 2)), "lse has dtype")
    _raises(lambda: api.attn_fwd(d, q, k, v, 0.125, o_part=_t(2, 460, 2, 64, dtype=F32)), "o_part has shape")
    _raises(lambda: api.attn_fwd(d, _t(460, 128), k, v, 0.125), "q must be [Tq, H, d]")
    _raises(lambda: api.attn_fwd(d, q, k, v, 0.125), "one GPU")


def test_ring_accumulators_need_only_cover_the_shard_rows():
    d = _desc()
    q, k, v = _t(460, 2, 64), _t(770, 2, 64), _t(770, 2, 64)
    out, lse = _t(460, 2, 64), _t(460, 2, dtype=F32)
    _raises(lambda: api.attn_fwd_step(d, q, k, v, 0.125, out, lse, _t(459, 2, 64, dtype=F32),
                                      _t(460, 2, dtype=F32), 0), "o_acc has shape")
    # more rows than the shard rows is fine (the step reaches the device check)
    _raises(lambda: api.attn_fwd_step(d, q, k, v, 0.125, out, lse, _t(500, 2, 64, dtype=F32),
                                      _t(500, 2, dtype=F32), 0), "one GPU")


def test_backward_checks_every_tensor():
    d = _desc()
    q, k, v = _t(460, 2, 64), _t(770, 2, 64), _t(770, 2, 64)
    out, do, lse = _t(460, 2, 64), _t(460, 2, 64), _t(460, 2, dtype=F32)
    _raises(lambda: api.attn_bwd(d, q, k, v, out, lse, _t(460, 2, 32), 0.125), "dout has shape")
    _raises(lambda: api.attn_bwd(d, q, k, v, out, lse, do, 0.125, dk=_t(700, 2, 64)), "dk has shape")
    _raises(lambda: api.attn_bwd(d, q, k, v, out, lse, do, 0.125), "one GPU")
    _raises(lambda: api.attn_bwd_step(d, q, k, v, out, lse, do, 0.125, _t(460, 2, 64), _t(770, 2, 64),
                                      _t(770, 2, 64), _t(100, 2, 64, dtype=F32), 0), "dq_acc has shape")


def test_merge_checks_partials():
    d = _desc()
    out, lse = _t(460, 2, 64), _t(460, 2, dtype=F32)
    _raises(lambda: api.lse_merge(d, _t(3, 460, 2, 64, dtype=F32), _t(2, 460, 2, dtype=F32), out, lse),
            "lse_part has shape")
    _raises(lambda: api.lse_merge(d, _t(3, 460, 2, 64, dtype=F32), _t(3, 460, 2, dtype=F32), out, lse), "one GPU")


def test_ulysses_staging_checks():
    q = _t(10, 4, 64)
    _raises(lambda: api.ulysses_pack_qkv(2, q, _t(10, 4, 64), _t(11, 4, 64)), "v has shape")
    _raises(lambda: api.ulysses_pack_qkv(2, q, q, q, send=_t(2, 10, 2, 64)), "send has shape")
    cu = [[0, 3, 5], [0, 2, 4]]  # 9 rows in all
    _raises(lambda: api.ulysses_unpack_qkv(2, cu, _t(8, 2, 3, 64), 4), "recv has shape")
    _raises(lambda: api.ulysses_pack_out(2, cu, _t(9, 2, 64), 4, send=_t(9, 2, 32)), "send has shape")
    _raises(lambda: api.ulysses_unpack_out(2, _t(2, 10, 2, 64), 4, out_local=_t(10, 2, 64)), "out_local has shape")
    _raises(lambda: api.ulysses_unpack_out(2, _t(2, 10, 2, 64), 4), "one GPU")
