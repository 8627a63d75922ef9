"""Call-time argument checks on the GPU: every call below is refused on the
host with WB_EINVAL before anything is launched (null, misaligned or
too-small buffers, a workspace below the plan's size, calls before upload)."""

import pytest
import torch

import paper_2609_25442_amd as wb
from synthetic_checkpoint.workloads import WORKLOADS

from gpu_util import workspace_for

pytestmark = pytest.mark.gpu


def _expect_einval(fn, *a):
    with pytest.raises(wb.WbError) as e:
        fn(*a)
    assert e.value.code == wb.WB_EINVAL, str(e.value)
    return str(e.value)


@pytest.fixture(autouse=True)
def fresh_cache():
    # allocation-range checks see the caching allocator's segments: start each
    # test with none cached, so a small tensor sits in a small segment
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    yield


@pytest.fixture(scope="module")
def plans():
    w = WORKLOADS["llama3_8b_fsdp8_to_tp1"]
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    rp = wb.Plan(tr, ro, wb.RECEIVER, 0)
    sp = wb.Plan(tr, ro, wb.SENDER, 0)
    return tr, ro, rp, sp


def test_upload_checks(plans):
    tr, ro, rp, sp = plans
    small = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    assert rp.workspace_bytes > small.numel()
    _expect_einval(rp.upload, small)
    ws = workspace_for(rp)
    _expect_einval(lambda: wb._check(wb.lib.wb_plan_upload(rp._h, ws.data_ptr() + 16, ws.numel() - 16, None)))


def test_unpack_buffer_checks(plans):
    tr, ro, rp, sp = plans
    ws = workspace_for(rp)
    rp.upload(ws)
    dst = wb.allocate_locals(ro, 0)
    small = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    assert "smaller" in _expect_einval(rp.unpack, small, dst)
    recv = torch.empty(rp.buffer_bytes + 64, dtype=torch.uint8, device="cuda")
    assert "aligned" in _expect_einval(rp.unpack, recv[1:], dst)
    assert "null" in _expect_einval(rp.unpack, 0, dst)
    bad = list(dst)
    bad[2] = 0                                                          # a null local tensor
    _expect_einval(rp.unpack, recv, bad)
    bad[2] = dst[2]
    bad[0] = torch.empty(2 << 20, dtype=torch.bfloat16, device="cuda")  # 4 MB for the 1 GB embedding
    assert dst[0].numel() * 2 > (512 << 20)
    assert "smaller" in _expect_einval(rp.unpack, recv, bad)
    _expect_einval(rp.pack, [0] * sp.num_local_tensors, recv)          # wrong role
    del recv, dst, bad
    torch.cuda.empty_cache()


def test_pack_buffer_checks(plans):
    tr, ro, rp, sp = plans
    ws = workspace_for(sp)
    # not uploaded (through the C ABI: the binding would refuse the small buffer first)
    ptrs = (wb.c_void_p * sp.num_local_tensors)()
    buf = torch.empty(16, dtype=torch.uint8, device="cuda")
    assert "uploaded" in _expect_einval(lambda: wb._check(wb.lib.wb_pack(sp._h, ptrs, buf.data_ptr(), None)))
    sp.upload(ws)
    src = wb.allocate_locals(tr, 0)
    send = torch.empty(sp.buffer_bytes + 64, dtype=torch.uint8, device="cuda")
    _expect_einval(sp.pack, src, send[8:])
    _expect_einval(sp.pack, src, torch.empty(1 << 20, dtype=torch.uint8, device="cuda"))
    _expect_einval(sp.pack, src[:-1] + [0], send)
    del src, send
    torch.cuda.empty_cache()


def test_forward_and_probe_checks():
    w = WORKLOADS["mixtral_ep8fsdp2_to_ep2"]
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    rp = wb.Plan(tr, ro, wb.RECEIVER, 0, node_size=1)
    assert rp.forward_bytes(1) > (64 << 20)
    ws = workspace_for(rp)
    rp.upload(ws)
    small = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    _expect_einval(rp.forward_round, 0, 1, small, small)              # receive buffer too small
    _expect_einval(rp.forward_round, 0, 3, small, small)              # no such stage
    x = torch.empty(1024, dtype=torch.bfloat16, device="cuda")
    _expect_einval(lambda: wb._check(wb.lib.wb_make_ids(x.data_ptr() + 1, wb.DTYPES["bf16"], 100, 1 << 24, 0, 16, None)))
    _expect_einval(lambda: wb._check(wb.lib.wb_make_ids(x.data_ptr(), wb.DTYPES["bf16"], 100, 1 << 24, 0, 8, None)))
    idx = torch.empty(16, dtype=torch.int64, device="cuda")
    val = torch.empty(16, dtype=torch.int32, device="cuda")
    cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
    _expect_einval(lambda: wb._check(wb.lib.wb_diff2(x.data_ptr() + 1, wb.DTYPES["bf16"], 4, 4, idx.data_ptr(),
                                                     val.data_ptr(), 16, cnt.data_ptr(), None)))
    _expect_einval(lambda: wb._check(wb.lib.wb_diff2(x.data_ptr(), wb.DTYPES["bf16"], 4, 4, idx.data_ptr(),
                                                     val.data_ptr(), 16, cnt.data_ptr() + 4, None)))
    f = [([x, x], "bf16", 16, 64)]
    arr = wb._field_array(f)
    need = wb.diff2_batch_workspace(f)
    ws = torch.empty(need + 64, dtype=torch.uint8, device="cuda")
    v64 = torch.empty(16, dtype=torch.int64, device="cuda")

    def batch(ws_ptr, ws_bytes, value_ptr, count_ptr, fields=arr):
        return wb._check(wb.lib.wb_diff2_batch(fields, 1, ws_ptr, ws_bytes, idx.data_ptr(), value_ptr, 16, count_ptr,
                                               None))

    assert "workspace" in _expect_einval(batch, ws.data_ptr(), need - 8, v64.data_ptr(), cnt.data_ptr())
    _expect_einval(batch, ws.data_ptr() + 4, need, v64.data_ptr(), cnt.data_ptr())        # misaligned workspace
    _expect_einval(batch, ws.data_ptr(), need, v64.data_ptr() + 4, cnt.data_ptr())        # misaligned values
    _expect_einval(batch, ws.data_ptr(), need, v64.data_ptr(), cnt.data_ptr() + 4)        # misaligned count
    bad = wb._field_array([([x.data_ptr() + 1, x.data_ptr()], "bf16", 16, 64)])
    assert "aligned" in _expect_einval(batch, ws.data_ptr(), need, v64.data_ptr(), cnt.data_ptr(), bad)
    torch.cuda.synchronize()


def _hip_pointer_type(ptr: int):
    """The HIP runtime's own classification of an address (hipPointerGetAttributes:
    None on an error, else the hipMemoryType; 0 is unregistered host memory)."""
    import ctypes

    class Attr(ctypes.Structure):
        _fields_ = [("type", ctypes.c_int), ("device", ctypes.c_int), ("devicePointer", ctypes.c_void_p),
                    ("hostPointer", ctypes.c_void_p), ("isManaged", ctypes.c_int), ("allocationFlags", ctypes.c_uint)]

    hip = ctypes.CDLL("libamdhip64.so.7")
    a = Attr()
    rc = hip.hipPointerGetAttributes(ctypes.byref(a), ctypes.c_void_p(ptr))
    if rc != 0:
        hip.hipGetLastError()
        return None
    return a.type


def test_pageable_host_memory_refused(plans):
    """Pageable host memory given as raw pointers is refused on the host before
    any launch. The runtime must classify it as the library's check expects
    (an error or type 0) before the library is handed it."""
    tr, ro, rp, sp = plans
    host = torch.empty(1 << 20, dtype=torch.uint8)            # pageable
    pinned = torch.empty(1 << 20, dtype=torch.uint8, pin_memory=True)
    assert _hip_pointer_type(pinned.data_ptr()) == 1            # hipMemoryTypeHost
    kind = _hip_pointer_type(host.data_ptr())
    if kind not in (None, 0):
        pytest.skip(f"runtime reports pageable memory as type {kind}")
    msg = _expect_einval(lambda: wb._check(wb.lib.wb_make_ids(host.data_ptr(), wb.DTYPES["bf16"], 100, 1 << 24, 0, 16,
                                                              None)))
    assert "pageable" in msg or "address" in msg
    ws = workspace_for(rp)
    rp.upload(ws)
    dst = wb.allocate_locals(ro, 0)
    ptrs = (wb.c_void_p * len(dst))(*[t.data_ptr() for t in dst])
    msg = _expect_einval(lambda: wb._check(wb.lib.wb_unpack(rp._h, host.data_ptr(), ptrs, None)))
    assert "recv_buf" in msg and ("pageable" in msg or "address" in msg)
    # the binding refuses pageable tensors itself
    assert "pinned" in _expect_einval(rp.unpack, host, dst)
    del dst
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
