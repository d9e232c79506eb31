"""foremoe_dispatch_static: steps 1-3 with the workspace in the library's
static device array (the call allocates nothing) against
foremoe_histogram_assign + foremoe_permute with a caller workspace. Outputs
must be bitwise equal, on two calls in a row, the second with a smaller
input (the array keeps the first call's contents)."""
import ctypes

import numpy as np
import pytest
import torch

from tests.gpu_helpers import config_workload, custom_workload, tdtype, to_dev


def _static_dispatch(lib, _lib, w, m, dev):
    """Steps 1-3 through foremoe_dispatch_static into preallocated,
    sentinel-filled outputs; returns them and the status words."""
    from paper_2606_11867_amd import api
    T, K = m.ids.shape
    n_cap = T * K
    plan = api.DevicePlan.from_host(m.plan, dev)
    cp = plan.c_struct()
    ids = torch.from_numpy(m.ids).to(dev)
    x = to_dev(w.x(m.index), tdtype(w), dev)
    nkeys = plan.E * max(plan.n_src, 1)
    i32 = dict(dtype=torch.int32, device=dev)
    out = dict(counts=torch.full((nkeys,), -7, **i32),
               rep_begin=torch.full((nkeys * (plan.R_max + 1),), -7, **i32),
               slot_count=torch.full((max(plan.S, 1),), -7, **i32),
               slot_offset=torch.full((plan.S + 1,), -7, **i32),
               x_perm=torch.zeros((n_cap, x.shape[1]), dtype=x.dtype, device=dev),
               row_to_pair=torch.full((n_cap,), -7, **i32), pair_to_row=torch.full((T * K,), -7, **i32),
               status=torch.full((3,), -7, **i32))
    rc = lib.foremoe_dispatch_static(
        ids.data_ptr(), T, K, ctypes.byref(cp), x.data_ptr(), _lib.BF16 if x.dtype == torch.bfloat16 else _lib.F32,
        x.shape[1], n_cap, out["counts"].data_ptr(), out["rep_begin"].data_ptr(), out["slot_count"].data_ptr(),
        out["slot_offset"].data_ptr(), out["x_perm"].data_ptr(), out["row_to_pair"].data_ptr(),
        out["pair_to_row"].data_ptr(), out["status"].data_ptr(), torch.cuda.current_stream(dev).cuda_stream)
    assert rc == 0, lib.foremoe_last_error()
    return out, plan, ids, x, n_cap


@pytest.mark.gpu
def test_dispatch_static_matches_workspace_calls(gpu):
    from paper_2606_11867_amd import _lib, api
    lib = _lib.load()
    cases = [("qwen3-30b-a3b EP=8 share, measured micro-step", config_workload("qwen3-30b-a3b-ep8-share"), None),
             ("custom share T=2048 K=4 E=32, micro-step 1", custom_workload("share"), 1)]
    for label, w, idx in cases:
        m = w.micro[w.measured if idx is None else idx]
        print(f"\n[case] dispatch_static: {label}, T={m.ids.shape[0]} K={m.ids.shape[1]} S={m.plan.S}", flush=True)
        got, plan, ids, x, n_cap = _static_dispatch(lib, _lib, w, m, gpu)
        ws = api.workspace(ids.shape[0], ids.shape[1], plan.E, gpu)
        counts, rb, sc, so = api.histogram_assign(ids, plan, ws)
        x_perm, r2p, p2r = api.permute(x, ids, plan, rb, so, n_cap, ws)
        torch.cuda.synchronize()
        N = int(so[-1].item())
        assert N > 0
        assert torch.equal(got["counts"], counts)
        assert torch.equal(got["rep_begin"], rb.reshape(-1))
        assert torch.equal(got["slot_count"][:plan.S], sc)
        assert torch.equal(got["slot_offset"], so)
        assert torch.equal(got["pair_to_row"], p2r)
        assert torch.equal(got["row_to_pair"][:N], r2p[:N])
        assert torch.equal(got["x_perm"][:N].view(torch.int16), x_perm[:N].view(torch.int16))
        status = ws[:256].view(torch.int32)[:3]
        assert torch.equal(got["status"], status)
        assert got["status"].cpu().tolist() == [0, 0, 0]


def test_dispatch_static_rejects_oversized_inputs():
    """Inputs whose workspace would not fit the static array are refused on
    the host, before any HIP call."""
    import os
    import paper_2606_11867_amd as fm
    from paper_2606_11867_amd import _lib
    if not os.path.exists(fm.LIB_PATH):
        from paper_2606_11867_amd import build
        build.build()
    lib = fm.load()
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: the size check fails first
    plan = _lib.Plan(256, 4, 2, 0, fake, fake, fake, None, fake, fake)
    T, K = 1 << 20, 8  # 16384 blocks x 257 keys x 4 bytes > 8 MiB
    assert lib.foremoe_workspace_size(T, K, 256) > _lib.STATIC_SCRATCH_BYTES
    rc = lib.foremoe_dispatch_static(fake, T, K, ctypes.byref(plan), fake, _lib.BF16, 2048, T * K, fake, fake,
                                     fake, fake, fake, fake, fake, None, None)
    assert rc == _lib.EINVAL
    assert b"static array" in lib.foremoe_last_error()
