"""vie_dense_topk_noalloc (the dense head on the library's static per-GPU
workspace, for callers that cannot allocate) against vie_dense_topk with a
caller workspace: the same ids and the same logit bits on two calls in a
row, the second smaller than the first, both through the C ABI."""
import ctypes as C
import os
import sys

import numpy as np
import pytest

from paper_2608_27460_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _ptr(t):
    return C.c_void_p(t.data_ptr())


def _call_both(vie, V, d, dtype, B, k, seed):
    W = synth.make_w(V, d, dtype, seed)
    H, _ = synth.make_queries(W, dtype, B, seed + 1)
    Wd = vie.host_to_torch(W, dtype).cuda()
    Hd = vie.host_to_torch(H, dtype).cuda()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    n = C.c_size_t()
    assert vie.lib.vie_dense_topk_workspace(V, d, B, k, C.byref(n)) == vie.OK
    ws = torch.empty(n.value, dtype=torch.uint8, device="cuda")
    ref_i = torch.empty((B, k), dtype=torch.int32, device="cuda")
    ref_l = torch.empty((B, k), dtype=torch.float32, device="cuda")
    got_i = torch.full((B, k), -7, dtype=torch.int32, device="cuda")
    got_l = torch.full((B, k), 7.0, dtype=torch.float32, device="cuda")
    assert vie.lib.vie_dense_topk(_ptr(Wd), dtype, V, d, _ptr(Hd), B, k, _ptr(ref_i), _ptr(ref_l), _ptr(ws),
                                  n.value, stream) == vie.OK
    assert vie.lib.vie_dense_topk_noalloc(_ptr(Wd), dtype, V, d, _ptr(Hd), B, k, _ptr(got_i), _ptr(got_l),
                                          stream) == vie.OK, vie.lib.vie_last_error()
    torch.cuda.synchronize()
    assert np.array_equal(got_i.cpu().numpy(), ref_i.cpu().numpy())
    assert np.array_equal(got_l.cpu().numpy().view(np.uint32), ref_l.cpu().numpy().view(np.uint32))


def test_noalloc_dense_matches_the_workspace_entry_point():
    assert torch.cuda.is_available(), "the gpu tests need an MI355X"
    from paper_2608_27460_amd import vie
    print("noalloc: matrix-core path, V=20011 d=256 B=16 k=50", flush=True)
    _call_both(vie, 20011, 256, synth.BF16, 16, 50, 71)
    print("noalloc: smaller, vector path, V=5003 d=128 B=1 k=20", flush=True)
    _call_both(vie, 5003, 128, synth.BF16, 1, 20, 72)
    print("noalloc: fp32 rows, V=4000 d=96 B=3 k=40", flush=True)
    _call_both(vie, 4000, 96, synth.F32, 3, 40, 73)
    # more than the static workspace holds: refused before anything is enqueued
    fake = C.c_void_p(4096)
    assert vie.lib.vie_dense_topk_noalloc(fake, synth.BF16, 262144, 640, fake, 64, 50, fake, fake,
                                          None) == vie.EUNSUPPORTED
    assert b"static one holds" in vie.lib.vie_last_error()
