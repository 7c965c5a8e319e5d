"""catekv_select_critical_noalloc, the selection for callers that cannot
allocate device memory, against catekv_select_critical with a caller
workspace: bit-identical chunk indices on two calls in a row, the second on a
smaller input (the shared scratch keeps the first call's contents)."""
import ctypes
import sys

import pytest
import torch

import paper_2608_30295_amd as ck
from paper_2608_30295_amd._lib import lib

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _select_noalloc(q, k, heads, cs, b):
    hq, l_obs, d = q.shape
    hkv, n, _ = k.shape
    idx = torch.full((len(heads), b), -7, dtype=torch.int32, device=DEV)
    harr = (ctypes.c_int32 * len(heads))(*heads)
    rc = lib().catekv_select_critical_noalloc(1, q.data_ptr(), k.data_ptr(), hq, hkv, l_obs, n, d, cs, harr,
                                              len(heads), b, idx.data_ptr(),
                                              torch.cuda.current_stream().cuda_stream)
    return rc, idx


def test_select_noalloc_matches_the_workspace_call():
    g = torch.Generator(device=DEV).manual_seed(3)
    # the benchmark's 128K selection, then a smaller one (other heads, window and budget)
    for n, heads, l_obs, b in [(131072, [1, 2, 3, 4, 5], 64, 256), (20000 + 37, [6, 0], 32, 100)]:
        print(f"select noalloc n={n} heads={heads} l_obs={l_obs} b={b}", flush=True)
        sys.stdout.flush()
        k = torch.randn((8, n, 128), generator=g, device=DEV).to(torch.bfloat16)
        q = torch.randn((32, l_obs, 128), generator=g, device=DEV).to(torch.bfloat16)
        want = ck.select_critical(q, k, heads, 8, b)
        rc, got = _select_noalloc(q, k, heads, 8, b)
        torch.cuda.synchronize()
        assert rc == 0, lib().catekv_last_error().decode()
        assert torch.equal(got, want)
        assert int((got >= 0).sum()) == len(heads) * b
