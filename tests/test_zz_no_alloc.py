"""The allocation-free entry point (bc_cosine_similarity_noalloc) against the
entry point with a caller workspace (bc_cosine_similarity), through the C ABI:
two calls in a row, the second on a smaller input, give the same bits as the
workspace entry point (same kernels, same fixed-order reduction); sizes
beyond the static scratch are refused; the calls change no device memory
reservation."""
import ctypes as C

import numpy as np
import pytest
import torch

import paper_2606_07571_amd as bc
from paper_2606_07571_amd import synth
from tests.parity import say

pytestmark = pytest.mark.gpu

MAX_N = 130_146_304   # 15,887 workgroup partials of 8192 elements


def _vectors(n, seed):
    a = synth.gaussian((n,), seed, device="cuda")
    noise = synth.gaussian((n,), seed + 1, device="cuda").float()
    b = (a.float() * 0.9 + 0.3 * noise).to(torch.bfloat16)
    return a, b


def _noalloc(a, b, n, out):
    L = bc.lib()
    st = L.bc_cosine_similarity_noalloc(C.c_void_p(a.data_ptr()), C.c_void_p(b.data_ptr()), n,
                                        C.c_void_p(out.data_ptr()),
                                        C.c_void_p(torch.cuda.current_stream().cuda_stream))
    return st


def test_noalloc_matches_workspace_entry_point():
    torch.cuda.set_device(0)
    # first the largest size the scratch serves, then two smaller ones: the
    # partials a later, smaller call leaves untouched must not reach its result
    for n, seed in ((MAX_N, 61000), (5_000_008, 61010), (8 * 1001, 61020)):
        say(f"no-alloc cosine: n={n}")
        a, b = _vectors(n, seed)
        ref = bc.cosine_similarity(a, b)
        torch.cuda.synchronize()
        out = torch.full((1,), float("nan"), dtype=torch.float64, device="cuda")
        free0 = torch.cuda.mem_get_info()[0]
        assert _noalloc(a, b, n, out) == 0, bc.lib().bc_last_error().decode()
        torch.cuda.synchronize()
        assert torch.cuda.mem_get_info()[0] == free0
        got, want = out.item(), ref.item()
        say(f"  noalloc {got!r} workspace {want!r}")
        assert np.isfinite(got)
        assert got == want, "no-alloc result differs from the workspace entry point"
        # and against fp64 on the host, on the small case
        if n <= 10_000_000:
            x = a.double().cpu().numpy()
            y = b.double().cpu().numpy()
            exact = float(x @ y) / (np.linalg.norm(x) * np.linalg.norm(y))
            assert abs(got - exact) <= 1e-6
        del a, b


def test_noalloc_refuses_sizes_beyond_scratch():
    a = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    out = torch.zeros(1, dtype=torch.float64, device="cuda")
    L = bc.lib()
    st = L.bc_cosine_similarity_noalloc(C.c_void_p(a.data_ptr()), C.c_void_p(a.data_ptr()), MAX_N + 8,
                                        C.c_void_p(out.data_ptr()), None)
    assert st == -6
    assert "static scratch" in L.bc_last_error().decode()
