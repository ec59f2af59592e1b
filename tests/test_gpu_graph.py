"""HIP graph capture of the library's calls (torch.cuda.graph over the
stream the binding passes): a whole denoising step at a depth with shallow
and deep layers, and the allocation-free similarity reduction.  Each graph is
replayed several times with eager work of the same kernels in between, and
every replay must give the eager result bit for bit.  The step enqueues only
kernel launches (no memset, no allocation: its workspace is the caller's)."""
import numpy as np
import pytest
import torch

import paper_2606_07571_amd as bc
from paper_2606_07571_amd import synth
from tests.parity import say

pytestmark = pytest.mark.gpu


def test_step_replays_from_a_graph():
    cfg = synth.model_config(n_layers=3, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn=512)
    B, m, n_s, d = 3, 129, 65, 1
    model = bc.Model(cfg, synth.to_device(synth.model_weights(cfg, 91000)), cache_capacity=1)
    try:
        xp, xs = synth.step_inputs(cfg, B, m, n_s, 91500, device="cuda")
        xs2 = synth.gaussian(tuple(xs.shape), 91600, device="cuda")
        key = bc.prefix_key(np.arange(m))
        model.populate(key, xp, cfg["n_layers"])
        static_in = xs.clone()
        static_out = torch.empty((B, n_s, cfg["hidden"]), dtype=torch.float32, device="cuda")
        # eager references (this also sizes the binding's workspace before capture)
        ref = model.step(key, xs, d).clone()
        ref2 = model.step(key, xs2, d).clone()
        torch.cuda.synchronize()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            model.step(key, static_in, d, out=static_out)      # warm-up on the capture stream
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        say("graph: capturing a step")
        with torch.cuda.graph(g):
            model.step(key, static_in, d, out=static_out)
        for rep, (inp, want) in enumerate([(xs, ref), (xs2, ref2), (xs, ref)]):
            static_in.copy_(inp)
            static_out.fill_(float("nan"))
            say(f"graph: replay {rep}")
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(static_out, want), f"replay {rep} differs from the eager step"
            # eager work of the same kernels between replays
            other = model.step(key, xs2 if rep % 2 == 0 else xs, d)
            torch.cuda.synchronize()
            assert torch.isfinite(other).all()
        del g
    finally:
        model.close()


def test_noalloc_similarity_replays_from_a_graph():
    n = 8 * 300_001
    a = synth.gaussian((n,), 92000, device="cuda")
    b = synth.gaussian((n,), 92001, device="cuda")
    c = synth.gaussian((n,), 92002, device="cuda")
    out = torch.zeros(1, dtype=torch.float64, device="cuda")
    ref_ab = bc.cosine_similarity(a, b).item()
    ref_ac = bc.cosine_similarity(a, c).item()
    sa, sb = a.clone(), b.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        bc.cosine_similarity_noalloc(sa, sb, out)          # warm-up: looks up the scratch address
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        bc.cosine_similarity_noalloc(sa, sb, out)
    for rep, (other, want) in enumerate([(b, ref_ab), (c, ref_ac), (b, ref_ab)]):
        sb.copy_(other)
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert out.item() == want, f"replay {rep}: {out.item()!r} != {want!r}"
        # eager use of the same scratch between replays
        bc.cosine_similarity_noalloc(a, c, out)
        torch.cuda.synchronize()
        assert out.item() == ref_ac
    del g
