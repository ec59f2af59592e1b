"""GPU checks at the full sizes of the step and populate workloads.

* The C3 layer shape (h 4096, 32 x 128 heads, SwiGLU 12288) at reduced
  length (2 layers, prefix 128, suffix 64, 2 requests), against the fp64
  oracle at every reuse depth: every GEMM runs at its full N and K.
* The full C3 step (32 layers, B 16, prefix 1536, suffix 512) in the launch
  configuration the benchmark times, at d = 0, 8 and 32, through properties
  that hold at any size (requests are independent given the shared cache):
  a request's output rows are bit-identical whether it runs alone or in the
  batch, reversing the batch reverses the outputs bit for bit, and a repeated
  step reproduces its output exactly.
* Deep-layer reuse at the full C3 size (d = 8): a reuse step right after a
  refresh reproduces it bit for bit (1536 is a whole number of key tiles),
  and a request refreshed and reused alone gives its batch rows.
* The C4 populate (prefix 8192, 8 layers of the C3 shape): the first layer's
  cached K/V at sampled positions against the oracle, computed row by row,
  and the first cached residual, which is the exact widening of the input.
"""
import numpy as np
import pytest
import torch

from oracle import transformer as OT
import paper_2606_07571_amd as bc
from paper_2606_07571_amd import synth
from paper_2606_07571_amd.synth import to_f64, weights_f64
from tests.parity import assert_close, assert_close_bf16_store, say

pytestmark = pytest.mark.gpu


def test_c3_layer_shape_every_depth():
    cfg = synth.model_config(n_layers=2)
    B, m, n_s = 2, 128, 64
    w_cpu = synth.model_weights(cfg, 31000)
    w_dev = synth.to_device(w_cpu)
    xp, xs = synth.step_inputs(cfg, B, m, n_s, 31500)
    model = bc.Model(cfg, w_dev, cache_capacity=2)
    try:
        key = bc.prefix_key(np.arange(m))
        say(f"C3 layer shape: populate m={m}")
        model.populate(key, xp.cuda(), cfg["n_layers"])
        torch.cuda.synchronize()
        w64 = weights_f64(w_cpu)
        cache64 = OT.populate(to_f64(xp), w64, cfg, cfg["n_layers"])
        xs_dev = xs.cuda()
        for d in range(cfg["n_layers"] + 1):
            say(f"C3 layer shape: step d={d}")
            out = torch.full(tuple(xs.shape), float("nan"), device="cuda")
            model.step(key, xs_dev, d, out=out)
            torch.cuda.synchronize()
            ref = OT.step(cache64, to_f64(xs), d, w64, cfg)
            assert_close(out.cpu().double().numpy(), ref, f"C3 layer shape d={d}")
    finally:
        model.close()


@pytest.fixture(scope="module")
def c3_full():
    cfg = synth.model_config()
    sc = synth.STEP_CONFIG
    B, m, n_s = sc["B"], sc["m"], sc["n_s"]
    say("C3 full: 32-layer weights on the device")
    weights = synth.model_weights(cfg, 3000, device="cuda")
    xp, xs = synth.step_inputs(cfg, B, m, n_s, 3500, device="cuda")
    model = bc.Model(cfg, weights, cache_capacity=2)
    key = bc.prefix_key(range(m))
    say("C3 full: populate")
    model.populate(key, xp, cfg["n_layers"])
    torch.cuda.synchronize()
    yield cfg, model, key, xs
    model.close()
    del weights
    torch.cuda.empty_cache()


@pytest.mark.parametrize("d", [0, 8, 32])
def test_c3_full_size_request_independence(c3_full, d):
    cfg, model, key, xs = c3_full
    B = xs.shape[0]
    say(f"C3 full: batch step d={d}")
    out = model.step(key, xs, d)
    again = model.step(key, xs, d)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
    assert torch.equal(out, again), "repeated step differs"
    say(f"C3 full: reversed batch d={d}")
    rev = model.step(key, xs.flip(0).contiguous(), d)
    torch.cuda.synchronize()
    assert torch.equal(rev.flip(0), out), "reversing the batch does not reverse the outputs"
    for b in (0, B - 1):
        say(f"C3 full: request {b} alone d={d}")
        one = model.step(key, xs[b:b + 1].contiguous(), d)
        torch.cuda.synchronize()
        assert torch.equal(one[0], out[b]), f"request {b} alone differs from its batch rows"
    # the reuse depth changes the result (shallow layers see the cached prefix)
    if d > 0:
        base = model.step(key, xs, 0)
        torch.cuda.synchronize()
        diff = (out - base).abs().max().item()
        say(f"  max |step(d={d}) - step(0)| = {diff:.3e}")
        assert diff > 0


def test_c4_populate_first_layer_sampled():
    cfg = synth.model_config(n_layers=8)
    m = synth.POPULATE_C4["m"]
    h, Hkv, dh = cfg["hidden"], cfg["n_kv_heads"], cfg["head_dim"]
    L = synth.POPULATE_C4["n_layers_to_cache"]
    w_cpu = synth.model_weights(cfg, 41000)
    w_dev = synth.to_device(w_cpu)
    xp = synth.gaussian((m, h), 41500)
    model = bc.Model(cfg, w_dev, cache_capacity=1)
    try:
        key = bc.prefix_key(np.arange(m))
        say(f"C4 populate m={m} L={L}")
        model.populate(key, xp.cuda(), L)
        torch.cuda.synchronize()
        mem = model.cache_tensor(key)
        kv_bytes = L * 2 * Hkv * m * dh * 2
        kv0 = mem[:2 * Hkv * m * dh * 2].view(torch.bfloat16).view(2, Hkv, m, dh)
        h_off = model.cache_offset(m, L, 0, 2, 0, 0, 0)
        assert h_off == kv_bytes
        H = mem[h_off:h_off + L * m * h * 4].view(torch.float32).view(L, m, h)
        # the first cached residual is the exact widening of the prefix input
        assert torch.equal(H[0].cpu(), xp.float())
        assert torch.isfinite(H).all()
        kv_all = mem[:kv_bytes].view(torch.bfloat16)
        assert torch.isfinite(kv_all.float()).all()
        # layer-0 K/V of sampled positions (first, last, tile edges, random)
        rng = np.random.default_rng(4)
        rows = np.unique(np.concatenate([[0, 1, 63, 64, 4095, 4096, m - 2, m - 1],
                                         rng.integers(0, m, 24)]))
        w64 = weights_f64(w_cpu[:1])[0]
        _, k_ref, v_ref = OT.project_qkv(to_f64(xp)[rows], w64, cfg, rows)
        k_got = kv0[0][:, rows].cpu().double().numpy()
        v_got = kv0[1][:, rows].cpu().double().numpy()
        assert_close_bf16_store(k_got, k_ref, "C4 KV$ layer 0 K (sampled rows)")
        assert_close_bf16_store(v_got, v_ref, "C4 KV$ layer 0 V (sampled rows)")
    finally:
        model.close()


def test_c3_full_size_deep_reuse(c3_full):
    """Deep-layer reuse (second case of Eq. 5) at the full C3 size, d = 8.
    The prefix (1536) is a whole number of 64-key tiles, so a reuse step right
    after a refresh with the same input walks the same key tiles in the same
    order and reproduces the refresh output bit for bit; a request refreshed
    and reused on its own gives its batch rows bit for bit."""
    cfg, model, key, xs = c3_full
    B, n_s = xs.shape[0], xs.shape[1]
    d = 8
    store = model.new_deep_store(key, B, n_s, d)
    say(f"C3 full: refresh with deep store d={d} ({store.numel() / 2**30:.1f} GiB)")
    ref = model.step(key, xs, d, deep="refresh", deep_store=store)
    say("C3 full: reuse step, same input")
    got = model.step(key, xs, d, deep="reuse", deep_store=store)
    torch.cuda.synchronize()
    assert torch.isfinite(got).all()
    assert torch.equal(got, ref), "reuse right after refresh differs from the refresh"
    # a changed suffix: the reuse step sees the new suffix, the stale prefix K/V
    xs2 = xs.clone()
    xs2[:, -16:] = xs.flip(0)[:, -16:]
    say("C3 full: reuse step, changed suffix")
    got2 = model.step(key, xs2, d, deep="reuse", deep_store=store)
    fresh2 = model.step(key, xs2, d)
    torch.cuda.synchronize()
    assert torch.isfinite(got2).all()
    assert not torch.equal(got2, got)
    # the last request alone: refresh and reuse in a store of its own
    b = B - 1
    one_store = model.new_deep_store(key, 1, n_s, d)
    say("C3 full: last request alone")
    model.step(key, xs[b:b + 1].contiguous(), d, deep="refresh", deep_store=one_store)
    one = model.step(key, xs2[b:b + 1].contiguous(), d, deep="reuse", deep_store=one_store)
    torch.cuda.synchronize()
    assert torch.equal(one[0], got2[b])
    diff = (got2 - fresh2).abs()
    say(f"  reuse vs fresh recompute with a changed suffix: max {diff.max().item():.3e} "
        f"mean {diff.mean().item():.3e}")
    del store, one_store
    torch.cuda.empty_cache()
