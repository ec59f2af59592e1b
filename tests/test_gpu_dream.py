"""GPU checks of the full step at the Dream-7B shape (GQA 28/4 x 128 heads,
hidden 3584, SwiGLU 18944, Q/K/V bias).

* A small GQA model with Q/K/V bias at every reuse depth against the oracle
  (the bias path on every projection kind: shallow, deep, populate).
* The Dream-7B layer width at reduced length (2 layers, prefix 64, suffix 33,
  2 requests) against the oracle at every depth: every GEMM at its full N and
  K, the 7-query-head groups, the bias.
* The full Dream-shaped step (28 layers, 64 requests, prefix 1024, suffix 384,
  the benchmark's seeds) against the fp64 oracle on requests 0 and 63 at
  d = 0 and 8 (the depths the benchmark times), and at d = 0, 8 and 28
  through properties that hold at any size: repeat runs and a request run
  alone are bit-identical to the batch rows, and d > 0 differs from d = 0.
"""
import numpy as np
import pytest
import torch

from oracle import transformer as OT
import paper_2606_07571_amd as bc
from paper_2606_07571_amd import synth
from paper_2606_07571_amd.synth import to_f64, weights_f64
from tests.parity import DeviceLayersF64, assert_close, say

pytestmark = pytest.mark.gpu


def _parity_every_depth(cfg, B, m, n_s, seed, label):
    w_cpu = synth.model_weights(cfg, seed)
    assert all(lw["b_qkv"] is not None for lw in w_cpu)
    model = bc.Model(cfg, synth.to_device(w_cpu), cache_capacity=2)
    try:
        xp, xs = synth.step_inputs(cfg, B, m, n_s, seed + 500)
        key = bc.prefix_key(np.arange(m) + seed)
        say(f"{label}: populate m={m}")
        model.populate(key, xp.cuda(), cfg["n_layers"])
        torch.cuda.synchronize()
        w64 = weights_f64(w_cpu)
        cache64 = OT.populate(to_f64(xp), w64, cfg, cfg["n_layers"])
        xs_dev = xs.cuda()
        for d in range(cfg["n_layers"] + 1):
            say(f"{label}: step d={d}")
            out = torch.full(tuple(xs.shape), float("nan"), device="cuda")
            model.step(key, xs_dev, d, out=out)
            torch.cuda.synchronize()
            ref = OT.step(cache64, to_f64(xs), d, w64, cfg)
            assert_close(out.cpu().double().numpy(), ref, f"{label} d={d}")
    finally:
        model.close()


def test_small_gqa_with_bias_every_depth():
    cfg = synth.model_config(n_layers=3, hidden=448, n_heads=7, n_kv_heads=1, head_dim=64, ffn=640,
                             rms_eps=1e-6, rope_theta=1e6, qkv_bias=True)
    _parity_every_depth(cfg, B=3, m=70, n_s=29, seed=71000, label="small GQA+bias")


def test_dream_layer_width_every_depth():
    cfg = synth.dream_config(n_layers=2)
    _parity_every_depth(cfg, B=2, m=64, n_s=33, seed=72000, label="Dream width")


@pytest.fixture(scope="module")
def dream_full():
    cfg = synth.dream_config()
    sc = synth.DREAM_STEP
    B, m, n_s = sc["B"], sc["m"], sc["n_s"]
    say("Dream full: 28-layer weights on the device")
    weights = synth.model_weights(cfg, 8000, device="cuda")
    xp, xs = synth.step_inputs(cfg, B, m, n_s, 8500, device="cuda")
    model = bc.Model(cfg, weights, cache_capacity=1)
    key = bc.prefix_key(range(m))
    say("Dream full: populate")
    model.populate(key, xp, cfg["n_layers"])
    torch.cuda.synchronize()
    yield cfg, model, key, xs, weights, xp
    model.close()
    del weights
    torch.cuda.empty_cache()


DREAM_DEPTHS = (0, 8)


@pytest.fixture(scope="module")
def dream_oracle(dream_full):
    """The oracle's prefix-only forward over the 8 layers d = 8 reuses, on the
    device weights widened to fp64 on first use."""
    cfg, model, key, xs, weights, xp = dream_full
    W = DeviceLayersF64(weights)
    say("Dream full: oracle populate of 8 layers (fp64)")
    cache = OT.populate(to_f64(xp), W, cfg, max(DREAM_DEPTHS))
    yield W, cache
    del W, cache


@pytest.mark.parametrize("d,b", [(d, b) for d in DREAM_DEPTHS for b in (0, 63)])
def test_dream_full_step_oracle_parity(dream_full, dream_oracle, d, b):
    """The benchmark's Dream-7B-shaped workload, element by element against
    the fp64 oracle (GQA 28/4, Q/K/V bias, Eq. 4 below d, the refresh case
    of Eq. 5 from d on)."""
    cfg, model, key, xs, weights, xp = dream_full
    W, cache = dream_oracle
    say(f"Dream full: GPU step d={d}")
    out = torch.full(tuple(xs.shape), float("nan"), device="cuda")
    model.step(key, xs, d, out=out)
    torch.cuda.synchronize()
    got = out[b].cpu().double().numpy()
    say(f"Dream full: oracle step d={d} request {b}")
    ref = OT.step(cache, to_f64(xs[b:b + 1]), d, W, cfg)[0]
    assert_close(got, ref, f"Dream full step d={d} request {b}")


@pytest.mark.parametrize("d", [0, 8, 28])
def test_dream_full_step_properties(dream_full, d):
    cfg, model, key, xs = dream_full[:4]
    B = xs.shape[0]
    say(f"Dream full: step d={d}")
    out = model.step(key, xs, d)
    again = model.step(key, xs, d)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
    assert torch.equal(out, again)
    for b in (0, B - 1):
        say(f"Dream full: request {b} alone d={d}")
        one = model.step(key, xs[b:b + 1].contiguous(), d)
        torch.cuda.synchronize()
        assert torch.equal(one[0], out[b])
    if d > 0:
        base = model.step(key, xs, 0)
        torch.cuda.synchronize()
        assert (out - base).abs().max().item() > 0
