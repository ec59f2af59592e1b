"""GPU parity of a batch over several cached prefixes (multi-tenant batches).

* Three groups with prefixes of different (ragged) lengths in one batch, at
  every reuse depth, against the fp64 oracle request by request.
* Each group's rows are bit-identical to the single-prefix step of that group
  alone: the batch-wide kernels are row-independent and the per-group ones see
  the same inputs.
* A key that appears in two groups, group order, and the error paths (a key
  not cached, counts that do not cover the batch, d beyond a partial entry).
* At the full C3 layer shape, two prefixes (1536 and 1024 tokens, 8 requests
  each, d = 8): each group bit-identical to its single-prefix step.
"""
import numpy as np
import pytest
import torch

from oracle import transformer as OT
import paper_2606_07571_amd as bc
from paper_2606_07571_amd import synth
from paper_2606_07571_amd.synth import to_f64, weights_f64
from tests.parity import assert_close, say

pytestmark = pytest.mark.gpu

CFG = synth.model_config(n_layers=3, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn=512)
PREFIX_M = (129, 64, 200)
COUNTS = (2, 1, 3)
N_S = 65


@pytest.fixture(scope="module")
def multi():
    cfg = CFG
    w_cpu = synth.model_weights(cfg, 51000)
    w_dev = synth.to_device(w_cpu)
    w64 = weights_f64(w_cpu)
    model = bc.Model(cfg, w_dev, cache_capacity=8)
    keys, caches = [], []
    for g, m in enumerate(PREFIX_M):
        xp = synth.gaussian((m, cfg["hidden"]), 51100 + g)
        key = bc.prefix_key(np.arange(m) * 7 + g)
        say(f"multi-prefix: populate group {g} m={m}")
        model.populate(key, xp.cuda(), cfg["n_layers"])
        keys.append(key)
        caches.append(OT.populate(to_f64(xp), w64, cfg, cfg["n_layers"]))
    torch.cuda.synchronize()
    xs = synth.gaussian((sum(COUNTS), N_S, cfg["hidden"]), 51200)
    yield cfg, model, keys, caches, w64, xs
    model.close()


def test_multi_prefix_every_depth_matches_oracle(multi):
    cfg, model, keys, caches, w64, xs = multi
    xs_dev = xs.cuda()
    for d in range(cfg["n_layers"] + 1):
        say(f"multi-prefix step d={d}")
        out = torch.full(tuple(xs.shape), float("nan"), device="cuda")
        model.step_multi(keys, COUNTS, xs_dev, d, out=out)
        torch.cuda.synchronize()
        ref = OT.step_multi(caches, list(COUNTS), to_f64(xs), d, w64, cfg)
        assert_close(out.cpu().double().numpy(), ref, f"multi-prefix d={d}")


def test_groups_bit_identical_to_single_prefix_steps(multi):
    cfg, model, keys, caches, w64, xs = multi
    xs_dev = xs.cuda()
    for d in (0, 1, cfg["n_layers"]):
        say(f"multi-prefix vs single d={d}")
        out = model.step_multi(keys, COUNTS, xs_dev, d)
        first = 0
        for key, cnt in zip(keys, COUNTS):
            one = model.step(key, xs_dev[first:first + cnt].contiguous(), d)
            torch.cuda.synchronize()
            assert torch.equal(out[first:first + cnt], one), f"group at {first} differs (d={d})"
            first += cnt


def test_repeated_key_and_group_order(multi):
    cfg, model, keys, caches, w64, xs = multi
    xs_dev = xs.cuda()
    d = 2
    say("multi-prefix: key in two groups, reordered groups")
    out = model.step_multi(keys, COUNTS, xs_dev, d)
    # the first group split in two groups of the same key
    split = model.step_multi([keys[0], keys[0], keys[1], keys[2]], [1, 1, 1, 3], xs_dev, d)
    # groups in reverse order (requests permuted accordingly)
    order = [3, 4, 5, 2, 0, 1]
    rev = model.step_multi(keys[::-1], COUNTS[::-1], xs_dev[order].contiguous(), d)
    torch.cuda.synchronize()
    assert torch.equal(split, out)
    assert torch.equal(rev, out[order])


def test_multi_prefix_errors(multi):
    cfg, model, keys, caches, w64, xs = multi
    xs_dev = xs.cuda()
    say("multi-prefix: error paths")
    with pytest.raises(bc.BiCacheError) as e:
        model.step_multi([keys[0], 12345], [3, 3], xs_dev, 1)
    assert e.value.status == -2
    with pytest.raises(ValueError):
        model.step_multi(keys, [1, 1, 1], xs_dev, 1)
    # an entry caching only the first layer cannot serve d = 2
    xp = synth.gaussian((40, cfg["hidden"]), 51300)
    part = bc.prefix_key(np.arange(40) + 999)
    model.populate(part, xp.cuda(), 1)
    torch.cuda.synchronize()
    with pytest.raises(bc.BiCacheError) as e:
        model.step_multi([keys[0], part], [3, 3], xs_dev, 2)
    assert e.value.status == -1
    model.step_multi([keys[0], part], [3, 3], xs_dev, 1)
    torch.cuda.synchronize()
    model.invalidate(part)


def test_c3_shape_two_prefixes_bit_identical():
    cfg = synth.model_config(n_layers=12)
    sc = synth.STEP_CONFIG
    n_s, d = sc["n_s"], 8
    say("C3 shape, 12 layers: weights")
    weights = synth.model_weights(cfg, 52000, device="cuda")
    model = bc.Model(cfg, weights, cache_capacity=2)
    try:
        keys = []
        for g, m in enumerate((1536, 1024)):
            xp = synth.gaussian((m, cfg["hidden"]), 52100 + g, device="cuda")
            keys.append(bc.prefix_key(np.arange(m) + 100000 * g))
            say(f"C3 shape: populate m={m}")
            model.populate(keys[-1], xp, cfg["n_layers"])
        xs = synth.gaussian((16, n_s, cfg["hidden"]), 52200, device="cuda")
        say("C3 shape: two-prefix step")
        out = model.step_multi(keys, [8, 8], xs, d)
        a = model.step(keys[0], xs[:8].contiguous(), d)
        b = model.step(keys[1], xs[8:].contiguous(), d)
        torch.cuda.synchronize()
        assert torch.isfinite(out).all()
        assert torch.equal(out[:8], a) and torch.equal(out[8:], b)
    finally:
        model.close()
        del weights
        torch.cuda.empty_cache()
