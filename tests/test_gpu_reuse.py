"""GPU parity of deep-layer reuse within a request (second case of Eq. 5).

* The attention kernel with a per-request prefix against the fp64 oracle
  (request by request), and bit-identical to the shared-prefix kernel when
  every request's prefix is the same copy (the tile walk is the same).
* Denoising sequences of 5 steps with refresh interval 3 (refresh at steps 1
  and 4) at every reuse depth, against the oracle's sequence step by step.
* The deep store a refresh step writes: the deep layers' prefix K/V against
  the oracle's recomputed ones.
* A reuse step right after a refresh with the same suffix input reproduces
  the refresh output (bit for bit when the prefix length is a multiple of the
  64-key tile, since then both walk the same key tiles in the same order).
* The tag checks: a reuse step on a store no refresh has written, or one
  written for another batch shape or depth, is refused.
"""
import math

import numpy as np
import pytest
import torch

from oracle import transformer as OT
from oracle.attention import shared_prefix_attention as oracle_spa
import paper_2606_07571_amd as bc
from paper_2606_07571_amd import synth
from paper_2606_07571_amd.synth import AttnShape, to_f64, weights_f64
from tests.parity import assert_close, assert_close_bf16_store, say

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------ attention kernel

REQ_SHAPES = [
    AttnShape(B=1, Hq=1, Hkv=1, m=1, n_s=1, dh=64),
    AttnShape(B=3, Hq=4, Hkv=2, m=129, n_s=65, dh=128),
    AttnShape(B=2, Hq=2, Hkv=2, m=64, n_s=64, dh=128),
    AttnShape(B=5, Hq=8, Hkv=1, m=200, n_s=7, dh=64),
    AttnShape(B=3, Hq=14, Hkv=2, m=257, n_s=97, dh=128),
    AttnShape(B=4, Hq=4, Hkv=4, m=0, n_s=40, dh=64),
]


def _req_inputs(shape, seed):
    """q, per-request k_pre/v_pre [B, Hkv, m, dh], k_suf, v_suf (bf16, CPU)."""
    s = shape
    std = 1.0
    q = synth.gaussian((s.B, s.Hq, s.n_s, s.dh), seed + 0, std)
    kp = synth.gaussian((s.B, s.Hkv, s.m, s.dh), seed + 1, std)
    vp = synth.gaussian((s.B, s.Hkv, s.m, s.dh), seed + 2, std)
    ks = synth.gaussian((s.B, s.Hkv, s.n_s, s.dh), seed + 3, std)
    vs = synth.gaussian((s.B, s.Hkv, s.n_s, s.dh), seed + 4, std)
    return q, kp, vp, ks, vs


@pytest.mark.parametrize("shape", REQ_SHAPES, ids=lambda s: f"B{s.B}H{s.Hq}/{s.Hkv}m{s.m}n{s.n_s}d{s.dh}")
def test_request_prefix_attention_matches_oracle(shape):
    say(f"request-prefix attention {shape}")
    cpu = _req_inputs(shape, 90)
    dev = [t.cuda() for t in cpu]
    scale = 1.0 / math.sqrt(shape.dh)
    out = torch.full((shape.B, shape.Hq, shape.n_s, shape.dh), float("nan"), device="cuda")
    bc.request_prefix_attention(*dev, scale=scale, out=out)
    torch.cuda.synchronize()
    got = out.cpu().double().numpy()
    q, kp, vp, ks, vs = [to_f64(t) for t in cpu]
    ref = np.concatenate([oracle_spa(q[b:b + 1], kp[b], vp[b], ks[b:b + 1], vs[b:b + 1], scale)
                          for b in range(shape.B)])
    assert_close(got, ref, f"request-prefix attention {shape}")


@pytest.mark.parametrize("shape", REQ_SHAPES[1:4], ids=lambda s: f"m{s.m}n{s.n_s}")
def test_request_prefix_with_one_copy_equals_shared(shape):
    say(f"request-prefix vs shared {shape}")
    q, kp, vp, ks, vs = [t.cuda() for t in _req_inputs(shape, 95)]
    kp1 = kp[:1].expand_as(kp).contiguous()
    vp1 = vp[:1].expand_as(vp).contiguous()
    per_req = bc.request_prefix_attention(q, kp1, vp1, ks, vs)
    shared = bc.shared_prefix_attention(q, kp[0].contiguous(), vp[0].contiguous(), ks, vs)
    torch.cuda.synchronize()
    assert torch.equal(per_req, shared)


# ------------------------------------------------------------ step sequences

SMALL = [
    # GQA, dh 64, ragged m and n_s
    dict(cfg=synth.model_config(n_layers=3, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn=512),
         m=129, n_s=65, B=3, n_gen=32, seed=21),
    # MHA, dh 128, tile-aligned prefix
    dict(cfg=synth.model_config(n_layers=2, hidden=512, n_heads=4, n_kv_heads=4, head_dim=128, ffn=1024),
         m=128, n_s=37, B=2, n_gen=16, seed=22),
]
T_STEPS, DELTA, PER_STEP = 5, 3, 2


class Seq:
    def __init__(self, spec):
        self.spec = spec
        cfg = spec["cfg"]
        self.cfg = cfg
        m, B, n_s = spec["m"], spec["B"], spec["n_s"]
        self.w_cpu = synth.model_weights(cfg, 1000 * spec["seed"])
        self.w_dev = synth.to_device(self.w_cpu)
        self.xp = synth.gaussian((m, cfg["hidden"]), 1000 * spec["seed"] + 400)
        self.xsteps = synth.denoise_inputs(cfg, T_STEPS, B, n_s, spec["n_gen"], PER_STEP,
                                           1000 * spec["seed"] + 500)
        self.w64 = weights_f64(self.w_cpu)
        self.model = bc.Model(cfg, self.w_dev, cache_capacity=2)
        self.key = bc.prefix_key(np.arange(m) + spec["seed"])
        say(f"reuse: populate {cfg} m={m}")
        self.model.populate(self.key, self.xp.cuda(), cfg["n_layers"])
        torch.cuda.synchronize()
        self.cache64 = OT.populate(to_f64(self.xp), self.w64, cfg, cfg["n_layers"])


@pytest.fixture(scope="module", params=range(len(SMALL)), ids=["gqa64", "mha128"])
def seq(request):
    s = Seq(SMALL[request.param])
    yield s
    s.model.close()


def test_denoise_sequence_every_depth(seq):
    s = seq
    cfg = s.cfg
    L = cfg["n_layers"]
    xs_dev = s.xsteps.cuda()
    x64 = to_f64(s.xsteps)
    B, n_s = s.spec["B"], s.spec["n_s"]
    for d in range(L + 1):
        ref = OT.denoise_steps(s.cache64, x64, d, DELTA, s.w64, cfg)
        store = s.model.new_deep_store(s.key, B, n_s, d)
        assert (store is None) == (d == L)
        for t in range(1, T_STEPS + 1):
            mode = "refresh" if bc.is_refresh_step(t, DELTA) else "reuse"
            say(f"reuse sequence d={d} t={t} {mode}")
            out = torch.full((B, n_s, cfg["hidden"]), float("nan"), device="cuda")
            s.model.step(s.key, xs_dev[t - 1], d, out=out, deep=mode, deep_store=store)
            torch.cuda.synchronize()
            assert_close(out.cpu().double().numpy(), ref[t - 1], f"d={d} t={t} ({mode})")


def test_refresh_writes_deep_prefix_kv(seq):
    s = seq
    cfg = s.cfg
    L, Hkv, dh = cfg["n_layers"], cfg["n_kv_heads"], cfg["head_dim"]
    B, n_s, m = s.spec["B"], s.spec["n_s"], s.spec["m"]
    N = m + n_s
    d = 1
    store = s.model.new_deep_store(s.key, B, n_s, d)
    say(f"deep store contents d={d}")
    s.model.step(s.key, s.xsteps[0].cuda(), d, deep="refresh", deep_store=store)
    torch.cuda.synchronize()
    assert s.model.deep_store_offset(m, B, n_s, d, d, 0, 0, 0, 0, 0) == 0
    body = (L - d) * 2 * B * Hkv * N * dh * 2            # K/V blocks; the 256-byte header follows
    assert store.numel() == body + 256
    kv = store[:body].view(torch.bfloat16).view(L - d, 2, B, Hkv, N, dh).cpu().double().numpy()
    x64 = to_f64(s.xsteps[0])
    for b in range(B):
        rec = {}
        OT.step_one(s.cache64, x64[b], d, s.w64, cfg, record=rec)
        for l in range(d, L):
            assert_close_bf16_store(kv[l - d, 0, b, :, :m], rec["deep_k"][l], f"deep K l={l} b={b}")
            assert_close_bf16_store(kv[l - d, 1, b, :, :m], rec["deep_v"][l], f"deep V l={l} b={b}")


def test_reuse_right_after_refresh_reproduces_it(seq):
    s = seq
    cfg = s.cfg
    B, n_s, m = s.spec["B"], s.spec["n_s"], s.spec["m"]
    xs = s.xsteps[2].cuda()
    for d in range(cfg["n_layers"]):
        store = s.model.new_deep_store(s.key, B, n_s, d)
        say(f"reuse after refresh d={d}")
        ref = s.model.step(s.key, xs, d, deep="refresh", deep_store=store)
        plain = s.model.step(s.key, xs, d)
        got = s.model.step(s.key, xs, d, deep="reuse", deep_store=store)
        again = s.model.step(s.key, xs, d, deep="reuse", deep_store=store)
        torch.cuda.synchronize()
        assert torch.equal(ref, plain), "storing the deep K/V changed the refresh output"
        assert torch.equal(got, again), "a reuse step changed the store"
        if m % 64 == 0:
            assert torch.equal(got, ref)
        else:
            assert_close(got.cpu().double().numpy(), ref.cpu().double().numpy(), f"reuse==refresh d={d}")


def test_reuse_store_tag_checks(seq):
    s = seq
    cfg = s.cfg
    B, n_s, m = s.spec["B"], s.spec["n_s"], s.spec["m"]
    L = cfg["n_layers"]
    xs = s.xsteps[0].cuda()
    store = s.model.new_deep_store(s.key, B, n_s, 0)
    say("reuse tag checks")
    with pytest.raises(bc.BiCacheError) as e:
        s.model.step(s.key, xs, 0, deep="reuse", deep_store=store)
    assert e.value.status == -5
    s.model.step(s.key, xs, 0, deep="refresh", deep_store=store)
    with pytest.raises(bc.BiCacheError) as e:    # another depth (a smaller store suffices)
        s.model.step(s.key, xs, 1, deep="reuse", deep_store=store)
    assert e.value.status == -5
    with pytest.raises(bc.BiCacheError) as e:    # another batch size
        s.model.step(s.key, xs[:1].contiguous(), 0, deep="reuse", deep_store=store)
    assert e.value.status == -5
    with pytest.raises(bc.BiCacheError) as e:    # no store at all
        s.model.step(s.key, xs, 0, deep="reuse", deep_store=None)
    assert e.value.status == -1
    with pytest.raises(bc.BiCacheError) as e:    # too small
        s.model.step(s.key, xs, 0, deep="reuse", deep_store=store[:1024])
    assert e.value.status == -1
    # at d = L there are no deep layers: reuse needs no store and equals the plain step
    a = s.model.step(s.key, xs, L, deep="reuse", deep_store=None)
    b = s.model.step(s.key, xs, L)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    # the tagged store still works for its own shape, until its tag is dropped
    s.model.step(s.key, xs, 0, deep="reuse", deep_store=store)
    torch.cuda.synchronize()
    bc.lib().bc_deep_store_reset(s.model._h, store.data_ptr())
    with pytest.raises(bc.BiCacheError) as e:
        s.model.step(s.key, xs, 0, deep="reuse", deep_store=store)
    assert e.value.status == -5


def test_reuse_of_an_overwritten_store_gives_nan(seq):
    """The host tag of a store is keyed by its address; the refresh also writes
    it, with a number unique to that refresh, into the store's last 256 bytes,
    and a reuse step checks it on the device.  A store whose memory was put to
    other use (here: zeroed) without bc_deep_store_reset passes the host check,
    and the reuse step then writes NaN to every output instead of results from
    stale K/V.  A refresh restores it; a refresh into another store at the same
    parameters does not make the first store's header valid for the second."""
    s = seq
    B, n_s = s.spec["B"], s.spec["n_s"]
    xs = s.xsteps[1].cuda()
    d = 1
    store = s.model.new_deep_store(s.key, B, n_s, d)
    ref = s.model.step(s.key, xs, d, deep="refresh", deep_store=store)
    good = s.model.step(s.key, xs, d, deep="reuse", deep_store=store)
    torch.cuda.synchronize()
    assert torch.isfinite(good).all()
    say("reuse of an overwritten store")
    store.zero_()                                          # memory put to other use
    bad = s.model.step(s.key, xs, d, deep="reuse", deep_store=store)
    torch.cuda.synchronize()
    assert torch.isnan(bad).all()
    # only the header overwritten: also refused
    s.model.step(s.key, xs, d, deep="refresh", deep_store=store)
    store[-256:].fill_(7)
    bad = s.model.step(s.key, xs, d, deep="reuse", deep_store=store)
    torch.cuda.synchronize()
    assert torch.isnan(bad).all()
    # a refresh restores it, bit for bit the same reuse output as before
    s.model.step(s.key, xs, d, deep="refresh", deep_store=store)
    again = s.model.step(s.key, xs, d, deep="reuse", deep_store=store)
    torch.cuda.synchronize()
    assert torch.equal(again, good)
    # a second store refreshed with the same parameters: copying its bytes over
    # the first carries its own refresh number, which the first's tag lacks
    other = s.model.new_deep_store(s.key, B, n_s, d)
    s.model.step(s.key, xs, d, deep="refresh", deep_store=other)
    store.copy_(other)
    bad = s.model.step(s.key, xs, d, deep="reuse", deep_store=store)
    torch.cuda.synchronize()
    assert torch.isnan(bad).all()
    assert torch.isfinite(ref).all()
