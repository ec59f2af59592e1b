"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle side.

This module holds no arithmetic of the method: it only draws Gaussian tensors
from seeded torch generators, scales them and rounds them to bf16
(round-to-nearest-even).  Both sides of every parity check receive the very
same bf16 tensors (the oracle widens them exactly to float64).

Seeds: tensor i of workload c is drawn from seed 1000*c + i.  Small tensors are
drawn on the CPU generator; the 32-layer weights of the full-step workload
(about 7e9 values) may be drawn on the device generator instead, because the
CPU generator needs minutes for them.  Whichever generator draws a tensor, the
oracle receives a host copy of exactly those bits.

Workloads (shapes from the paper's setting: LLaDA-8B / Dream-7B style models,
shared-prefix ratios r = m / (m + n_s) inside the 0.76-0.97 range the paper
reports for real system-prompt workloads):
  C0 tiny attention      B=2,   Hq=Hkv=4,  dh=64,  m=128,  n_s=64
  C1 LLaDA-8B attention  B=32,  Hq=Hkv=32, dh=128, m=2048, n_s=512  (r=0.80)
  C2 Dream-7B attention  B=64,  Hq=28, Hkv=4, dh=128, m=1024, n_s=384 (r=0.73)
  C3 full step           32 layers, h=4096, 32x128 heads, F=12288, B=16,
                         m=1536, n_s=512 (r=0.75), d in {0,4,8,16}
  C4 long prefix         B=128, Hq=Hkv=32, dh=128, m=8192, n_s=256 (r=0.97),
                         plus an 8-layer populate with the C3 layer shape
"""
import math
from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class AttnShape:
    B: int
    Hq: int
    Hkv: int
    m: int
    n_s: int
    dh: int


ATTN_CONFIGS = {
    0: AttnShape(B=2, Hq=4, Hkv=4, m=128, n_s=64, dh=64),
    1: AttnShape(B=32, Hq=32, Hkv=32, m=2048, n_s=512, dh=128),
    2: AttnShape(B=64, Hq=28, Hkv=4, m=1024, n_s=384, dh=128),
    4: AttnShape(B=128, Hq=32, Hkv=32, m=8192, n_s=256, dh=128),
}


def model_config(n_layers=32, hidden=4096, n_heads=32, n_kv_heads=32, head_dim=128,
                 ffn=12288, rms_eps=1e-5, rope_theta=500000.0, qkv_bias=False):
    """The C3 layer shape by default (hidden 4096, 32 x 128 heads, SwiGLU 12288)."""
    return dict(n_layers=n_layers, hidden=hidden, n_heads=n_heads, n_kv_heads=n_kv_heads,
                head_dim=head_dim, ffn=ffn, rms_eps=rms_eps, rope_theta=rope_theta,
                qkv_bias=qkv_bias)


def dream_config(n_layers=28):
    """The Dream-7B shape (its Qwen2.5-7B base: hidden 3584, 28 query and 4 KV
    heads of 128, SwiGLU 18944, Q/K/V bias, RMSNorm eps 1e-6, RoPE base 1e6)."""
    return model_config(n_layers=n_layers, hidden=3584, n_heads=28, n_kv_heads=4, head_dim=128,
                        ffn=18944, rms_eps=1e-6, rope_theta=1000000.0, qkv_bias=True)


# Full step of the Dream-7B shape over the GQA workload's sizes: 64 requests,
# shared prefix 1024, suffix 384.
DREAM_STEP = dict(B=64, m=1024, n_s=384)


STEP_CONFIG = dict(B=16, m=1536, n_s=512, depths=(0, 4, 8, 16))
POPULATE_C4 = dict(m=8192, n_layers_to_cache=8)


def _gen(seed, device):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def gaussian(shape, seed, std=1.0, mean=0.0, device="cpu"):
    """N(mean, std^2) draws in fp32 from the given seed, rounded to bf16 (RNE)."""
    x = torch.randn(*shape, generator=_gen(seed, device), device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    if mean != 0.0:
        x.add_(mean)
    return x.to(torch.bfloat16)


def attention_inputs(shape: AttnShape, seed_base: int, std=None, device="cpu"):
    """q, k_pre, v_pre, k_suf, v_suf in bf16, N(0,1) * std (default 1/sqrt(dh)).

    Layouts: q [B,Hq,n_s,dh]; k_pre, v_pre [Hkv,m,dh]; k_suf, v_suf [B,Hkv,n_s,dh].
    """
    s = shape
    std = (1.0 / math.sqrt(s.dh)) if std is None else std
    q = gaussian((s.B, s.Hq, s.n_s, s.dh), seed_base + 0, std, device=device)
    kp = gaussian((s.Hkv, s.m, s.dh), seed_base + 1, std, device=device)
    vp = gaussian((s.Hkv, s.m, s.dh), seed_base + 2, std, device=device)
    ks = gaussian((s.B, s.Hkv, s.n_s, s.dh), seed_base + 3, std, device=device)
    vs = gaussian((s.B, s.Hkv, s.n_s, s.dh), seed_base + 4, std, device=device)
    return q, kp, vp, ks, vs


def layer_weights(cfg, layer, seed_base, device="cpu"):
    """Random-init weights of one layer (bf16, [out, in] row-major).

    Q/K/V, gate and up ~ N(0, 1/fan_in); W_o and W_down ~ N(0, 1/fan_in)/sqrt(2L)
    (depth-scaled so that the fp32 residual stream stays O(1) over 32 layers);
    norm gains 1 + N(0, 0.1^2); with cfg["qkv_bias"], a Q/K/V bias ~ N(0, 0.1^2).
    """
    h, F, L = cfg["hidden"], cfg["ffn"], cfg["n_layers"]
    Hq, Hkv, dh = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    base = seed_base + 10 + 6 * layer
    depth = 1.0 / math.sqrt(2.0 * L)
    return {
        "w_qkv": gaussian(((Hq + 2 * Hkv) * dh, h), base + 0, 1.0 / math.sqrt(h), device=device),
        "w_o": gaussian((h, Hq * dh), base + 1, depth / math.sqrt(Hq * dh), device=device),
        "w_gate_up": gaussian((2 * F, h), base + 2, 1.0 / math.sqrt(h), device=device),
        "w_down": gaussian((h, F), base + 3, depth / math.sqrt(F), device=device),
        "attn_norm": gaussian((h,), base + 4, 0.1, mean=1.0, device=device),
        "ffn_norm": gaussian((h,), base + 5, 0.1, mean=1.0, device=device),
        "b_qkv": (gaussian(((Hq + 2 * Hkv) * dh,), seed_base + 10_000_000 + layer, 0.1, device=device)
                  if cfg.get("qkv_bias") else None),
    }


def model_weights(cfg, seed_base, device="cpu"):
    return [layer_weights(cfg, l, seed_base, device=device) for l in range(cfg["n_layers"])]


def step_inputs(cfg, B, m, n_s, seed_base, device="cpu"):
    """x_prefix [m, h] and x_suffix [B, n_s, h], N(0, 1) in bf16."""
    h = cfg["hidden"]
    xp = gaussian((m, h), seed_base + 0, device=device)
    xs = gaussian((B, n_s, h), seed_base + 1, device=device)
    return xp, xs


def to_f64(t):
    """Exact widening of a (bf16) torch tensor to a float64 NumPy array on the host."""
    return t.detach().to("cpu", torch.float32).double().numpy()


def weights_f64(layers):
    return [{k: (to_f64(v) if v is not None else None) for k, v in lw.items()} for lw in layers]


def denoise_inputs(cfg, T, B, n_s, n_gen, per_step, seed_base, device="cpu"):
    """Suffix inputs of T consecutive denoising steps, [T, B, n_s, h] bf16.

    A request's suffix is its own prompt rows (n_s - n_gen rows, N(0, 1)) then
    n_gen generation slots that start as one shared [MASK] embedding row; each
    step fills per_step more slots (left to right) with fresh N(0, 1) rows, as
    the tokens denoised at the previous step enter the input.
    """
    h = cfg["hidden"]
    assert 0 <= n_gen <= n_s
    x = gaussian((B, n_s, h), seed_base + 0).float()
    mask_row = gaussian((h,), seed_base + 1).float()
    x[:, n_s - n_gen:] = mask_row
    fresh = gaussian((T, B, n_gen, h), seed_base + 2).float()
    out = []
    for t in range(T):
        out.append(x.clone())
        lo = n_s - n_gen + t * per_step
        hi = min(n_s, lo + per_step)
        if lo < hi:
            x[:, lo:hi] = fresh[t, :, :hi - lo]
    return torch.stack(out).to(torch.bfloat16).to(device)


def to_device(layers, device="cuda"):
    """Copy per-layer weight dicts to the device (absent entries stay None)."""
    return [{k: (v.to(device) if v is not None else None) for k, v in lw.items()} for lw in layers]
