"""Shared helpers of the GPU parity tests (test infrastructure)."""
import sys

import numpy as np

# Tolerance of the GPU path against the fp64 oracle, on bf16 inputs with fp32
# accumulation: every compared element within MAX_ABS, and their mean within MEAN_ABS.
MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def say(msg):
    """Progress line, flushed before a GPU step so a fault names its case."""
    print(msg, flush=True)
    sys.stdout.flush()


def assert_close(got, ref, label, max_abs=MAX_ABS, mean_abs=MEAN_ABS):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (label, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{label}: non-finite output (unwritten element?)"
    err = np.abs(got - ref)
    mx, mn = float(err.max()), float(err.mean())
    rel = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))
    say(f"  {label}: max_abs={mx:.3e} mean_abs={mn:.3e} rel_fro={rel:.3e}")
    assert mx <= max_abs and mn <= mean_abs, f"{label}: max_abs={mx:.3e} mean_abs={mn:.3e}"
    return mx, mn


# Tolerance of a bf16-STORED intermediate (the KV$ cache) against fp64.  Two
# bf16 roundings set its error: (1) the GEMM's input operand, rounded to bf16
# (relative RMS 2^-9/sqrt(3) per element), which reaches every output element
# as Gaussian noise of ~1.1e-3 x RMS(output) -- so ~6e-3 x RMS at the extreme
# of ~1e5 elements; (2) the stored value itself, off by at most half an ulp,
# i.e. 2^-9 x |value| <= 2^-9 x max|ref|.  The bound takes each term with a
# 2x margin; in norm the relative error stays near 2.5e-3 (bound 5e-3).
STORE_MAX_REL = 2.0 ** -8
STORE_RMS_REL = 1.2e-2
STORE_REL_FRO = 5e-3


def assert_close_bf16_store(got, ref, label):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (label, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{label}: non-finite value"
    err = np.abs(got - ref)
    rms = float(np.sqrt(np.mean(ref * ref)))
    bound = STORE_MAX_REL * float(np.abs(ref).max()) + STORE_RMS_REL * rms
    rel = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))
    say(f"  {label}: rel_fro={rel:.3e} max_abs={err.max():.3e} (bound {bound:.3e}, rms {rms:.3f})")
    assert rel <= STORE_REL_FRO and err.max() <= bound, f"{label}: rel_fro={rel:.3e} max_abs={err.max():.3e}"


class DeviceLayersF64:
    """The oracle's view of device-resident weights: a sequence of per-layer
    dicts of host float64 arrays, each layer copied from the device and widened
    exactly (bf16 -> fp64) the first time it is used, then kept.  Lets the
    oracle run over weights that were drawn on the device."""

    def __init__(self, device_layers):
        self._dev = device_layers
        self._host = {}

    def __len__(self):
        return len(self._dev)

    def __getitem__(self, l):
        if l < 0:
            l += len(self._dev)
        if l not in self._host:
            self._host[l] = {k: (None if v is None else
                                 v.detach().to("cpu").float().double().numpy())
                             for k, v in self._dev[l].items()}
        return self._host[l]

    def __iter__(self):
        return (self[l] for l in range(len(self)))
