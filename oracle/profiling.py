"""Shared-prefix profiling (Sec. 4.1, 4.2, 5.1): KV similarity, the shallow
depth b of one request, and the lookup table T from shared-prefix ratio r to b.

Test infrastructure: plain fp64 NumPy, imported only by the tests, the smoke
check and the benchmark's CPU baseline; it shares no code with the HIP path.

* kv_similarity (Eq. 3): cosine of the flattened cached KVs KV$_l against the
  KVs of the same prefix positions computed from the full input, KV^ref_{l,t}.
  K and V of every head and position form one vector (footnote of Sec. 4.1).
* profile_request: sim_{l,1} for every layer, from the prefix-only forward and
  the un-cached full forward of (p, z) at the first step (Sec. 5.1, Profiler).
* shallow_depth: b = the largest b in {0..L} such that sim_l >= tau for every
  1-based layer l <= b (Sec. 4.2; tau = 0.97).
* build_table / lookup_depth: T over ratio buckets r = k / n_buckets; T[k] is
  the mean of the profiled b_i of bucket k, rounded down (the mean of integers
  is fractional; rounding down is the conservative reading); a lookup at an
  arbitrary r uses the bucket at or below it that has data.
"""
import math

import numpy as np

from oracle import transformer as TR


def kv_similarity(kv_cached, kv_ref):
    """Eq. 3: cos(flatten(kv_cached), flatten(kv_ref)) in fp64."""
    a = np.asarray(kv_cached, dtype=np.float64).ravel()
    b = np.asarray(kv_ref, dtype=np.float64).ravel()
    assert a.shape == b.shape and a.size > 0
    na, nb = math.sqrt(float(a @ a)), math.sqrt(float(b @ b))
    assert na > 0 and nb > 0, "cosine of a zero vector"
    return float(a @ b) / (na * nb)


def profile_request(x_prefix, x_suffix_one, layers, cfg):
    """sim_{l,1} for l = 1..L of one request (returned 0-based, [L]).

    KV$_l from the prefix-only forward (populate); KV^ref_{l,1} = the prefix
    rows' K/V of the un-cached forward of (p, z) at the first step."""
    L = cfg["n_layers"]
    m = np.asarray(x_prefix).shape[0]
    cache = TR.populate(x_prefix, layers, cfg, L)
    rec = {}
    TR.full_forward(x_prefix, x_suffix_one, layers, cfg, record=rec)
    sims = []
    for l in range(L):
        cached = np.stack([cache["k"][l], cache["v"][l]])
        ref = np.stack([rec["k"][l][:, :m], rec["v"][l][:, :m]])
        sims.append(kv_similarity(cached, ref))
    return np.array(sims)


def shallow_depth(sims, tau):
    """Sec. 4.2: the largest b with sims[l-1] >= tau for every l in 1..b."""
    b = 0
    for s in sims:
        if s >= tau:
            b += 1
        else:
            break
    return b


def bucket_of(r, n_buckets):
    """Bucket k in 1..n_buckets of a profiled ratio r = k / n_buckets."""
    k = int(round(r * n_buckets))
    assert 1 <= k <= n_buckets and abs(k / n_buckets - r) < 1e-9, "ratio is not a bucket value"
    return k


def build_table(ratios, depths, n_buckets=100):
    """T[k] = floor(mean of the depths profiled at r = k / n_buckets), or -1
    for a bucket without requests.  Returns a list indexed 0..n_buckets
    (entry 0 unused, -1)."""
    sums = [0] * (n_buckets + 1)
    cnts = [0] * (n_buckets + 1)
    for r, b in zip(ratios, depths):
        k = bucket_of(r, n_buckets)
        sums[k] += int(b)
        cnts[k] += 1
    return [sums[k] // cnts[k] if cnts[k] else -1 for k in range(n_buckets + 1)]


def lookup_depth(table, r):
    """b for a request of shared-prefix ratio r: the entry of the largest
    bucket k <= r * n_buckets that has data (the conservative side, since b
    grows with r); 0 if there is none."""
    n_buckets = len(table) - 1
    k = min(n_buckets, int(math.floor(r * n_buckets + 1e-9)))
    while k >= 1:
        if table[k] >= 0:
            return table[k]
        k -= 1
    return 0


def shared_prefix_ratio(m, n_suffix):
    """r: shared prefix tokens over all tokens of the input string (Sec. 5.1)."""
    return m / (m + n_suffix)
