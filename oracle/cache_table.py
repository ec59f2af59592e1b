"""Oracle: a Python model of the KV store H with FIFO eviction (Appendix C).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

H maps a prefix key to its cached KVs.  A lookup is a dictionary access.  On a
miss the caller computes the prefix KVs and inserts them; when the store is
full the entry inserted earliest is evicted first (first in, first out).
Re-inserting a key that is present is refused (the caller invalidates first),
and invalidation removes the entry from both the map and the FIFO order.
"""
from collections import OrderedDict


class FifoTable:
    def __init__(self, capacity):
        assert capacity >= 1
        self.capacity = capacity
        self.entries = OrderedDict()        # key -> metadata, in insertion order

    def lookup(self, key):
        return self.entries.get(key)

    def insert(self, key, meta):
        """Returns the evicted key, or None.  Raises KeyError on a duplicate."""
        if key in self.entries:
            raise KeyError("duplicate key")
        evicted = None
        if len(self.entries) >= self.capacity:
            evicted, _ = self.entries.popitem(last=False)
        self.entries[key] = meta
        return evicted

    def invalidate(self, key):
        """Returns True if the key was present."""
        return self.entries.pop(key, None) is not None

    def order(self):
        return list(self.entries.keys())
