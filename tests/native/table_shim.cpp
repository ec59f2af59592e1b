// Host-only C shim over the runtime's KV-store table and prefix-key hash, so
// the CPU tests can drive the FIFO bookkeeping without a GPU.  Test
// infrastructure: built next to the tests, never linked into libbicache.so.
//
// The shim replaces the global operator new of its own code (it is linked
// with -Bsymbolic) with one that can be told to fail: bct_fail_allocs_after(n)
// lets n more allocations succeed and then throws std::bad_alloc, so the
// tests can check that a failed host allocation leaves the table unchanged.
#include <stdint.h>
#include <stdlib.h>

#include <new>

#include "cache_table.hpp"

namespace {
long g_allocs_left = -1;  // < 0: never fail
}

void* operator new(size_t n) {
  if (g_allocs_left == 0) throw std::bad_alloc();
  if (g_allocs_left > 0) --g_allocs_left;
  void* p = malloc(n ? n : 1);
  if (!p) throw std::bad_alloc();
  return p;
}
void operator delete(void* p) noexcept { free(p); }
void operator delete(void* p, size_t) noexcept { free(p); }

extern "C" {

void bct_fail_allocs_after(long n) { g_allocs_left = n; }

void* bct_create(int capacity) { return new bc::CacheTable(capacity); }
void bct_destroy(void* t) { delete static_cast<bc::CacheTable*>(t); }

// 0 = inserted, 1 = inserted after evicting *evicted, -1 = key already
// present, -2 = a host allocation failed (table unchanged)
int bct_insert(void* t, uint64_t key, int m, uint64_t* evicted) {
  auto* tb = static_cast<bc::CacheTable*>(t);
  if (tb->contains(key)) return -1;
  bc::CacheEntry e;
  e.m = m;
  try {
    return tb->insert(key, e, evicted) ? 1 : 0;
  } catch (const std::bad_alloc&) {
    return -2;
  }
}

int bct_erase(void* t, uint64_t key) { return static_cast<bc::CacheTable*>(t)->erase(key) ? 1 : 0; }

int bct_lookup(void* t, uint64_t key) {
  const bc::CacheEntry* e = static_cast<bc::CacheTable*>(t)->find(key);
  return e ? e->m : -1;
}

int bct_keys(void* t, uint64_t* out, int max) {
  int i = 0;
  for (uint64_t k : static_cast<bc::CacheTable*>(t)->order()) {
    if (i < max) out[i] = k;
    ++i;
  }
  return i;
}

uint64_t bct_xxh64(const void* data, uint64_t len, uint64_t seed) { return bc::xxh64(data, len, seed); }
}
