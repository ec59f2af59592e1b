// Command-line driver of the KV-store table and the prefix-key hash, for a
// CPU test that builds it with AddressSanitizer and UndefinedBehaviorSanitizer
// and replays random operations against the Python FIFO model and the xxhash
// package.  Test infrastructure, never part of libbicache.so.
//
// Commands on stdin, one per line; one result line per command on stdout:
//   C cap            new table of capacity cap           -> "ok"
//   I key m          insert                              -> "<r> <evicted>" (r as bct_insert)
//   E key            erase                               -> "0" | "1"
//   L key            lookup                              -> m | "-1"
//   K                keys, oldest first                  -> "<n> k1 k2 ..."
//   F n              let n more allocations succeed, then fail (-1: never) -> "ok"
//   H seed hex       XXH64 of the bytes (hex, "-" = none) -> hash
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <memory>
#include <new>
#include <string>
#include <vector>

#include "cache_table.hpp"

namespace {
long g_allocs_left = -1;
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

int main() {
  std::unique_ptr<bc::CacheTable> t;
  char line[1 << 16];
  while (fgets(line, sizeof line, stdin)) {
    char op = line[0];
    if (op == 'C') {
      int cap = atoi(line + 2);
      t.reset(new bc::CacheTable(cap));
      printf("ok\n");
    } else if (op == 'I') {
      unsigned long long key;
      int m;
      sscanf(line + 2, "%llu %d", &key, &m);
      if (t->contains(key)) {
        printf("-1 0\n");
        continue;
      }
      bc::CacheEntry e;
      e.m = m;
      uint64_t ev = 0;
      int r;
      try {
        r = t->insert(key, e, &ev) ? 1 : 0;
      } catch (const std::bad_alloc&) {
        r = -2;
      }
      printf("%d %llu\n", r, (unsigned long long)ev);
    } else if (op == 'E') {
      unsigned long long key = strtoull(line + 2, nullptr, 10);
      printf("%d\n", t->erase(key) ? 1 : 0);
    } else if (op == 'L') {
      unsigned long long key = strtoull(line + 2, nullptr, 10);
      const bc::CacheEntry* e = t->find(key);
      printf("%d\n", e ? e->m : -1);
    } else if (op == 'K') {
      printf("%zu", t->order().size());
      for (uint64_t k : t->order()) printf(" %llu", (unsigned long long)k);
      printf("\n");
    } else if (op == 'F') {
      g_allocs_left = atol(line + 2);
      printf("ok\n");
    } else if (op == 'H') {
      char hex[1 << 16];
      unsigned long long seed;
      sscanf(line + 2, "%llu %s", &seed, hex);
      std::vector<unsigned char> bytes;
      if (strcmp(hex, "-") != 0)
        for (size_t i = 0; hex[i] && hex[i + 1]; i += 2) {
          char b[3] = {hex[i], hex[i + 1], 0};
          bytes.push_back((unsigned char)strtoul(b, nullptr, 16));
        }
      printf("%llu\n", (unsigned long long)bc::xxh64(bytes.data(), bytes.size(), seed));
    }
    fflush(stdout);
  }
  return 0;
}
