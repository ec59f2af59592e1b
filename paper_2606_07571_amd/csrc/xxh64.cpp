// 64-bit xxHash (XXH64), the prefix-key hash of Appendix C: the published
// algorithm with four lane accumulators over 32-byte stripes, an 8/4/1-byte
// tail and a final avalanche.  Portable (byte-wise little-endian reads).
#include <string.h>

#include "cache_table.hpp"

namespace bc {
namespace {

constexpr uint64_t P1 = 0x9E3779B185EBCA87ull;
constexpr uint64_t P2 = 0xC2B2AE3D27D4EB4Full;
constexpr uint64_t P3 = 0x165667B19E3779F9ull;
constexpr uint64_t P4 = 0x85EBCA77C2B2AE63ull;
constexpr uint64_t P5 = 0x27D4EB2F165667C5ull;

inline uint64_t rotl(uint64_t x, int r) { return (x << r) | (x >> (64 - r)); }

inline uint64_t le64(const unsigned char* p) {
  uint64_t v = 0;
  for (int i = 7; i >= 0; --i) v = (v << 8) | p[i];
  return v;
}
inline uint32_t le32(const unsigned char* p) {
  return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}

inline uint64_t round1(uint64_t acc, uint64_t lane) {
  acc += lane * P2;
  acc = rotl(acc, 31);
  return acc * P1;
}
inline uint64_t merge(uint64_t acc, uint64_t v) {
  acc ^= round1(0, v);
  return acc * P1 + P4;
}

}  // namespace

uint64_t xxh64(const void* data, size_t len, uint64_t seed) {
  const unsigned char* p = static_cast<const unsigned char*>(data);
  const unsigned char* end = p + len;
  uint64_t acc;
  if (len >= 32) {
    uint64_t v1 = seed + P1 + P2, v2 = seed + P2, v3 = seed, v4 = seed - P1;
    while (p + 32 <= end) {
      v1 = round1(v1, le64(p));
      v2 = round1(v2, le64(p + 8));
      v3 = round1(v3, le64(p + 16));
      v4 = round1(v4, le64(p + 24));
      p += 32;
    }
    acc = rotl(v1, 1) + rotl(v2, 7) + rotl(v3, 12) + rotl(v4, 18);
    acc = merge(acc, v1);
    acc = merge(acc, v2);
    acc = merge(acc, v3);
    acc = merge(acc, v4);
  } else {
    acc = seed + P5;
  }
  acc += (uint64_t)len;
  while (p + 8 <= end) {
    acc ^= round1(0, le64(p));
    acc = rotl(acc, 27) * P1 + P4;
    p += 8;
  }
  if (p + 4 <= end) {
    acc ^= (uint64_t)le32(p) * P1;
    acc = rotl(acc, 23) * P2 + P3;
    p += 4;
  }
  while (p < end) {
    acc ^= (uint64_t)(*p) * P5;
    acc = rotl(acc, 11) * P1;
    ++p;
  }
  acc ^= acc >> 33;
  acc *= P2;
  acc ^= acc >> 29;
  acc *= P3;
  acc ^= acc >> 32;
  return acc;
}

}  // namespace bc
