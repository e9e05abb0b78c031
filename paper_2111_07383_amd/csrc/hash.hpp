// The coordinate hash table of the rule book (Sec. 3.2: the hash table of active sites): 64-bit
// slots key << 32 | row, key = ((b*G0 + x)*G1 + y)*G2 + z (32 bits, ~0 reserved for empty),
// open addressing from mix32(key) with linear probing.  Shared by every kernel that reads it.
#pragma once

#include "common.hpp"

namespace ssconv {

constexpr uint64_t kEmpty = ~0ull;

// The finaliser of MurmurHash3 (Appleby): scatters neighbouring keys over the table.
__device__ __forceinline__ uint32_t mix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85ebca6bu;
  h ^= h >> 13;
  h *= 0xc2b2ae35u;
  h ^= h >> 16;
  return h;
}

__device__ __forceinline__ uint32_t site_key(int b, int x, int y, int z, int g0, int g1, int g2) {
  return (uint32_t)((((uint64_t)b * g0 + x) * g1 + y) * g2 + z);
}

// Row of the site with this key, or -1.
__device__ __forceinline__ int hash_find(const uint64_t* __restrict__ slots, uint64_t mask, uint32_t key) {
  uint64_t pos = mix32(key) & mask;
  for (uint64_t probe = 0; probe <= mask; ++probe) {
    uint64_t v = slots[pos];
    if (v == kEmpty) return -1;
    if ((uint32_t)(v >> 32) == key) return (int)(uint32_t)v;
    pos = (pos + 1) & mask;
  }
  return -1;
}

}  // namespace ssconv
