// Internal definitions shared by the host table builder and the HIP library.
#pragma once
#include <cstdint>

namespace lmbr {

constexpr int kWordBits = 21;                       // (word + 1) per packed context field
constexpr uint64_t kEmptyKey = ~0ull;               // unused hash slot
constexpr uint64_t kCtxMask = (1ull << 63) - 1;     // three 21-bit fields

// SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014).
inline uint64_t splitmix64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Pack up to three words, oldest first, newest in the low 21 bits.
uint64_t pack_context(const int32_t *words, int n_words);

}  // namespace lmbr
