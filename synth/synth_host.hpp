// Seeded synthetic inputs on the host: the C++ twin of synth.hip and of the
// numpy functions in synth/__init__.py.
//
// Holds none of the collectives' arithmetic: it only turns (seed, counter)
// into values, exactly as the device fill does, so that a CPU checker can
// regenerate any element of a buffer the device filled without reading it.
//
// Generator: SplitMix64 (G. Steele, D. Lea, C. Flood, "Fast splittable
// pseudorandom number generators", OOPSLA 2014).  Value n of the stream seeded
// with s is mix(s + (n + 1) * golden gamma), mix being the published 64-bit
// finaliser.  Element i of rank x's buffer uses counter (x << 36) + i.
//
// Kinds (the same numbering as synth.hip):
//   0  int32  lo + floor(((h >> 32) * span) / 2^32)   (Lemire's multiply-shift)
//   1  fp32   ((h >> 40) - 2^23) * 2^-23               (uniform on [-1, 1))
//   2  16-bit table[h >> 48]   (65536 entries supplied by the caller)
//   3  32-bit table[h >> 48]
#pragma once

#include <cstdint>
#include <cstring>

namespace synth_host {

constexpr int kRankShift = 36;

inline uint64_t splitmix64_at(uint64_t seed, uint64_t n) {
  uint64_t z = seed + (n + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

struct Source {
  int kind = 0;
  uint64_t seed = 0;
  int64_t lo = 0;
  uint64_t span = 0;
  const void* table = nullptr;  // kinds 2 and 3

  // Raw bits of elements [i0, i0 + n) of rank x's buffer (int32, float32 or
  // bf16 bits, the latter in the low half), one kind per call.
  void row(int64_t x, int64_t i0, int64_t n, uint32_t* out) const {
    const uint64_t base = (uint64_t(x) << kRankShift) + uint64_t(i0);
    switch (kind) {
      case 0:
        for (int64_t i = 0; i < n; ++i) {
          const uint64_t h = splitmix64_at(seed, base + uint64_t(i));
          out[i] = uint32_t(int32_t(lo + int64_t(((h >> 32) * span) >> 32)));
        }
        break;
      case 1:
        for (int64_t i = 0; i < n; ++i) {
          const uint64_t h = splitmix64_at(seed, base + uint64_t(i));
          const float f = float(int32_t(h >> 40) - (1 << 23)) * 0x1.0p-23f;
          std::memcpy(&out[i], &f, 4);
        }
        break;
      case 2: {
        const uint16_t* t = static_cast<const uint16_t*>(table);
        for (int64_t i = 0; i < n; ++i) out[i] = t[splitmix64_at(seed, base + uint64_t(i)) >> 48];
        break;
      }
      default: {
        const uint32_t* t = static_cast<const uint32_t*>(table);
        for (int64_t i = 0; i < n; ++i) out[i] = t[splitmix64_at(seed, base + uint64_t(i)) >> 48];
        break;
      }
    }
  }

  // Raw bits of element i of rank x's buffer (int32, float32 or bf16 bits).
  uint32_t bits(int64_t x, int64_t i) const {
    const uint64_t h = splitmix64_at(seed, (uint64_t(x) << kRankShift) + uint64_t(i));
    switch (kind) {
      case 0: {
        const uint64_t off = ((h >> 32) * span) >> 32;
        return uint32_t(int32_t(lo + int64_t(off)));
      }
      case 1: {
        const float f = float(int32_t(h >> 40) - (1 << 23)) * 0x1.0p-23f;
        uint32_t u;
        std::memcpy(&u, &f, 4);
        return u;
      }
      case 2: return static_cast<const uint16_t*>(table)[h >> 48];
      default: return static_cast<const uint32_t*>(table)[h >> 48];
    }
  }
};

}  // namespace synth_host
