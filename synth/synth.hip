// Seeded synthetic inputs, filled on the device.
//
// Holds none of the collective's arithmetic: it only turns (seed, counter)
// into values.  The Python twin in synth/__init__.py computes the very same
// values on the host, so a checker can regenerate any element without reading
// device memory.
//
// Generator: SplitMix64 (G. Steele, D. Lea, C. Flood, "Fast splittable
// pseudorandom number generators", OOPSLA 2014).  Value n of the stream
// seeded with s is mix(s + (n + 1) * 0x9E3779B97F4A7C15), mix being the
// published 64-bit finaliser.  Element i of a buffer uses n = base + i.
//
// Kinds:
//   0  int32  lo + floor(((h >> 32) * span) / 2^32)   (span <= 2^32, Lemire's
//      multiply-shift range reduction)
//   1  fp32   ((h >> 40) - 2^23) * 2^-23, i.e. uniform on [-1, 1) in steps of
//      2^-23 (exact in fp32)
//   2  16-bit table[h >> 48]  (a 65536-entry table supplied by the caller)
//   3  32-bit table[h >> 48]

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

__device__ __forceinline__ uint64_t splitmix64_at(uint64_t seed, uint64_t n) {
  uint64_t z = seed + (n + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ void fill_kernel(void* dst, uint64_t n, uint64_t seed, uint64_t base, int kind,
                            int64_t lo, uint64_t span, const void* table) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint64_t h = splitmix64_at(seed, base + i);
    switch (kind) {
      case 0: {
        const uint64_t off = ((h >> 32) * span) >> 32;
        ((int32_t*)dst)[i] = (int32_t)(lo + (int64_t)off);
        break;
      }
      case 1: {
        const int32_t k = (int32_t)(h >> 40) - (1 << 23);
        ((float*)dst)[i] = (float)k * 0x1.0p-23f;
        break;
      }
      case 2:
        ((uint16_t*)dst)[i] = ((const uint16_t*)table)[h >> 48];
        break;
      default:
        ((uint32_t*)dst)[i] = ((const uint32_t*)table)[h >> 48];
        break;
    }
  }
}

}  // namespace

// Fill n elements at dst.  Returns 0 on success, the hipError_t otherwise.
extern "C" int synth_fill(void* dst, uint64_t n, uint64_t seed, uint64_t base, int kind,
                          int64_t lo, uint64_t span, const void* table_dev, hipStream_t stream) {
  if (n == 0) return 0;
  if (kind < 0 || kind > 3 || dst == nullptr) return (int)hipErrorInvalidValue;
  if ((kind >= 2) && table_dev == nullptr) return (int)hipErrorInvalidValue;
  const int threads = 256;
  uint64_t blocks = (n + threads - 1) / threads;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(threads), 0, stream, dst, n, seed,
                     base, kind, lo, span, table_dev);
  return (int)hipGetLastError();
}
