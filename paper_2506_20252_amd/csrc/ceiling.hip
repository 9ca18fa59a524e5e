// Streaming ceilings of the GPU for the step kernels' access shapes, measured
// by the benchmark beside the collectives: a copy (one read, one write, the
// shape of an all-gather step into leaves), a copy into two buffers (one
// read, two writes, the shape of an all-gather step into forwarding
// receivers) and a float32 add of two streams into a third (two reads, one
// write, the shape of a reduce-scatter step).  One 16-byte vector per lane, 256 lanes per
// workgroup, nontemporal loads and stores: the fastest form of each on
// MI355X among 1, 2, 4 and 8 vectors per lane.  Not part of the collectives.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
#define PAT_GLOBAL __attribute__((address_space(1)))

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void copy_kernel(const v4u* src, v4u* dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) {
    const v4u x = __builtin_nontemporal_load((const PAT_GLOBAL v4u*)(src + i));
    __builtin_nontemporal_store(x, (PAT_GLOBAL v4u*)(dst + i));
  }
}

__global__ __launch_bounds__(kThreads) void copy2_kernel(const v4u* src, v4u* dst, v4u* dst2, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) {
    const v4u x = __builtin_nontemporal_load((const PAT_GLOBAL v4u*)(src + i));
    __builtin_nontemporal_store(x, (PAT_GLOBAL v4u*)(dst + i));
    __builtin_nontemporal_store(x, (PAT_GLOBAL v4u*)(dst2 + i));
  }
}

__global__ __launch_bounds__(kThreads) void add_kernel(const v4f* a, const v4f* b, v4f* c, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) {
    const v4f x = __builtin_nontemporal_load((const PAT_GLOBAL v4f*)(a + i));
    const v4f y = __builtin_nontemporal_load((const PAT_GLOBAL v4f*)(b + i));
    __builtin_nontemporal_store(x + y, (PAT_GLOBAL v4f*)(c + i));
  }
}

int launch_check(int64_t n) {
  // bytes must be whole 16-byte vectors and the grid must fit one dimension
  return (n > 0 && (n + kThreads - 1) / kThreads < (int64_t(1) << 31)) ? 0 : (int)hipErrorInvalidValue;
}

}  // namespace

// dst[0 .. bytes) = src[0 .. bytes); bytes a multiple of 16, pointers 16-byte
// aligned device memory.  Returns a hipError_t value (0: launched).
extern "C" int pat_ceiling_copy(const void* src, void* dst, size_t bytes, hipStream_t stream) {
  if (!src || !dst || bytes % 16 || ((uintptr_t)src | (uintptr_t)dst) % 16) return (int)hipErrorInvalidValue;
  const int64_t n = (int64_t)(bytes / 16);
  if (int e = launch_check(n)) return e;
  hipLaunchKernelGGL(copy_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream,
                     (const v4u*)src, (v4u*)dst, n);
  return (int)hipGetLastError();
}

// dst[0 .. bytes) = dst2[0 .. bytes) = src[0 .. bytes); same rules as the copy.
extern "C" int pat_ceiling_copy2(const void* src, void* dst, void* dst2, size_t bytes, hipStream_t stream) {
  if (!src || !dst || !dst2 || bytes % 16 || ((uintptr_t)src | (uintptr_t)dst | (uintptr_t)dst2) % 16)
    return (int)hipErrorInvalidValue;
  const int64_t n = (int64_t)(bytes / 16);
  if (int e = launch_check(n)) return e;
  hipLaunchKernelGGL(copy2_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream,
                     (const v4u*)src, (v4u*)dst, (v4u*)dst2, n);
  return (int)hipGetLastError();
}

// c = a + b over float32 buffers of `bytes` each; same rules as the copy.
extern "C" int pat_ceiling_add(const void* a, const void* b, void* c, size_t bytes, hipStream_t stream) {
  if (!a || !b || !c || bytes % 16 || ((uintptr_t)a | (uintptr_t)b | (uintptr_t)c) % 16)
    return (int)hipErrorInvalidValue;
  const int64_t n = (int64_t)(bytes / 16);
  if (int e = launch_check(n)) return e;
  hipLaunchKernelGGL(add_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream,
                     (const v4f*)a, (const v4f*)b, (v4f*)c, n);
  return (int)hipGetLastError();
}
