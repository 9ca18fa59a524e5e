// Streaming ceilings of the GPU for the step kernels' access shapes, measured
// by the benchmark beside the collectives: a copy (one read, one write, the
// shape of an all-gather step into leaves), a copy into two buffers (one
// read, two writes, the shape of an all-gather step into forwarding
// receivers) and a float32 add of two streams into a third (two reads, one
// write, the shape of a reduce-scatter step); and a read-only and a
// write-only stream, the two ends of that mix.  One 16-byte vector per lane, 256 lanes per
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

// Read-only and write-only streams: the two ends of the mix the step
// kernels run.  The read folds each lane's vector into a value that is
// stored only if it equals a pattern no probe input holds, so the loads stay.
__global__ __launch_bounds__(kThreads) void read_kernel(const v4u* src, v4u* sink, int64_t n, v4u never) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) {
    const v4u x = __builtin_nontemporal_load((const PAT_GLOBAL v4u*)(src + i));
    if (x.x == never.x && x.y == never.y && x.z == never.z && x.w == never.w) sink[threadIdx.x] = x;
  }
}

__global__ __launch_bounds__(kThreads) void write_kernel(v4u* dst, int64_t n, v4u value) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) __builtin_nontemporal_store(value, (PAT_GLOBAL v4u*)(dst + i));
}

// Chunk copies at a skew: chunk c (16 vectors of 16 bytes) of the chunks with
// c % 2 == parity (every chunk if parity < 0) copies src + 256 c + skew to
// dst + 256 c + skew with 16-byte vectors at skew-aligned addresses.  Written
// in two launches (even chunks, then odd ones) the lines that two chunks
// share are written partly in each, as the all-gather's steps fill a receive
// buffer chunk by chunk.
typedef v4u v4u_skewed __attribute__((aligned(4)));

__global__ __launch_bounds__(kThreads) void chunk_copy_kernel(const char* src, char* dst, int64_t chunks, int skew,
                                                              int parity) {
  const int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t per = parity < 0 ? chunks : (chunks - parity + 1) / 2;
  if (g >= per * 16) return;
  const int64_t c = parity < 0 ? g / 16 : (g / 16) * 2 + parity;
  const int64_t o = c * 256 + skew + (g % 16) * 16;
  const v4u x = *(const PAT_GLOBAL v4u_skewed*)(src + o);
  *(PAT_GLOBAL v4u_skewed*)(dst + o) = x;
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

// Reads src[0 .. bytes); `sink` (16-byte aligned, 4096 bytes) is written only
// if some 16-byte vector of src equals {1, 2, 3, 4} (words).  Same rules as
// the copy.
extern "C" int pat_ceiling_read(const void* src, void* sink, size_t bytes, hipStream_t stream) {
  if (!src || !sink || bytes % 16 || ((uintptr_t)src | (uintptr_t)sink) % 16) return (int)hipErrorInvalidValue;
  const int64_t n = (int64_t)(bytes / 16);
  if (int e = launch_check(n)) return e;
  const v4u never = {1u, 2u, 3u, 4u};
  hipLaunchKernelGGL(read_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream,
                     (const v4u*)src, (v4u*)sink, n, never);
  return (int)hipGetLastError();
}

// dst[0 .. bytes) = the word `value`, repeated; same rules as the copy.
extern "C" int pat_ceiling_write(void* dst, size_t bytes, uint32_t value, hipStream_t stream) {
  if (!dst || bytes % 16 || (uintptr_t)dst % 16) return (int)hipErrorInvalidValue;
  const int64_t n = (int64_t)(bytes / 16);
  if (int e = launch_check(n)) return e;
  const v4u v = {value, value, value, value};
  hipLaunchKernelGGL(write_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream,
                     (v4u*)dst, n, v);
  return (int)hipGetLastError();
}

// Copies `chunks` 256-byte chunks at byte offset `skew` (0, 4, 8 or 12) of
// src to the same offsets of dst, every chunk in one launch (parity < 0) or
// only the chunks of one parity (0 or 1); both buffers must hold
// 256 * chunks + 16 bytes and be 16-byte aligned.
extern "C" int pat_ceiling_chunk_copy(const void* src, void* dst, int64_t chunks, int skew, int parity,
                                      hipStream_t stream) {
  if (!src || !dst || chunks <= 0 || skew < 0 || skew > 12 || skew % 4 || parity > 1 ||
      ((uintptr_t)src | (uintptr_t)dst) % 16)
    return (int)hipErrorInvalidValue;
  const int64_t per = parity < 0 ? chunks : (chunks - parity + 1) / 2;
  if (int e = launch_check(per * 16)) return e;
  hipLaunchKernelGGL(chunk_copy_kernel, dim3((unsigned)((per * 16 + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                     stream, (const char*)src, (char*)dst, chunks, skew, parity);
  return (int)hipGetLastError();
}
