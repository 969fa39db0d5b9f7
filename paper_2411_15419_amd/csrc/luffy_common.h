// Shared device/host helpers of the HIP path (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stddef.h>
#include <stdint.h>

#include "luffy.h"

namespace luffy {

// ---------------------------------------------------------------- types
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

union Pack16 {          // 16 bytes seen as 8 bf16 or raw words
  uint4 u4;
  uint16_t h[8];
  bf16x8 v;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Two floats -> two bf16 (round to nearest even) packed low/high in one
// word: a single v_cvt_pk_bf16_f32 on gfx950.
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const unsigned lane = threadIdx.x & 63u;
  return lane == 0 ? 0ull : (~0ull >> (64u - lane));
}

// Relaxed agent-scope accesses for flags other waves update in place.
__device__ __forceinline__ int load_flag(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_flag(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------- host-side helpers
void set_error(const char* fmt, ...);
int fail(int status, const char* fmt, ...);
int check_launch(const char* what);
// Compute units of the current device (cached); grid of the persistent
// kernels, which run one 512-thread block per CU.
int persistent_grid();

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Carves a caller-provided workspace into aligned sub-buffers.  With a null
// base it only measures, so size queries and the real carve share one
// layout.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <class T>
  T* take(size_t n) {
    off = align_up(off, 256);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
  size_t size() const { return align_up(off, 256); }
};

inline int elem_bytes(int dtype) { return dtype == LUFFY_BF16 ? 2 : 4; }

// Timing hook (luffy_profile_kernel): when `name` is the selected kernel,
// profile_begin returns true with two events; launch() hands them to
// hipExtLaunchKernel, which records them with the kernel's own dispatch (its
// start and its end) rather than as separate stream commands, so the
// measured interval is the kernel alone.  profile_end queues the pair for
// luffy_profile_read.
bool profile_begin(const char* name, hipEvent_t* start, hipEvent_t* stop);
void profile_end(hipEvent_t start, hipEvent_t stop);

// kernel<<<grid, block, shmem, s>>>(args...), timed when selected.
template <typename... KArgs, typename... Args>
inline void launch(const char* name, void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t shmem, hipStream_t s,
                   Args... args) {
  hipEvent_t start = nullptr, stop = nullptr;
  if (profile_begin(name, &start, &stop)) {
    hipExtLaunchKernelGGL(kernel, grid, block, static_cast<uint32_t>(shmem), s, start, stop, 0,
                          static_cast<KArgs>(args)...);
    profile_end(start, stop);
  } else {
    kernel<<<grid, block, shmem, s>>>(static_cast<KArgs>(args)...);
  }
}

constexpr int kMaxExperts = 64;

}  // namespace luffy
