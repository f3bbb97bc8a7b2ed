// vd_hw.hpp -- gfx950 helpers shared by the library's kernels: wave-uniform
// values, vector-memory wait counts, direct global-to-LDS copies, unpaired
// LDS reads, an LDS-only workgroup barrier, and the host's per-device LDS
// limit and chip geometry.  No arithmetic of any result lives here.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace vd {

__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Direct global-to-LDS copy of 16 bytes per lane: lane l's bytes land at LDS
// byte address m0val + 16 l.  Issued as inline assembly so that the compiler
// does not make every later LDS read wait for all such copies; the kernel
// waits for them itself with wait_vmcnt.  M0 is saved and restored.
__device__ __forceinline__ void lds_dma16(const void* src, uint32_t m0val) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(m0val)
      : "memory");
}

// N direct global-to-LDS copies of 1 KB (N = 2 or 4) with one M0 setting:
// copy i moves lane l's 16 bytes from src + 1024 i to LDS byte address
// m0val + 1024 i + 16 l (the instruction's immediate offset moves both the
// global and the LDS address).  M0 is saved and restored, as in lds_dma16.
template <int N>
__device__ __forceinline__ void lds_dma16_run(const void* src, uint32_t m0val) {
  static_assert(N == 2 || N == 4, "copies per M0 setting");
  uint32_t saved;
  if constexpr (N == 4)
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off\n\t"
        "global_load_lds_dwordx4 %1, off offset:1024\n\t"
        "global_load_lds_dwordx4 %1, off offset:2048\n\t"
        "global_load_lds_dwordx4 %1, off offset:3072\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(src), "s"(m0val)
        : "memory");
  else
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off\n\t"
        "global_load_lds_dwordx4 %1, off offset:1024\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(src), "s"(m0val)
        : "memory");
}

// 8-byte LDS read issued as its own ds_read_b64.  Volatile, so that the
// compiler does not pair it with a neighbour at another offset into one
// two-address read: the two halves of a matrix operand come from two page
// blocks, and a paired read would land them in the wrong registers and cost
// register copies.
template <class T8>
__device__ __forceinline__ T8 lds_read8(const void* p) {
  static_assert(sizeof(T8) == 8, "8-byte value");
  return *(const volatile __attribute__((address_space(3))) T8*)(uintptr_t)p;
}

// Workgroup barrier that orders LDS accesses only (global memory operations
// in flight are not waited for).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Host: raises a kernel's dynamic LDS limit to `bytes` on the current device,
// once per (call site, device).  The attribute belongs to the device, and a
// process may drive several GPUs; `done` is the call site's own flag array.
// Two threads may both set it the first time, which is harmless.
constexpr int kMaxDevices = 64;
inline hipError_t set_lds_limit(const void* fn, int bytes,
                                std::atomic<unsigned char> (&done)[kMaxDevices]) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const bool tracked = dev >= 0 && dev < kMaxDevices;
  if (tracked && done[dev].load(std::memory_order_acquire)) return hipSuccess;
  e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess && tracked) done[dev].store(1, std::memory_order_release);
  return e;
}

// Host: the current device's geometry, read once per device.  cus: compute
// units; xcds: the accelerator dies the dispatcher spreads workgroups over,
// workgroup b landing on die b mod xcds (a power of two: the 32-CU dies of
// gfx950, 8 on a whole MI355X, fewer when the GPU is partitioned).  Only
// launch shapes and the order in which workgroups take work items depend on
// it, never a value.
struct Geometry {
  int cus, xcds, xcd_shift;
};

inline Geometry device_geometry() {
  static std::atomic<int> cache[kMaxDevices];  // cus + 1, 0: not read yet
  constexpr int kCusPerXcd = 32;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = -1;
  const bool tracked = dev >= 0 && dev < kMaxDevices;
  if (tracked) cus = cache[dev].load(std::memory_order_acquire) - 1;
  if (cus <= 0) {
    if (dev < 0 || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                       hipSuccess || cus <= 0)
      cus = 256;
    if (tracked) cache[dev].store(cus + 1, std::memory_order_release);
  }
  Geometry g;
  g.cus = cus;
  g.xcd_shift = 0;
  while (g.xcd_shift < 3 && (kCusPerXcd << (g.xcd_shift + 1)) <= cus) ++g.xcd_shift;
  g.xcds = 1 << g.xcd_shift;
  return g;
}

}  // namespace vd
