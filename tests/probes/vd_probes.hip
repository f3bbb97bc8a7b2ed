// Probes of gfx950 instruction behaviour that the attention kernels' bitwise
// guarantees rest on (test infrastructure, not part of libvdattn): each entry
// point runs one instruction over caller-supplied device arrays and writes
// the raw results, which tests/test_gpu_hw_facts.py compares on the host.
//
//   vdp_mfma_bf16: D = v_mfma_f32_16x16x32_bf16(A, B, C) per 16 x 16 tile,
//                  A [tiles][16][32] bf16, B [tiles][32][16] bf16,
//                  C, D [tiles][16][16] fp32 (row-major, device memory).
//   vdp_exp2:      y[i] = v_exp_f32(x[i]).
//   vdp_cvt_bf16:  y[i] = v_cvt_pk_bf16_f32(x[i]) (bf16 bits).
//   vdp_row_swap:  one wavefront: v_permlane16_swap_b32 and
//                  v_permlane32_swap_b32 on the registers (a[l], b[l]),
//                  written as out[0..63] / out[64..127] (first and second
//                  register after the 16-lane swap) and out[128..191] /
//                  out[192..255] (after the 32-lane swap); a, b [64] fp32.
//   vdp_claims:    wgs one-wavefront workgroups (spread over every die), each
//                  taking per values from one counter with atomicAdd(c, 1)
//                  from lane 0 (the split launch's slot claims); out [wgs *
//                  per] int32 gets them in claim order, counter [1] int32 is
//                  zeroed by a fill launch first.
//
// Every entry point returns 0, or -1 for a bad size or pointer (nothing is
// launched then), or -2 if the launch failed.  One wavefront per tile or per
// 64 elements; every access stays inside the arrays the sizes describe.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

// Operand layout of the instruction (the one the attention kernels use):
// lane l holds A[l % 16][8 (l / 16) + e] and B[8 (l / 16) + e][l % 16] for
// e = 0..7, and D[4 (l / 16) + i][l % 16] for i = 0..3.
__global__ __launch_bounds__(64) void mfma_tile_kernel(const uint16_t* a, const uint16_t* b,
                                                       const float* c, float* d, int tiles) {
  const int t = blockIdx.x;
  if (t >= tiles) return;
  const int l = threadIdx.x, r = l % 16, g = l / 16;
  const uint16_t* at = a + (int64_t)t * 16 * 32;
  const uint16_t* bt = b + (int64_t)t * 32 * 16;
  const float* ct = c + (int64_t)t * 256;
  float* dt = d + (int64_t)t * 256;
  u16x8 av, bv;
  for (int e = 0; e < 8; ++e) {
    av[e] = at[r * 32 + 8 * g + e];
    bv[e] = bt[(8 * g + e) * 16 + r];
  }
  f32x4 acc;
  for (int i = 0; i < 4; ++i) acc[i] = ct[(4 * g + i) * 16 + r];
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av),
                                                __builtin_bit_cast(bf16x8, bv), acc, 0, 0, 0);
  for (int i = 0; i < 4; ++i) dt[(4 * g + i) * 16 + r] = acc[i];
}

__global__ __launch_bounds__(64) void exp2_kernel(const float* x, float* y, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (i < n) y[i] = __builtin_amdgcn_exp2f(x[i]);
}

__global__ __launch_bounds__(64) void cvt_bf16_kernel(const float* x, uint16_t* y, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (i < n) y[i] = __builtin_bit_cast(uint16_t, (__bf16)x[i]);
}

// The attention kernels' row exchanges, with the same two wait states before
// each swap.
__global__ __launch_bounds__(64) void row_swap_kernel(const float* a, const float* b, float* out) {
  const int l = threadIdx.x;
  float a16 = a[l], b16 = b[l], a32 = a[l], b32 = b[l];
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a16), "+v"(b16));
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a32), "+v"(b32));
  out[l] = a16;
  out[64 + l] = b16;
  out[128 + l] = a32;
  out[192 + l] = b32;
}

__global__ __launch_bounds__(64) void zero_kernel(int32_t* c) {
  if (threadIdx.x == 0) *c = 0;
}

__global__ __launch_bounds__(64) void claims_kernel(int32_t* c, int32_t* out, int per) {
  for (int i = 0; i < per; ++i) {
    int v = 0;
    if (threadIdx.x == 0) v = atomicAdd(c, 1);
    v = __builtin_amdgcn_readfirstlane(v);
    if (threadIdx.x == 0) out[(int64_t)blockIdx.x * per + i] = v;
  }
}

int launched() { return hipGetLastError() == hipSuccess ? 0 : -2; }

}  // namespace

extern "C" {

int vdp_mfma_bf16(const void* a, const void* b, const void* c, void* d, int tiles,
                  hipStream_t stream) {
  if (tiles < 0 || (tiles > 0 && (!a || !b || !c || !d))) return -1;
  if (tiles == 0) return 0;
  hipLaunchKernelGGL(mfma_tile_kernel, dim3((unsigned)tiles), dim3(64), 0, stream,
                     static_cast<const uint16_t*>(a), static_cast<const uint16_t*>(b),
                     static_cast<const float*>(c), static_cast<float*>(d), tiles);
  return launched();
}

int vdp_exp2(const void* x, void* y, int64_t n, hipStream_t stream) {
  if (n < 0 || (n > 0 && (!x || !y)) || n > ((int64_t)1 << 36)) return -1;
  if (n == 0) return 0;
  hipLaunchKernelGGL(exp2_kernel, dim3((unsigned)((n + 63) / 64)), dim3(64), 0, stream,
                     static_cast<const float*>(x), static_cast<float*>(y), n);
  return launched();
}

int vdp_cvt_bf16(const void* x, void* y, int64_t n, hipStream_t stream) {
  if (n < 0 || (n > 0 && (!x || !y)) || n > ((int64_t)1 << 36)) return -1;
  if (n == 0) return 0;
  hipLaunchKernelGGL(cvt_bf16_kernel, dim3((unsigned)((n + 63) / 64)), dim3(64), 0, stream,
                     static_cast<const float*>(x), static_cast<uint16_t*>(y), n);
  return launched();
}

int vdp_row_swap(const void* a, const void* b, void* out, hipStream_t stream) {
  if (!a || !b || !out) return -1;
  hipLaunchKernelGGL(row_swap_kernel, dim3(1), dim3(64), 0, stream, static_cast<const float*>(a),
                     static_cast<const float*>(b), static_cast<float*>(out));
  return launched();
}

int vdp_claims(void* counter, void* out, int wgs, int per, hipStream_t stream) {
  if (!counter || !out || wgs < 1 || wgs > (1 << 20) || per < 1 || per > 64) return -1;
  hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(64), 0, stream, static_cast<int32_t*>(counter));
  hipLaunchKernelGGL(claims_kernel, dim3((unsigned)wgs), dim3(64), 0, stream,
                     static_cast<int32_t*>(counter), static_cast<int32_t*>(out), per);
  return launched();
}

}  // extern "C"
