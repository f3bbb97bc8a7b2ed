// vd_linear.hip -- the batch-invariant linear layer of libvdattn.so (gfx950).
//
// c[m][n] = bf16_RNE( sum_k a[m][k] * b[n][k] ): the matmul contract of the
// paper's Section 5.4 (Fig. 3): the output row of a token depends only on that
// token's input row and on the weights, however many rows the call holds and
// wherever the row sits among them.
//
// Canonical arithmetic (one chain per output element, fixed by K alone):
//   acc = +0 (fp32); for k0 = 0, 32, 64, ... < K (ascending):
//     acc = v_mfma_f32_16x16x32_bf16(a[m][k0 .. k0+31], b[n][k0 .. k0+31], acc)
//   c[m][n] = bf16 round-to-nearest-even of acc.
// The result of one MFMA output cell depends only on its own row of the A
// operand, its own column of the B operand and its accumulator cell (the
// property vd_cas.hpp relies on), so neither the tiling, nor the workgroup that
// computes a row, nor the other rows of the call reach its bits; only K (the
// chain length and order) does, and there is no split over K.
//
// Launch: one workgroup of 8 wavefronts (4 x 2) per 256 x 192 output tile,
// each wavefront a 64 x 96 part (4 x 6 MFMA blocks of 16 x 16).  K advances
// in steps of 64 through a 2-stage LDS ring of A and B tiles (256 and 192
// rows x 64 values; 112 KB, one workgroup and two wavefronts per SIMD on a
// CU) filled by direct global-to-LDS copies, with one barrier per step; the 16-byte chunks of each
// 128-byte LDS row are XOR-swizzled by the row so that the 16 rows one operand
// read touches fall in different banks.  Tiles are taken in groups of 4 row
// tiles sweeping the column tiles, and each XCD (workgroup id mod the die
// count, 8 on a whole MI355X) takes a contiguous range of that order, so the A
// and B panels of its workgroups are shared in its L2.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/vdattn.h"
#include "vd_cas.hpp"
#include "vd_hw.hpp"

using namespace vd;

namespace {

// Tile configuration: kWM x kWN wavefronts, each computing kXB x kYB MFMA
// blocks of 16 x 16; K advances kBK per step (kBK / 32 MFMA chunks).  On the
// Llama-3-8B QKV shape, 4 x 2 wavefronts of 4 x 6 blocks (a 256 x 192 tile,
// one workgroup per CU) ran 9% faster than 2 x 2 wavefronts of 4 x 4 blocks
// (128 x 128, two workgroups per CU), which beat 4 x 8 or 8 x 4 blocks per
// wavefront at 4 wavefronts, 2 x 4 / 4 x 2 wavefronts of 4 x 4, 4 x 8 or
// 8 x 4 blocks, and 192 x 256 tiles.
constexpr int kWM = 4, kWN = 2;
constexpr int kXB = 4, kYB = 6, kBK = 64;
constexpr int kWaves = kWM * kWN;
constexpr int kThreads = 64 * kWaves;
constexpr int kBM = kWM * 16 * kXB;         // rows of a (tokens) per workgroup tile
constexpr int kBN = kWN * 16 * kYB;         // rows of b (output features) per workgroup tile
constexpr int kRowBytes = kBK * 2;          // one staged row of a tile
constexpr int kChunks = kRowBytes / 16;     // 16-byte chunks per staged row
constexpr int kRowsPerCopy = 1024 / kRowBytes;
constexpr int kGroupM = 4;                  // row tiles per group of the tile order
constexpr int kTileA = kBM * kRowBytes, kTileB = kBN * kRowBytes;
constexpr int kStageBytes = kTileA + kTileB;
constexpr int kLinLds = 2 * kStageBytes;    // 2-stage ring
constexpr int kCopiesA = kTileA / 1024 / kWaves, kCopiesB = kTileB / 1024 / kWaves;  // per wavefront
static_assert(kChunks == 4 || kChunks == 8, "staged rows of 64 or 128 bytes");
static_assert(kCopiesA * 1024 * kWaves == kTileA && kCopiesB * 1024 * kWaves == kTileB,
              "copy split");

// Swizzle key of staged row r: chunk ch of the row sits in 16-byte slot
// ch ^ key(r), so that 8 consecutive rows read at one chunk fill 8 distinct
// 16-byte slots of a 128-byte bank window.
__device__ __forceinline__ int swz_key(int r) {
  return kChunks == 8 ? (r & 7) : ((r >> 1) & 3);
}
__device__ __forceinline__ int swz(int r, int ch) {
  return r * kRowBytes + ((ch ^ swz_key(r)) << 4);
}

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void linear_kernel(
    const uint16_t* a, int64_t lda, const uint16_t* b, int64_t ldb, uint16_t* c, int64_t ldc,
    int64_t M, int N, int K, int tiles_m, int tiles_n, int xcd_shift) {
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  const int wave = uni(threadIdx.x >> 6);
  const int lane = __lane_id();
  // tile order: groups of kGroupM row tiles, each sweeping the column tiles
  // (row tile fastest); XCD x takes the x-th contiguous share of the order
  const int64_t total = (int64_t)tiles_m * tiles_n;
  const int xcds = 1 << xcd_shift;
  const int64_t per_xcd = (total + xcds - 1) >> xcd_shift;
  const int64_t jx = blockIdx.x >> xcd_shift;
  if (jx >= per_xcd) return;
  const int64_t i = (int64_t)(blockIdx.x & (xcds - 1)) * per_xcd + jx;
  if (i >= total) return;
  const int64_t group = i / ((int64_t)kGroupM * tiles_n);
  const int64_t first_m = group * kGroupM;
  const int size_m = (int)((tiles_m - first_m) < kGroupM ? (tiles_m - first_m) : kGroupM);
  const int in_group = (int)(i - group * (int64_t)kGroupM * tiles_n);
  const int64_t m0 = (first_m + in_group % size_m) * kBM;
  const int n0 = (in_group / size_m) * kBN;

  // Copies: the staged A tile is kCopiesA * kWaves copies of 1 KB (kRowsPerCopy
  // rows each), wavefront w taking copies w * kCopiesA + j; the same for B.
  // Lane l of a copy carries row l / kChunks of it and 16-byte slot
  // l % kChunks, i.e. source chunk slot ^ key(row) (the copy's first row is a
  // multiple of kRowsPerCopy, so the key depends on the lane alone).  Rows
  // past M (or N) repeat the last row: in bounds, and never stored.
  const int lrow = lane / kChunks;
  const int cch = (lane % kChunks) ^ swz_key(lrow);
  const uint16_t* asrc[kCopiesA];
  const uint16_t* bsrc[kCopiesB];
#pragma unroll
  for (int j = 0; j < kCopiesA; ++j) {
    const int r = (wave * kCopiesA + j) * kRowsPerCopy + lrow;
    const int64_t ra = m0 + r < M ? m0 + r : M - 1;
    asrc[j] = a + ra * lda + 8 * cch;
  }
#pragma unroll
  for (int j = 0; j < kCopiesB; ++j) {
    const int r = (wave * kCopiesB + j) * kRowsPerCopy + lrow;
    const int rb = n0 + r < N ? n0 + r : N - 1;
    bsrc[j] = b + (int64_t)rb * ldb + 8 * cch;
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
  auto fetch = [&](int step, int buf) {
    const int k0 = step * kBK;
    const uint32_t st = lds0 + buf * kStageBytes;
#pragma unroll
    for (int j = 0; j < kCopiesA; ++j)
      lds_dma16(asrc[j] + k0, uni((int)(st + 1024 * (wave * kCopiesA + j))));
#pragma unroll
    for (int j = 0; j < kCopiesB; ++j)
      lds_dma16(bsrc[j] + k0, uni((int)(st + kTileA + 1024 * (wave * kCopiesB + j))));
  };

  // this wavefront's part: rows wm .. wm + 16 kXB - 1, columns wn .. wn + 16 kYB - 1
  const int wm = 16 * kXB * (wave / kWN), wn = 16 * kYB * (wave % kWN);
  const int col = lane & 15, grp = lane >> 4;
  f32x4 acc[kXB][kYB];
#pragma unroll
  for (int x = 0; x < kXB; ++x)
#pragma unroll
    for (int y = 0; y < kYB; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One barrier per step: after it, step t's copies are visible to every
  // wavefront and every wavefront is done with step t - 1, whose stage the
  // copies of step t + 1 then refill while step t is computed.
  const int steps = K / kBK;
  if (steps > 0) fetch(0, 0);
  for (int t = 0; t < steps; ++t) {
    wait_vmcnt<0>();  // this wavefront's copies of step t have landed
    lds_barrier();
    if (t + 1 < steps) fetch(t + 1, (t + 1) & 1);
    const char* TA = reinterpret_cast<const char*>(lds) + (t & 1) * kStageBytes;
    const char* TB = TA + kTileA;
#pragma unroll
    for (int kc = 0; kc < kBK / 32; ++kc) {
      // operand of lane (col, grp): row col of the block, k = 32 kc + 8 grp .. + 7
      u16x8 af[kXB], bf[kYB];
#pragma unroll
      for (int x = 0; x < kXB; ++x)
        af[x] = *reinterpret_cast<const u16x8*>(TA + swz(wm + 16 * x + col, 4 * kc + grp));
#pragma unroll
      for (int y = 0; y < kYB; ++y)
        bf[y] = *reinterpret_cast<const u16x8*>(TB + swz(wn + 16 * y + col, 4 * kc + grp));
#pragma unroll
      for (int x = 0; x < kXB; ++x)
#pragma unroll
        for (int y = 0; y < kYB; ++y) acc[x][y] = mfma(af[x], bf[y], acc[x][y]);
    }
  }

  // accumulator cell i of block (x, y) in lane (col, grp): row 16 x + 4 grp + i, column 16 y + col
#pragma unroll
  for (int x = 0; x < kXB; ++x)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t row = m0 + wm + 16 * x + 4 * grp + i;
      if (row >= M) continue;
#pragma unroll
      for (int y = 0; y < kYB; ++y) {
        const int cn = n0 + wn + 16 * y + col;
        if (cn < N) c[row * ldc + cn] = bf16_rne(acc[x][y][i]);
      }
    }
}

}  // namespace

extern "C" int vd_linear(const void* a, int64_t lda, const void* b, int64_t ldb, void* c,
                         int64_t ldc, int64_t M, int32_t N, int32_t K, hipStream_t stream) {
  if (M < 0 || N < 0 || K < 0) return VD_ERR_INVALID_ARG;
  if (M == 0 || N == 0) return VD_OK;
  if (!c || ldc < N || (uintptr_t)c % 2 != 0) return VD_ERR_INVALID_ARG;
  if (K % kBK != 0) return VD_ERR_UNSUPPORTED;
  // a and b are read only when K > 0 (K = 0: every output is the empty sum, +0)
  if (K > 0) {
    if (!a || !b) return VD_ERR_INVALID_ARG;
    if (lda < K || ldb < K || lda % 8 != 0 || ldb % 8 != 0) return VD_ERR_INVALID_ARG;
    if (((uintptr_t)a | (uintptr_t)b) % 16 != 0) return VD_ERR_INVALID_ARG;
  }
  const int64_t tiles_m = (M + kBM - 1) / kBM, tiles_n = ((int64_t)N + kBN - 1) / kBN;
  const int64_t total = tiles_m * tiles_n;
  const Geometry geo = device_geometry();
  const int64_t blocks = (total + geo.xcds - 1) / geo.xcds * geo.xcds;
  if (tiles_m > INT32_MAX || blocks > INT32_MAX) return VD_ERR_INVALID_ARG;
  static std::atomic<unsigned char> lds_set[kMaxDevices];
  if (set_lds_limit(reinterpret_cast<const void*>(&linear_kernel), kLinLds, lds_set) != hipSuccess)
    return VD_ERR_LAUNCH;
  hipLaunchKernelGGL(linear_kernel, dim3((unsigned)blocks), dim3(kThreads), kLinLds, stream,
                     static_cast<const uint16_t*>(a), lda, static_cast<const uint16_t*>(b), ldb,
                     static_cast<uint16_t*>(c), ldc, M, N, K, (int)tiles_m, (int)tiles_n,
                     geo.xcd_shift);
  return hipGetLastError() == hipSuccess ? VD_OK : VD_ERR_LAUNCH;
}
