// vd_cas.hpp -- the canonical arithmetic every attention kernel executes.
//
// Every kernel of the library computes each output row with exactly the
// floating-point operations written here, in this order, on operands laid
// out in registers the same way.  That is the design rule of the paper's
// Section 3 (the runtime may vary batching, storage and access but must keep
// each position's floating-point operation sequence) applied to the online
// softmax update of Appendix A.2 ("A Simplified Tile IR"), plus a split-KV
// merge in a fixed order.  Compile with -ffp-contract=off: no multiply-add is
// fused unless written as one.
//
// Tiling (fixed per handle, never chosen from the batch):
//   * key tile     = 64 logical positions = 4 pages of 16
//   * split        = 1024 logical positions (16 tiles); split k covers keys
//                    [1024k, 1024k + 1024); a row at position p has
//                    ceil((p + 1) / 1024) splits
//   * dot products = v_mfma_f32_16x16x32_bf16, keys in the M dimension and
//                    query-head rows ("columns") in the N dimension, D / 32
//                    instructions chained in ascending d for Q.K and two
//                    chained in ascending key halves for P.V.
//
// Wavefront layout of one 16-column block (lane l, col = l & 15, grp = l >> 4):
//   Q operand (B of Q.K, chunk ks):  q[col][32 ks + 8 grp + j], j = 0..7
//   K operand (A of Q.K, page b, ks): K[key 16 b + col][32 ks + 8 grp + j]
//   score accumulator of page b:     S[key 16 b + 4 grp + i][col], i = 0..3
//   P operand (B of P.V, half h):    slot j <-> key 32 h + 16 (j / 4) + 4 grp + j % 4
//   V operand (A of P.V, d-block m, half h): V[that key][16 m + col]
//   U accumulator of d-block m:      U[16 m + 4 grp + i][col]
// The MFMA result of one (key, column) or (d, column) cell depends only on
// its own row of A, column of B and accumulator cell (checked on gfx950:
// moving a row or column to another slot, or putting NaN in another column,
// leaves its bits unchanged), so the lane a row lands on does not matter.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vd {

constexpr int kPage = 16;       // tokens per page
constexpr int kTileKeys = 64;   // keys per online-softmax step
constexpr int kSplitKeys = 1024; // keys per split (256 and 2048 measured slower on decode)
constexpr int kTilesPerSplit = kSplitKeys / kTileKeys;
constexpr int kPagesPerTile = kTileKeys / kPage;
constexpr int kSplitCols = 32;  // query-head rows per (request, KV head) on the split path
constexpr int kChunkCols = 128; // query-head rows per work item on the chunk path

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma(const u16x8& a, const u16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// exp2 of the hardware transcendental unit (v_exp_f32); one function for
// every kernel.  exp2(-inf) = 0 and exp2(+-0) = 1 exactly.
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// fp32 -> bf16 bits, round to nearest even (v_cvt_pk_bf16_f32; the inputs
// here are finite).
__device__ __forceinline__ uint16_t bf16_rne(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// Output cast: bf16 RNE, with -0 mapped to +0 (an all-zero row may carry
// either sign depending on masked lanes; the canonical output is +0).
__device__ __forceinline__ uint16_t bf16_out(float f) {
  uint16_t b = bf16_rne(f);
  return b == 0x8000u ? (uint16_t)0 : b;
}

__device__ __forceinline__ float fmax_(float a, float b) { return __builtin_fmaxf(a, b); }

// Row exchanges of the vector ALU (a row is 16 lanes): v_permlane16_swap
// trades the odd rows of its first register with the even rows of its second,
// v_permlane32_swap the upper half of the first with the lower half of the
// second.  Both registers holding x, the first then holds the even row (lower
// half) of every pair of lanes l, l ^ 16 (l, l ^ 32) and the second the odd
// row (upper half).  The two wait states before each swap are its hazard
// after a vector-ALU write of either register.  Every lane of the wavefront
// must be active (the callers' tile loops are wave-uniform).
__device__ __forceinline__ void swap_rows16(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void swap_rows32(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}

// The maximum (sum) over the four lanes of a column, l, l ^ 16, l ^ 32 and
// l ^ 48, in every one of them: first each pair of rows (even, odd), then the
// two halves (lower, upper) -- the operands always in that order.
__device__ __forceinline__ float column_max(float x) {
  float a = x, b = x;
  swap_rows16(a, b);
  a = b = fmax_(a, b);
  swap_rows32(a, b);
  return fmax_(a, b);
}
__device__ __forceinline__ float column_sum(float x) {
  float a = x, b = x;
  swap_rows16(a, b);
  a = b = a + b;
  swap_rows32(a, b);
  return a + b;
}

// Online-softmax state of one column (replicated in the 4 lanes of the
// column): running maximum m, normaliser z, and the D/16 accumulator blocks.
template <int D>
struct State {
  float m, z;
  f32x4 u[D / 16];
};

template <int D>
__device__ __forceinline__ void state_init(State<D>& st) {
  st.m = -__builtin_inff();
  st.z = 0.0f;
#pragma unroll
  for (int b = 0; b < D / 16; ++b) st.u[b] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// Score blocks of one tile for NB column blocks: Q.K over D in ascending
// 32-wide chunks, one accumulator chain per (column block, page).  kf(b, ks)
// yields the K operand of page b, chunk ks; a K operand is shared by the
// column blocks, each chain is independent.
template <int D, int NB, class KF>
__device__ __forceinline__ void tile_scores(const KF& kf, const u16x8 (&qf)[NB][D / 32],
                                            f32x4 (&acc)[NB][kPagesPerTile]) {
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int b = 0; b < kPagesPerTile; ++b) acc[nb][b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b)
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const u16x8 k = kf(b, ks);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb][b] = mfma(k, qf[nb][ks], acc[nb][b]);
    }
}

// First key visible to position p: 0, or with a sliding window of w > 0
// keys (Appendix A.5) the window's start, so that key j is visible when
// lo <= j <= p.
__device__ __forceinline__ int window_lo(int p, int w) {
  return (w > 0 && p - w + 1 > 0) ? p - w + 1 : 0;
}

// Softmax half of Appendix A.2's update for the tile starting at logical key
// j0, for the column at position p whose visible keys are lo..p (p < 0: a
// padding column, never visible); c is the base-two scale applied to the raw
// dot.  Produces the weights (cast
// to bf16, the cache type, as the B operand of P.V), alpha, and the candidate
// (m, z); h says whether the column sees any key of the tile.
struct TileWeights {
  u16x8 pf[2];
  float alpha, m_new, z_new;
  uint32_t h;  // 0 or 1; a 32-bit field like the others (a bool here is kept
               // as bytes by the compiler and repacked on every tile)
};

//
// MASKED = false may be used only when every key of the tile is visible to
// every column of the wavefront (lo <= j0 and p >= j0 + 63 in all lanes): all
// selects then take their first operand, so both forms give the same bits.
// WIN = false may be used only when lo = 0 (no sliding window): the test
// key >= lo is then always true and is left out.
template <int D, bool MASKED = true, bool WIN = true>
__device__ __forceinline__ TileWeights tile_softmax(const State<D>& st,
                                                    const f32x4 (&acc)[kPagesPerTile], int j0,
                                                    int p, int lo, float c) {
  const int grp = __lane_id() >> 4;
  float g[kPagesPerTile][4];
  bool lam[kPagesPerTile][4];
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = j0 + 16 * b + 4 * grp + i;
      lam[b][i] = !MASKED || (key <= p && (!WIN || key >= lo));
      g[b][i] = acc[b][i] * c;
    }
  // masked maximum over the tile: fixed tree in the lane, then lanes ^16, ^32
  float t[kPagesPerTile];
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b) {
    const float g0 = lam[b][0] ? g[b][0] : -__builtin_inff();
    const float g1 = lam[b][1] ? g[b][1] : -__builtin_inff();
    const float g2 = lam[b][2] ? g[b][2] : -__builtin_inff();
    const float g3 = lam[b][3] ? g[b][3] : -__builtin_inff();
    t[b] = fmax_(fmax_(g0, g1), fmax_(g2, g3));
  }
  float mx = fmax_(fmax_(t[0], t[1]), fmax_(t[2], t[3]));
  mx = column_max(mx);
  TileWeights w;
  w.h = !MASKED || (j0 <= p && (!WIN || j0 + kTileKeys - 1 >= lo));  // any visible key
  w.m_new = fmax_(st.m, mx);
  // A column with no visible key keeps its state: its weights are all +0
  // (every lam is false), so with alpha = 1 the P.V step adds only zero
  // products to U * 1 = U, which the matrix core returns bit for bit (probe on
  // gfx950: every finite accumulator, denormals included, except -0, which
  // comes back +0 -- and U is never -0: it starts at +0 and only non-negative
  // weights enter it); z * 1 + 0 = z, and tile_commit keeps (m, z).  (m is
  // -inf before the first visible key: ex2 of -inf - -inf would be NaN.)
  w.alpha = w.h ? ex2(st.m - w.m_new) : 1.0f;
  float a[kPagesPerTile][4];
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) a[b][i] = lam[b][i] ? ex2(g[b][i] - w.m_new) : 0.0f;
  // tile sum of the weights: fixed tree in the lane, then lanes ^16, ^32
  float sb[kPagesPerTile];
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b) sb[b] = (a[b][0] + a[b][1]) + (a[b][2] + a[b][3]);
  float s = (sb[0] + sb[1]) + (sb[2] + sb[3]);
  s = column_sum(s);
  w.z_new = st.z * w.alpha + s;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int j = 0; j < 8; ++j) w.pf[hh][j] = bf16_rne(a[2 * hh + j / 4][j % 4]);
  return w;
}

// P.V for d-block m: U <- dot(bf16(A), V, U * alpha), keys in two 32-wide
// halves in ascending order (v0: keys 0-31 of the tile, v1: keys 32-63).  For
// a column without a visible key (h = 0) this is the identity step described
// in tile_softmax: alpha = 1 and zero weights leave U as it was, so no select
// follows the products.  V must be finite for the keys of the tile (keys past
// n are zeroed by the kernels; the others are the cache's values).
template <int D>
__device__ __forceinline__ void tile_pv_block(State<D>& st, const TileWeights& w, int m,
                                              const u16x8& v0, const u16x8& v1) {
  f32x4 u = st.u[m] * w.alpha;
  u = mfma(v0, w.pf[0], u);
  st.u[m] = mfma(v1, w.pf[1], u);
}

// (m, z) <- select(h, new, old)
template <int D>
__device__ __forceinline__ void tile_commit(State<D>& st, const TileWeights& w) {
  st.m = w.h ? w.m_new : st.m;
  st.z = w.h ? w.z_new : st.z;
}

// Merge of split partial states in ascending split order (a left fold):
//   (M, Z, W) <- partial 0;  for k >= 1:
//   M' = max(M, m_k), a = exp2(M - M'), b = exp2(m_k - M'),
//   Z <- Z a + z_k b,  W <- W a + U_k b.
struct FoldScalars {
  float M, Z, a, b;
};

__device__ __forceinline__ FoldScalars fold_scalars(float M, float Z, float mk, float zk) {
  FoldScalars f;
  const float Mn = fmax_(M, mk);
  f.a = ex2(M - Mn);
  f.b = ex2(mk - Mn);
  f.Z = Z * f.a + zk * f.b;
  f.M = Mn;
  return f;
}

__device__ __forceinline__ float fold_value(float W, float uk, const FoldScalars& f) {
  return W * f.a + uk * f.b;
}

// Final normalisation: o = cast(W * select(Z > 0, 1 / Z, 0)), IEEE division.
__device__ __forceinline__ float final_scale(float Z) { return Z > 0.0f ? 1.0f / Z : 0.0f; }

// Log-sum-exp of the row's visible scaled scores, in natural log: the state
// (M, Z) holds M = the largest base-two score c * dot and Z = the sum of
// exp2(score - M) (at least 1 for a row with a visible key), so
// ln sum exp(scale * dot) = (M + log2 Z) * ln 2; log2 is v_log_f32.
constexpr float kLn2 = 0.693147180559945309417f;
__device__ __forceinline__ float final_lse(float M, float Z) {
  return (M + __builtin_amdgcn_logf(Z)) * kLn2;
}

}  // namespace vd
