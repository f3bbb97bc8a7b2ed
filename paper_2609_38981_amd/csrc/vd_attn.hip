// vd_attn.hip -- HIP kernels for gfx950 and the C ABI of libvdattn.so.
//
// Kernels of one attention call, all on the caller's stream:
//   plan kernel   launched only when needed (more than 256 requests, new
//                 tokens the split items do not write, or the shared_pages
//                 hint).  Workgroup 0 reads the per-request lengths and
//                 writes the split work list and, with the hint, the
//                 shared-prefix plan (groups of adjacent requests whose page
//                 tables share leading splits) into the workspace, with no
//                 device-to-host synchronisation; its other workgroups write
//                 the call's new tokens into the pool.  Without a plan
//                 launch, the split and chunk workgroups derive their items
//                 from the lengths themselves.
//   prefix kernel one workgroup (4 wavefronts x 32 columns) per (KV head,
//                 listed group, 128 query-head rows of its members, shared
//                 split): each shared split is read once for all member rows;
//                 writes the same partial states their split items would.
//   split kernel  one wavefront (workgroup) per (request, KV head, 1024-key
//                 split, 16 query-head rows) for requests with at most 32
//                 query-head rows per KV head (decode, verify).  K/V go
//                 straight from HBM to registers in the matrix-core operand
//                 layout; writes a partial state.  Whole 1024-key splits are
//                 listed before the shorter last splits, and those by
//                 decreasing length, so the shortest items fill the end of
//                 the launch.
//   chunk kernel  one workgroup (4 wavefronts x 32 columns) per (request,
//                 KV head, 128 query-head rows) for longer chunks (prefill);
//                 K/V tiles are staged in LDS and shared by the wavefronts;
//                 the splits are folded in registers with the merge's fold.
//   merge kernel  folds the split partial states in ascending split order
//                 and writes the output rows of the split-path requests.
// The work decomposition differs between kernels; the operations applied to
// any one output row, and their order (vd_cas.hpp), do not.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <new>

#include "../../include/vdattn.h"
#include "vd_cas.hpp"
#include "vd_hw.hpp"

using namespace vd;

namespace {

struct Params {
  const uint16_t* q;
  const int32_t* cu;
  const int32_t* ctx;
  const int32_t* pt;
  const uint16_t* kpool;
  const uint16_t* vpool;
  uint16_t* out;
  int32_t* off_full;   // [num_seqs + 1] prefix offsets of whole-split items
  int32_t* off_part;   // [num_seqs + 1] prefix offsets of last-split items
  int32_t* off_chunk;  // [num_seqs + 1] prefix offsets of q-tiles (per KV head)
  int32_t* items;      // [num_seqs * Hkv * max_splits][8] split work list
  float* ws_m;
  float* ws_z;
  float* ws_u;
  int64_t T;
  int32_t num_pages;  // page ids are int32: pages past INT32_MAX are unreachable
  int num_seqs, pt_stride, max_q, max_ctx, max_splits, split_cols;
  // partial states per (request, KV head, split): one per query-head row of
  // the split path, min(max_q * G, 32) of them (the layout's column stride)
  int ws_cols;
  int hq, hkv, G;
  // the dies workgroups are dispatched over (workgroup b on die b mod xcds,
  // xcds = 1 << xcd_shift); item ranges are assigned per die
  int xcds, xcd_shift;
  int window;  // sliding window in keys (Appendix A.5), 0 = the full causal prefix
  float c;  // softmax scale * log2(e), rounded once to fp32 on the host
  // optional K/V of the call's query rows ([T, Hkv, D]), written into the pool
  // before attention reads it: by the plan launch, or (fuse_write) by the
  // split launch -- the split items write the rows of their own requests, and
  // the launch's last append_wgs workgroups (0: none) those of the chunk-path
  // requests, which the chunk launch reads after it
  const uint16_t* knew;
  const uint16_t* vnew;
  int fuse_write, append_wgs;
  // a split item covers all 32 query-head rows of its split (two column
  // blocks over one read of each tile) instead of 16
  int wide;
  // the split workgroups derive their items from the lengths (no plan launch)
  int inwave;
  float* lse;  // optional [T, Hq] log-sum-exp output
  // shared-prefix pass (calls with the shared_pages hint): the plan launch
  // finds groups of adjacent requests whose page tables start with the same
  // pages; the shared-prefix kernel computes their leading splits once
  int casc;
  int32_t* casc_hdr;  // {listed groups, items per KV head}
  int32_t* casc_seq;  // [num_seqs] leading splits of the request computed by it (0: none)
  int32_t* casc_off;  // [listed groups + 1] first item of each group
  int4* casc_grp;     // [listed groups] {first member, last member + 1, splits, first token}
  // split slots past the first grid are claimed from this counter, zeroed by
  // a fill launch just before the split launch (nullptr: every workgroup runs
  // the slots b, b + grid, ... of its own die)
  int32_t* claim;
};

struct Req {
  int q0, s, n;
  bool valid;
};

// Reads request r's lengths and decides whether it may be processed without
// touching memory outside the described buffers.
__device__ __forceinline__ Req make_req(const Params& P, int q0, int q1, int n) {
  Req R;
  R.q0 = q0;
  R.s = q1 - q0;
  R.n = n;
  const int npages = (n + kPage - 1) / kPage;
  R.valid = q0 >= 0 && R.s >= 1 && R.s <= n && (int64_t)q1 <= P.T && R.s <= P.max_q &&
            n <= P.max_ctx && npages <= P.pt_stride;
  return R;
}

__device__ __forceinline__ Req load_req(const Params& P, int r) {
  return make_req(P, P.cu[r], P.cu[r + 1], P.ctx[r]);
}


// Largest r in [0, nseq) with off[r] <= i, for a non-decreasing off[] with
// off[0] = 0 <= i < off[nseq]: the request whose item range holds item i.
// 64-ary search, one vector load per level (wave-uniform result).
__device__ __forceinline__ int find_req(const int32_t* off, int nseq, int i) {
  const int lane = __lane_id();
  int lo = 0, hi = nseq;
  while (hi - lo > 1) {
    const int step = (hi - lo + 63) / 64;
    const int cand = lo + lane * step;
    const bool le = cand < hi && off[cand] <= i;
    const unsigned long long m = __ballot(le);
    const int j = 63 - __clzll(m);
    lo = uni(lo + j * step);
    hi = uni(min(hi, lo + step));
  }
  return lo;
}

// Index of the (page, kv_head) page block, or -1 when the logical page lp is
// past the request's keys or its id is outside the pool.
__device__ __forceinline__ int64_t page_block(const Params& P, const int32_t* ptrow, int lp,
                                              int n, int g) {
  const int npages = (n + kPage - 1) / kPage;
  if (lp >= npages) return -1;
  // the page table is read-only for the whole call: a scalar load
  typedef __attribute__((address_space(4))) const int32_t const_i32;
  const int32_t page = ((const_i32*)ptrow)[lp];
  if (page < 0 || page >= P.num_pages) return -1;
  return (int64_t)page * P.hkv + g;
}

template <int D>
__device__ __forceinline__ const uint16_t* block_ptr(const uint16_t* pool, int64_t pb) {
  return pool + pb * (int64_t)(kPage * D);
}

__device__ __forceinline__ u16x8 zero8() { return u16x8{0, 0, 0, 0, 0, 0, 0, 0}; }

// Tile kt lies wholly below key n.
__device__ __forceinline__ bool j0_full(int kt, int n) { return (kt + 1) * kTileKeys <= n; }

__device__ __forceinline__ u16x8 cat4(u16x4 a, u16x4 b) {
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Keeps the 4 bf16 values of slots 4 grp .. 4 grp + 3 whose key is < n.
__device__ __forceinline__ u16x4 mask4(u16x4 v, int key0, int n) {
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = (key0 + i < n) ? v[i] : (uint16_t)0;
  return v;
}

template <int D>
__device__ __forceinline__ void load_q(const Params& P, u16x8 (&qf)[D / 32], int tok, int head,
                                       bool valid) {
  const int grp = __lane_id() >> 4;
  const uint16_t* base = P.q + ((int64_t)tok * P.hq + head) * D + 8 * grp;
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks)
    qf[ks] = valid ? *reinterpret_cast<const u16x8*>(base + 32 * ks) : zero8();
}

// Splits that hold a visible key of some row of request R: from the split of
// the first row's window start through the split of key n - 1.  When it is
// one, the split kernel writes the rows; otherwise the merge kernel does.
__device__ __forceinline__ int request_splits(const Req& R, int window) {
  return (R.n - 1) / kSplitKeys + 1 - window_lo(R.n - R.s, window) / kSplitKeys;
}

// Stores one column's output row from its accumulator blocks (lane layout of
// the U accumulator: d = 16 m + 4 grp + i), and its log-sum-exp when asked.
template <int D>
__device__ __forceinline__ void store_row(const Params& P, const f32x4 (&u)[D / 16], float M,
                                          float Z, int64_t tok, int head) {
  const int grp = __lane_id() >> 4;
  const float rho = final_scale(Z);
  if (P.lse && grp == 0) P.lse[tok * P.hq + head] = final_lse(M, Z);
  uint16_t* o = P.out + (tok * P.hq + head) * D + 4 * grp;
#pragma unroll
  for (int m = 0; m < D / 16; ++m) {
    u16x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = bf16_out(u[m][i] * rho);
    *reinterpret_cast<u16x4*>(o + 16 * m) = v;
  }
}

// Stores 8 consecutive d (chunk dc) of one token's K and V at slot s of the
// page block starting at element blk, in the pool layout:
//   K block: element (slot, d) at ((d / 8) * 16 + slot) * 8 + d % 8
//   V block: element (slot, d) at ((d / 16) * 4 + slot / 4) * 64 + (d % 16) * 4 + slot % 4
template <int D>
__device__ __forceinline__ void put_kv8(uint16_t* kpool, uint16_t* vpool, int64_t blk, int s,
                                        int dc, const u16x8& kv, const u16x8& vv) {
  *reinterpret_cast<u16x8*>(kpool + blk + ((int64_t)dc * kPage + s) * 8) = kv;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int d = 8 * dc + e;
    vpool[blk + ((d / 16) * 4 + s / 4) * 64 + (d % 16) * 4 + s % 4] = vv[e];
  }
}

// Writes one (token, KV head, 8 consecutive d) of new K/V to the token's slot.
template <int D>
__device__ __forceinline__ void kv_write_one(const uint16_t* knew, const uint16_t* vnew,
                                             const int64_t* slots, int64_t ntok, uint16_t* kpool,
                                             uint16_t* vpool, int64_t num_pages, int hkv,
                                             int64_t id) {
  const int64_t per_tok = (int64_t)hkv * (D / 8);
  if (id >= ntok * per_tok) return;
  const int64_t t = id / per_tok;
  const int hd = (int)(id % per_tok);
  const int h = hd / (D / 8);
  const int dc = hd % (D / 8);
  const int64_t slot = slots[t];
  if (slot < 0 || slot >= num_pages * kPage) return;
  const int64_t page = slot / kPage;
  const int64_t src = (t * hkv + h) * D + 8 * dc;
  put_kv8<D>(kpool, vpool, (page * hkv + h) * (int64_t)(kPage * D), (int)(slot % kPage), dc,
             *reinterpret_cast<const u16x8*>(knew + src),
             *reinterpret_cast<const u16x8*>(vnew + src));
}

// Calls of at most this many requests find a row's request with one load of
// all the lengths instead of a search.
constexpr int kAppendInWaveSeqs = 256;

// Writes the K/V of the call's query rows (every KV head) at the slots their
// positions have in the request's page table.  The wavefront of query row t
// writes the rows of t's 4-slot group (positions p .. up to the next multiple
// of 4), when t is the request's first row or starts such a group; the V
// layout keeps 4 consecutive slots of one d contiguous, so a whole group is
// written with 8-byte stores.
template <int D>
__device__ __forceinline__ void append_rows(const Params& P, int64_t t) {
  if (t >= P.T) return;
  int r;
  Req R;
  if (P.num_seqs <= kAppendInWaveSeqs) {
    // one round trip: lane l holds the lengths of requests l, 64 + l, ...;
    // row t belongs to the request after every request that ends at or
    // before it
    constexpr int C = kAppendInWaveSeqs / 64;
    const int lane = __lane_id();
    int cq0[C], cq1[C], cn[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const int rr = min(64 * c + lane, P.num_seqs - 1);
      cq0[c] = P.cu[rr];
      cq1[c] = P.cu[rr + 1];
      cn[c] = P.ctx[rr];
    }
    r = 0;
#pragma unroll
    for (int c = 0; c < C; ++c) r += __popcll(__ballot(64 * c + lane < P.num_seqs && cq1[c] <= t));
    r = uni(r);
    if (r >= P.num_seqs) return;
    int q0 = 0, q1 = 0, n = 0;
#pragma unroll
    for (int c = 0; c < C; ++c)
      if (c == r / 64) {
        q0 = __builtin_amdgcn_readlane(cq0[c], r % 64);
        q1 = __builtin_amdgcn_readlane(cq1[c], r % 64);
        n = __builtin_amdgcn_readlane(cn[c], r % 64);
      }
    R = make_req(P, q0, q1, n);
  } else {
    r = find_req(P.cu, P.num_seqs, (int)t);
    R = load_req(P, r);
  }
  if (!R.valid || t < R.q0 || t >= (int64_t)R.q0 + R.s) return;
  const int p0 = R.n - R.s;
  const int p = p0 + (int)(t - R.q0);
  if (p != p0 && (p & 3) != 0) return;  // written by the wavefront of its group's first row
  const int cnt = min(R.n, (p & ~3) + 4) - p;  // rows t .. t + cnt - 1
  // the page id is loaded with the first batch of K rows (one round trip)
  const int32_t* pte = P.pt + (int64_t)r * P.pt_stride + p / kPage;
  int32_t page = -1;
  const int slot0 = p % kPage;
  const int lane = __lane_id();
  const int64_t rs = (int64_t)P.hkv * D;  // elements per row of k_new / v_new
  uint16_t* kpool = const_cast<uint16_t*>(P.kpool);
  uint16_t* vpool = const_cast<uint16_t*>(P.vpool);
  // Loads are issued in batches of B before their stores (the compiler must
  // assume that the pool stores may alias k_new / v_new).
  constexpr int B = 8;
  // K: one 16-byte piece per (row, head, 8 d): element (slot, d) at ((d / 8) * 16 + slot) * 8 + d % 8
  const int nk = cnt * P.hkv * (D / 8);
  for (int x0 = 0; x0 < nk; x0 += 64 * B) {
    u16x8 v[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int x = x0 + 64 * u + lane;
      if (x < nk) {
        const int i = x / (P.hkv * (D / 8)), hd = x % (P.hkv * (D / 8));
        v[u] = *reinterpret_cast<const u16x8*>(P.knew + (t + i) * rs + hd * 8);
      }
    }
    if (x0 == 0) {
      page = *pte;
      if (page < 0 || page >= P.num_pages) return;
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int x = x0 + 64 * u + lane;
      if (x < nk) {
        const int i = x / (P.hkv * (D / 8)), hd = x % (P.hkv * (D / 8));
        const int h = hd / (D / 8), dc = hd % (D / 8);
        const int64_t blk = ((int64_t)page * P.hkv + h) * (kPage * D);
        *reinterpret_cast<u16x8*>(kpool + blk + ((int64_t)dc * kPage + slot0 + i) * 8) = v[u];
      }
    }
  }
  // V: per (head, d) the group's values: element (slot, d) at
  // ((d / 16) * 4 + slot / 4) * 64 + (d % 16) * 4 + slot % 4
  const int nv = P.hkv * D;
  for (int x0 = 0; x0 < nv; x0 += 64 * B) {
    u16x4 v[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int x = x0 + 64 * u + lane;
      if (x < nv) {
        const uint16_t* src = P.vnew + t * rs + x;  // x = h * D + d
#pragma unroll
        for (int i = 0; i < 4; ++i) v[u][i] = i < cnt ? src[i * rs] : (uint16_t)0;
      }
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int x = x0 + 64 * u + lane;
      if (x < nv) {
        const int h = x / D, d = x % D;
        uint16_t* dst = vpool + ((int64_t)page * P.hkv + h) * (kPage * D) +
                        ((d / 16) * 4 + slot0 / 4) * 64 + (d % 16) * 4 + slot0 % 4;
        if (cnt == 4) {  // a whole group (slot0 % 4 == 0)
          *reinterpret_cast<u16x4*>(dst) = v[u];
        } else {
          for (int i = 0; i < cnt; ++i) dst[i] = v[u][i];
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// plan kernel: workgroup 0 (1024 threads) plans; workgroups 1.. write the
// call's new tokens into the pool
// ---------------------------------------------------------------------------
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = __lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}

// A split item covers 16 query-head rows ("columns") of its request: a
// request with more (s * G in 17 .. 32) has an item per split and column half
// -- or, in a call with wide items, one item covering both halves.
__device__ __forceinline__ int column_halves(const Params& P, const Req& R) {
  return !P.wide && R.s * P.G > 16 ? 2 : 1;
}

// Length of the split work list: an upper bound of the split items.
__host__ __device__ __forceinline__ int64_t split_slots(const Params& P) {
  return (int64_t)P.num_seqs * P.hkv * P.max_splits * (P.wide ? 1 : P.split_cols / 16);
}

// Work-list entry of one split item: request, KV head, split index, the
// request's lengths, the column half and the request's leading splits that the
// shared-prefix kernel computes, so that a split wavefront reaches its first
// K/V loads after a single scalar load.  r = -1 marks an unused slot.
constexpr int kItemInts = 8;  // {r, g, k, n, q0, s, half, pre}
// Number of counters of the planning scan: whole splits, chunk q-tiles, and
// the last (partial) splits by their tile count, 16 down to 1.
constexpr int kPlanCounters = 2 + kTilesPerSplit;

__device__ __forceinline__ void put_item(const Params& P, int64_t idx, int r, int g, int k,
                                         const Req& R, int half, int pre) {
  int4* e = reinterpret_cast<int4*>(P.items + idx * kItemInts);
  e[0] = int4{r, g, k, R.n};
  e[1] = int4{R.q0, R.s, half, pre};
}

// ---------------------------------------------------------------------------
// shared-prefix planning (plan workgroup 0, calls with the shared_pages hint)
// ---------------------------------------------------------------------------
// Requests of a call the shared-prefix pass examines, and the leading splits
// of a request it may cover.
constexpr int kCascMaxSeqs = 1024;
constexpr int kCascMaxSplits = 32;
constexpr int kPagesPerSplit = kSplitKeys / kPage;

// Inclusive prefix sum over the 1024 threads of the workgroup; *total gets
// the sum over all of them.  Every thread of the workgroup must call it.
__device__ __forceinline__ int block_incl_scan(int v, int* total) {
  __shared__ int wtot[16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int x = wave_incl_scan(v);
  if (lane == 63) wtot[wave] = x;
  __syncthreads();
  int pre = 0, all = 0;
  for (int w = 0; w < 16; ++w) {
    const int t = wtot[w];
    pre += w < wave ? t : 0;
    all += t;
  }
  __syncthreads();  // wtot is reused by the next call
  *total = all;
  return x + pre;
}

// Reduction over the lanes from this one to the end of its run of equal
// keys, for keys that do not decrease across the lanes (a run is contiguous):
// the first lane of each run gets the run's min (MIN) or sum.
template <bool MIN>
__device__ __forceinline__ int run_reduce(int v, int key) {
  const int lane = __lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_down(v, o, 64), tk = __shfl_down(key, o, 64);
    if (lane + o < 64 && tk == key) v = MIN ? min(v, t) : v + t;
  }
  return v;
}

__device__ __forceinline__ bool run_start(int key) {
  const int lane = __lane_id();
  const int prev = __shfl_up(key, 1, 64);
  return lane == 0 || prev != key;
}

// Groups of adjacent requests that share leading splits, listed for the
// shared-prefix kernel.
//  * Requests r - 1 and r (both valid) share split k when their page-table
//    entries of splits 0 .. k are equal: the same physical pages, hence the
//    same keys and values.  sh(r) counts the leading splits they share (at
//    most kCascMaxSplits, within both contexts).
//  * A group is a maximal run of requests with sh >= 1 between neighbours; it
//    shares c = the smallest sh of the run.  An invalid request is a group of
//    its own, so the query rows of a group's requests are consecutive.
//  * A member is a request of a group on the split path whose query rows all
//    lie past the c shared splits (n - s >= 1024 c): each of its rows sees
//    every key of them, and none of them is a new token of the call.
//  * A group with at least two members is listed: its members' splits
//    0 .. c - 1 are computed by the shared-prefix kernel (csq[r] = c), their
//    later splits by the split kernel.  Its items are (tile of 128 query-head
//    rows over the members' query rows, shared split).
// Requires num_seqs <= kCascMaxSeqs and 1024 threads.  One round trip to
// memory: the lengths and every page-table entry compared are loaded
// together (the comparison runs over the first E entries of every row,
// E = 64 * min(kCascMaxSplits, max_context_len / 1024) within the table stride,
// and is cut to the pair's own contexts afterwards).
template <int W>  // entries per load: 1, or 4 for a 16-byte aligned table
__device__ __forceinline__ void compare_rows(const Params& P, int B, int E, int* fd) {
  typedef int vec __attribute__((ext_vector_type(W)));
  const int U = E / W;                        // loads per row
  const int flat = (B - 1) * U;               // pairs (r - 1, r), r = 1 .. B - 1
  constexpr int J = 32 / W < 16 ? 32 / W : 16;  // loads of each row per thread and round
  for (int f0 = 0; f0 < flat; f0 += 1024 * J) {
    vec a[J], b[J];
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int f = f0 + (int)threadIdx.x + 1024 * j;
      const bool ok = f < flat;
      const int r = 1 + (ok ? f / U : 0), u = ok ? f % U : 0;
      const vec* row = reinterpret_cast<const vec*>(P.pt + (int64_t)r * P.pt_stride) + u;
      a[j] = ok ? row[0] : vec{};
      b[j] = ok ? *reinterpret_cast<const vec*>(P.pt + (int64_t)(r - 1) * P.pt_stride + u * W) : vec{};
    }
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int f = f0 + (int)threadIdx.x + 1024 * j;
      if (f < flat) {
        int e = E;  // first differing entry of the unit
#pragma unroll
        for (int w = W - 1; w >= 0; --w)
          if (a[j][w] != b[j][w]) e = (f % U) * W + w;
        if (e < E) atomicMin(&fd[1 + f / U], e);
      }
    }
  }
}

__device__ void plan_prefix(const Params& P, int* csq) {
  __shared__ int fd[kCascMaxSeqs];   // first entry where rows r - 1 and r differ
  __shared__ int sq[kCascMaxSeqs + 1], sn[kCascMaxSeqs];  // cu and n
  __shared__ int gmin[kCascMaxSeqs], gcnt[kCascMaxSeqs], gfirst[kCascMaxSeqs],
      glast[kCascMaxSeqs];
  const int tid = threadIdx.x;
  const int B = P.num_seqs;
  const int r = tid;
  const int E = kPagesPerSplit * min(kCascMaxSplits, min(P.max_ctx / kSplitKeys,
                                                          P.pt_stride / kPagesPerSplit));
  fd[tid] = E;
  __syncthreads();
  int q0 = 0, q1 = 0, n = 0;
  if (r < B) {
    q0 = P.cu[r];
    q1 = P.cu[r + 1];
    n = P.ctx[r];
  }
  if (E > 0) {
    if ((reinterpret_cast<uintptr_t>(P.pt) % 16 == 0) && P.pt_stride % 4 == 0)
      compare_rows<4>(P, B, E, fd);
    else
      compare_rows<1>(P, B, E, fd);
  }
  if (r < B) {
    sq[r] = q0;
    sn[r] = n;
    if (r == B - 1) sq[B] = q1;
  }
  __syncthreads();
  // Requests r - 1 and r (both valid) share split k when their entries of
  // splits 0 .. k are equal and both contexts reach past split k.
  int sh = 0, vis = -1;
  if (r < B) {
    const Req R = make_req(P, q0, q1, n);
    if (R.valid && R.s * P.G <= P.split_cols) vis = (R.n - R.s) / kSplitKeys;
    if (r > 0 && R.valid && make_req(P, sq[r - 1], q0, sn[r - 1]).valid)
      sh = min(fd[r] / kPagesPerSplit, min(R.n, sn[r - 1]) / kSplitKeys);
  }
  const bool head = r < B && (r == 0 || sh == 0);
  int ngroups;
  const int gid = block_incl_scan(head ? 1 : 0, &ngroups) - 1;  // group of r (r < B)
  if (head) {
    gmin[gid] = kCascMaxSplits + 1;  // a group of one request shares nothing
    gcnt[gid] = 0;
    gfirst[gid] = kCascMaxSeqs;
    glast[gid] = -1;
  }
  __syncthreads();
  // per-group statistics: a wavefront's lanes are consecutive requests, so
  // each run of one group in it adds one atomic
  const int key = r < B ? gid : kCascMaxSeqs;  // gid does not decrease with r
  {
    const int v = run_reduce<true>(r < B && !head ? sh : kCascMaxSplits + 1, key);
    if (r < B && run_start(key)) atomicMin(&gmin[gid], v);
  }
  __syncthreads();
  const int c = r < B ? gmin[gid] : 0;
  const bool member = r < B && c <= kCascMaxSplits && vis >= c;
  {
    const int cnt = run_reduce<false>(member ? 1 : 0, key);
    const int lo = run_reduce<true>(member ? r : kCascMaxSeqs, key);
    const int hi = -run_reduce<true>(member ? -r : 1, key);
    if (r < B && run_start(key) && cnt > 0) {
      atomicAdd(&gcnt[gid], cnt);
      atomicMin(&gfirst[gid], lo);
      atomicMax(&glast[gid], hi);
    }
  }
  __syncthreads();
  const int take = member && gcnt[gid] >= 2 ? c : 0;
  if (r < B) {
    csq[r] = take;
    P.casc_seq[r] = take;
  }
  // the list: groups with at least two members, in request order, each with
  // an item per (tile of 128 query-head rows over the members' query rows,
  // shared split)
  const int gi = tid;
  const bool listed = gi < ngroups && gcnt[gi] >= 2;
  int items = 0;
  if (listed)
    items = gmin[gi] *
            (int)(((int64_t)(sq[glast[gi] + 1] - sq[gfirst[gi]]) * P.G + kChunkCols - 1) /
                  kChunkCols);
  int nlisted, nitems;
  const int li = block_incl_scan(listed ? 1 : 0, &nlisted) - 1;
  const int ioff = block_incl_scan(items, &nitems) - items;
  if (listed) {
    P.casc_grp[li] = int4{gfirst[gi], glast[gi] + 1, gmin[gi], sq[gfirst[gi]]};
    P.casc_off[li] = ioff;
  }
  if (tid == 0) {
    P.casc_off[nlisted] = nitems;
    P.casc_hdr[0] = nlisted;
    P.casc_hdr[1] = nitems;
  }
  __syncthreads();
}

template <int D>
__global__ __launch_bounds__(1024) void plan_kernel(Params P) {
  if (blockIdx.x > 0) {
    // the K/V of the call's query rows (workgroups 1..: a wavefront per row)
    append_rows<D>(P, (int64_t)(blockIdx.x - 1) * 16 + (threadIdx.x >> 6));
    return;
  }
  __shared__ int csq[kCascMaxSeqs];  // leading splits of request r the shared-prefix kernel runs
  if (P.casc) plan_prefix(P, csq);
  if (P.inwave) return;  // the split and chunk workgroups plan for themselves
  constexpr int NC = kPlanCounters;
  __shared__ int wsum[NC][16];  // per-wavefront totals of each counter
  __shared__ int wpre[NC][16];  // offset of each (counter, wavefront)
  __shared__ int sbase[NC];     // running totals over the request chunks
  __shared__ int pstart[NC];    // first item of each partial-split class
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const unsigned long long below = (1ull << lane) - 1;
  if (tid < NC) sbase[tid] = 0;
  __syncthreads();
  // Pass 1: prefix offsets.  Split items: every whole split, then the last
  // partial splits ordered by decreasing tile count (longest first), so that
  // the items that start late in the launch are the shortest.  Counter 0:
  // whole-split items; 1: chunk q-tiles per KV head; 2 + 16 - t: requests whose
  // last split has t tiles (Hkv items each), counted with ballots.
  for (int r0 = 0; r0 < P.num_seqs; r0 += 1024) {
    const int r = r0 + tid;
    int cfull = 0, cchunk = 0, cls = -1, h = 1;
    if (r < P.num_seqs) {
      const Req R = load_req(P, r);
      if (R.valid) {
        const int ncols = R.s * P.G;
        if (ncols <= P.split_cols) {
          h = column_halves(P, R);
          // splits before the one holding the first row's window start
          // hold no visible key and get no item
          const int lo_min = window_lo(R.n - R.s, P.window);
          // (and before those of the shared-prefix kernel)
          const int kfirst = max(lo_min / kSplitKeys, P.casc ? csq[r] : 0);
          const int nfull = R.n / kSplitKeys;
          cfull = P.hkv * h * max(0, nfull - kfirst);
          if (R.n % kSplitKeys) {
            // tiles the last split's items run
            const int t = (R.n + kTileKeys - 1) / kTileKeys -
                          max(nfull * kTilesPerSplit, lo_min / kTileKeys);
            cls = 2 + kTilesPerSplit - t;
          }
        } else if (ncols > kSplitCols) {
          cchunk = (ncols + kChunkCols - 1) / kChunkCols;  // q-tiles per KV head
        }
      }
    }
    const int ifull = wave_incl_scan(cfull), ichunk = wave_incl_scan(cchunk);
    int rank = 0;  // items per KV head of the same class below this lane in the wavefront
#pragma unroll
    for (int c = 2; c < NC; ++c) {
      const unsigned long long m = __ballot(cls == c), m2 = __ballot(cls == c && h == 2);
      rank = cls == c ? __popcll(m & below) + __popcll(m2 & below) : rank;
      if (lane == 0) wsum[c][wave] = (__popcll(m) + __popcll(m2)) * P.hkv;
    }
    if (lane == 63) {
      wsum[0][wave] = ifull;
      wsum[1][wave] = ichunk;
    }
    __syncthreads();
    if (tid < NC * 16) {
      const int c = tid / 16, w = tid % 16;
      int pre = sbase[c];
      for (int x = 0; x < w; ++x) pre += wsum[c][x];
      wpre[c][w] = pre;
    }
    __syncthreads();
    if (r < P.num_seqs) {
      P.off_full[r] = wpre[0][wave] + ifull - cfull;
      P.off_part[r] = cls >= 2 ? wpre[cls][wave] + rank * P.hkv : 0;  // within its class
      P.off_chunk[r] = wpre[1][wave] + ichunk - cchunk;
    }
    if (tid < NC) sbase[tid] = wpre[tid][15] + wsum[tid][15];
    __syncthreads();
  }
  if (tid == 0) {
    int t = sbase[0];
    for (int c = 2; c < NC; ++c) {
      pstart[c] = t;
      t += sbase[c];
    }
    pstart[0] = t;  // total number of split items
    P.off_full[P.num_seqs] = sbase[0];
    P.off_part[P.num_seqs] = t - sbase[0];
    P.off_chunk[P.num_seqs] = sbase[1];
  }
  __syncthreads();
  const int total = pstart[0];
  // Pass 2: the split work list.  Wavefront w lists the items of requests
  // w, w + 16, ...: lane j first reads the lengths and offsets of request
  // w + 16 j, then the wavefront takes the requests in turn, its lanes
  // writing one entry each.  Whole splits kfirst .. nfull - 1 of a request
  // are listed KV-head-major: item off_full + g * (nfull - kfirst) + k - kfirst.
  for (int rb = 0; rb < P.num_seqs; rb += 1024) {
    const int rl = rb + wave + 16 * lane;
    int q0 = 0, s = 0, n = 0, fo = 0, po = -1;  // po < 0: no split items
    if (rl < P.num_seqs) {
      const Req R = load_req(P, rl);
      if (R.valid && R.s * P.G <= P.split_cols) {
        q0 = R.q0;
        s = R.s;
        n = R.n;
        fo = P.off_full[rl];
        if (R.n % kSplitKeys) {
          const int lo_min = window_lo(R.n - R.s, P.window);
          const int t = (R.n + kTileKeys - 1) / kTileKeys -
                        max(R.n / kSplitKeys * kTilesPerSplit, lo_min / kTileKeys);
          po = pstart[2 + kTilesPerSplit - t] + P.off_part[rl];
        } else {
          po = 0;
        }
      }
    }
    for (int j = 0; j < 64; ++j) {
      const int r = rb + wave + 16 * j;
      if (r >= P.num_seqs) break;
      if (__builtin_amdgcn_readlane(po, j) < 0) continue;
      Req R;
      R.q0 = __builtin_amdgcn_readlane(q0, j);
      R.s = __builtin_amdgcn_readlane(s, j);
      R.n = __builtin_amdgcn_readlane(n, j);
      R.valid = true;
      const int rfo = __builtin_amdgcn_readlane(fo, j), rpo = __builtin_amdgcn_readlane(po, j);
      const int nfull = R.n / kSplitKeys;
      const int kfirst = max(window_lo(R.n - R.s, P.window) / kSplitKeys, P.casc ? csq[r] : 0);
      const int nf = nfull - kfirst;  // whole splits with items
      const int h = column_halves(P, R);
      const int pre = P.casc ? csq[r] : 0;
      // items (KV head, split, half), halves adjacent
      for (int idx = lane; idx < P.hkv * nf * h; idx += 64)
        put_item(P, (int64_t)rfo + idx, r, idx / (nf * h), kfirst + idx % (nf * h) / h, R, idx % h,
                 pre);
      if (R.n % kSplitKeys)
        for (int x = lane; x < P.hkv * h; x += 64)
          put_item(P, (int64_t)rpo + x, r, x / h, nfull, R, x % h, pre);
    }
  }
  // Pass 3: slots past the list end the split workgroups' loops
  const int64_t upper = split_slots(P);
  for (int64_t i = total + tid; i < upper; i += 1024) P.items[i * kItemInts] = -1;
}

// ---------------------------------------------------------------------------
// split kernel
// ---------------------------------------------------------------------------
// Issue the loads of one tile's K (resp. V) operands.  Every lane loads from
// a valid page block (a page id that is out of range or past n reads block 0
// instead), so the load sequence is the same on every tile; the values that
// must not be used are zeroed afterwards by mask_k / mask_v.
// NT: non-temporal loads (the data streams past the caches; each page is read
// once), else ordinary loads (pages shared by several requests stay cached).
template <bool NT, class V>
__device__ __forceinline__ V load_kv(const uint16_t* p) {
  if (NT) return __builtin_nontemporal_load(reinterpret_cast<const V*>(p));
  return *reinterpret_cast<const V*>(p);
}

template <int D, bool NT>
__device__ __forceinline__ void load_k(const Params& P, const int64_t (&pb)[kPagesPerTile],
                                       u16x8 (&kf)[kPagesPerTile][D / 32]) {
  const int lane = __lane_id();
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b) {
    const int64_t blk = pb[b] < 0 ? 0 : pb[b];
    const uint16_t* kb = block_ptr<D>(P.kpool, blk) + 8 * lane;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) kf[b][ks] = load_kv<NT, u16x8>(kb + 512 * ks);
  }
}

template <int D, bool NT>
__device__ __forceinline__ void load_v(const Params& P, const int64_t (&pb)[kPagesPerTile],
                                       u16x4 (&vh)[D / 16][kPagesPerTile]) {
  const int lane = __lane_id();
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b) {
    const int64_t blk = pb[b] < 0 ? 0 : pb[b];
    const uint16_t* vb = block_ptr<D>(P.vpool, blk) + 4 * lane;  // = 64 grp + 4 col
#pragma unroll
    for (int m = 0; m < D / 16; ++m) vh[m][b] = load_kv<NT, u16x4>(vb + 256 * m);
  }
}

// Zeroes K rows and V entries of keys >= n or of invalid pages (the last,
// ragged tile of a request only).
template <int D>
__device__ __forceinline__ void mask_k(const int64_t (&pb)[kPagesPerTile], int j0, int n,
                                       u16x8 (&kf)[kPagesPerTile][D / 32]) {
  const int col = __lane_id() & 15;
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b) {
    const bool ok = pb[b] >= 0 && j0 + 16 * b + col < n;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) kf[b][ks] = ok ? kf[b][ks] : zero8();
  }
}

template <int D>
__device__ __forceinline__ void mask_v(const int64_t (&pb)[kPagesPerTile], int j0, int n,
                                       u16x4 (&vh)[D / 16][kPagesPerTile]) {
  const int grp = __lane_id() >> 4;
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b) {
    const int key0 = j0 + 16 * b + 4 * grp;
    const bool ok = pb[b] >= 0;
#pragma unroll
    for (int m = 0; m < D / 16; ++m)
      vh[m][b] = ok ? mask4(vh[m][b], key0, n) : u16x4{0, 0, 0, 0};
  }
}

// The call's new tokens on the split path (at most 16 query rows per
// request): keys p0 = n - s .. n - 1 come from k_new / v_new (row q0 + key -
// p0) instead of the pool, and the item that reads them also stores them to
// their pool slots for later calls; nothing waits on these stores.
//   K: a lane whose K row of page b is a new key loads its operand piece (16
//      contiguous bytes) from k_new instead of the pool, in the same load
//      instruction, and stores it to the pool address it would have read.
//   V: before the tile's pool loads, the new rows of v_new are copied to LDS
//      (direct global-to-LDS loads, no registers); once every load of the tile
//      has landed, a lane's V entries of new keys are read from there.
constexpr int kMaxNewRows = kPage;  // query rows a split item writes itself

__device__ __forceinline__ bool is_new_key(int key, const Req& R) {
  return key >= R.n - R.s && key < R.n;
}

template <int D, bool NT>
__device__ __forceinline__ void load_k_new(const Params& P, const int64_t (&pb)[kPagesPerTile],
                                           u16x8 (&kf)[kPagesPerTile][D / 32], int j0, int g,
                                           const Req& R) {
  const int lane = __lane_id(), col = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b) {
    const int key = j0 + 16 * b + col;
    const bool nk = is_new_key(key, R);
    const int64_t blk = pb[b] < 0 ? 0 : pb[b];
    const uint16_t* src =
        nk ? P.knew + ((int64_t)(R.q0 + key - (R.n - R.s)) * P.hkv + g) * D + 8 * grp
           : block_ptr<D>(P.kpool, blk) + 8 * lane;
    const int stride = nk ? 32 : 512;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) kf[b][ks] = load_kv<NT, u16x8>(src + stride * ks);
  }
}

template <int D>
__device__ __forceinline__ void store_k_new(const Params& P, const int64_t (&pb)[kPagesPerTile],
                                            const u16x8 (&kf)[kPagesPerTile][D / 32], int j0,
                                            const Req& R) {
  const int lane = __lane_id(), col = lane & 15;
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b) {
    if (is_new_key(j0 + 16 * b + col, R) && pb[b] >= 0) {
      uint16_t* dst = const_cast<uint16_t*>(P.kpool) + pb[b] * (kPage * D) + 8 * lane;
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) *reinterpret_cast<u16x8*>(dst + 512 * ks) = kf[b][ks];
    }
  }
}

// Copies rows 0 .. s - 1 of the request's v_new (KV head g) to lds[row * D]:
// 1 KB per copy instruction, the last row repeated into unused rows.
template <int D>
__device__ __forceinline__ void stage_v_new(const Params& P, uint16_t* lds, int g, const Req& R) {
  constexpr int RPI = 64 / (D / 8);  // rows per copy
  const int lane = __lane_id();
  for (int c = 0; c * RPI < R.s; ++c) {
    const int row = min(c * RPI + lane / (D / 8), R.s - 1);
    const uint16_t* src = P.vnew + ((int64_t)(R.q0 + row) * P.hkv + g) * D + 8 * (lane % (D / 8));
    lds_dma16(src, uni((int)(uintptr_t)(lds + c * RPI * D)));
  }
}

// Substitutes the new V rows into the tile's operands; with `store` also
// writes them to their pool slots.
template <int D>
__device__ __forceinline__ void apply_v_new(const Params& P, const uint16_t* lds,
                                            const int64_t (&pb)[kPagesPerTile],
                                            u16x4 (&vh)[D / 16][kPagesPerTile], int j0,
                                            const Req& R, bool store) {
  const int lane = __lane_id(), col = lane & 15, grp = lane >> 4;
  wait_vmcnt<0>();  // the staged rows (and every load of the tile) have landed
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // the page of the tile (at most one, s <= 16) whose slot 4 grp + i is a new key
    int bv = -1;
#pragma unroll
    for (int b = 0; b < kPagesPerTile; ++b) bv = is_new_key(j0 + 16 * b + 4 * grp + i, R) ? b : bv;
    if (bv >= 0) {
      const uint16_t* src = lds + (j0 + 16 * bv + 4 * grp + i - (R.n - R.s)) * D + col;
      uint16_t t[D / 16];
#pragma unroll
      for (int m = 0; m < D / 16; ++m) t[m] = src[16 * m];
#pragma unroll
      for (int b = 0; b < kPagesPerTile; ++b)
#pragma unroll
        for (int m = 0; m < D / 16; ++m) vh[m][b][i] = bv == b ? t[m] : vh[m][b][i];
      int64_t blk = -1;
#pragma unroll
      for (int b = 0; b < kPagesPerTile; ++b) blk = bv == b ? pb[b] : blk;
      if (store && blk >= 0) {
        uint16_t* dst = const_cast<uint16_t*>(P.vpool) + blk * (kPage * D) + 4 * lane + i;
#pragma unroll
        for (int m = 0; m < D / 16; ++m) dst[256 * m] = t[m];
      }
    }
  }
}

// A request whose splits 0 .. pre - 1 the shared-prefix kernel computed (a
// launch before this one) and whose last split is split pre: that split's
// items fold the earlier partial states with their own and store the rows,
// and the merge kernels leave the request alone.
__device__ __forceinline__ bool folds_prefix(const Req& R, int pre) {
  return pre >= 1 && (R.n - 1) / kSplitKeys == pre;
}

// One split item: the tiles of split k of request r, KV head g, for NA
// column blocks of 16 query-head rows, from column 16 * NA * half.  WIN: the
// handle has a sliding window.  vlds: LDS rows for the call's new V rows
// (kMaxNewRows * D bf16); the item of half 0 writes them to the pool.  pre:
// the request's leading splits computed by the shared-prefix kernel.
template <int D, int NA, bool WIN, bool NT>
__device__ __forceinline__ void split_item(const Params& P, int r, int g, int k, const Req& R,
                                           uint16_t* vlds, int half, int pre) {
  const int window = WIN ? P.window : 0;
  const int lane = __lane_id();
  const int col = lane & 15, grp = lane >> 4;
  const int ncols = R.s * P.G;
  const int MS = P.max_splits;

  int pos[NA], lo[NA];  // visible keys of the column: lo .. pos
  u16x8 qf[NA][D / 32];
  State<D> st[NA];
  const int cbase = 16 * NA * half;
#pragma unroll
  for (int nb = 0; nb < NA; ++nb) {
    const int c = cbase + nb * 16 + col;
    const bool v = c < ncols;
    pos[nb] = v ? R.n - R.s + c / P.G : -1;
    lo[nb] = window_lo(pos[nb], window);
    load_q<D>(P, qf[nb], R.q0 + (v ? c / P.G : 0), g * P.G + (v ? c % P.G : 0), v);
    state_init(st[nb]);
  }

  const int32_t* ptrow = P.pt + (int64_t)r * P.pt_stride;
  // this call's new tokens in split k, written before any of its keys is loaded
  const int kt0 = k * kTilesPerSplit;
  const int kt_end = min(kt0 + kTilesPerSplit, (R.n + kTileKeys - 1) / kTileKeys);
  // the request's first row has the smallest window start: tiles before it
  // hold no visible key for any column (identity steps), so they are skipped
  const int lo_min = window_lo(R.n - R.s, window);
  const int kt_first = max(kt0, lo_min / kTileKeys);
  int64_t pb[kPagesPerTile];
#pragma unroll
  for (int b = 0; b < kPagesPerTile; ++b)
    pb[b] = page_block(P, ptrow, kt_first * kPagesPerTile + b, R.n, g);
  // a tile holding this call's new tokens (wave-uniform)
  auto has_new = [&](int kt) { return P.fuse_write && (kt + 1) * kTileKeys > R.n - R.s; };
  u16x8 kf[kPagesPerTile][D / 32];
  bool k_issued = false;  // the tile's K loads were issued during the previous tile
  for (int kt = kt_first; kt < kt_end; ++kt) {
    const int j0 = kt * kTileKeys;
    const bool full = j0 + kTileKeys <= R.n && pb[0] >= 0 && pb[1] >= 0 && pb[2] >= 0 && pb[3] >= 0;
    u16x4 vh[D / 16][kPagesPerTile];
    const bool newtile = has_new(kt);
    if (newtile) {
      stage_v_new<D>(P, vlds, g, R);
      load_k_new<D, NT>(P, pb, kf, j0, g, R);
    } else if (!k_issued) {
      load_k<D, NT>(P, pb, kf);
    }
    // all K loads are issued before the V loads: Q.K can start on them first
    __builtin_amdgcn_sched_barrier(0);
    load_v<D, NT>(P, pb, vh);
    const int64_t pb_cur[kPagesPerTile] = {pb[0], pb[1], pb[2], pb[3]};
    // page ids of the next tile, while this tile's loads are in flight
#pragma unroll
    for (int b = 0; b < kPagesPerTile; ++b)
      pb[b] = page_block(P, ptrow, (kt + 1) * kPagesPerTile + b, R.n, g);
    if (newtile && half == 0) store_k_new<D>(P, pb_cur, kf, j0, R);
    if (!full) mask_k<D>(pb_cur, j0, R.n, kf);
    f32x4 acc[NA][kPagesPerTile];
    tile_scores<D, NA>([&](int b, int ks) { return kf[b][ks]; }, qf, acc);
    // The K registers are free: the next tile's K loads fly during this
    // tile's softmax and P.V (a tile with new tokens loads its own, after
    // this one's; it is the request's last or next to last).
    k_issued = kt + 1 < kt_end && !has_new(kt + 1);
    if (k_issued) load_k<D, NT>(P, pb, kf);
    __builtin_amdgcn_sched_barrier(0);
    if (newtile) apply_v_new<D>(P, vlds, pb_cur, vh, j0, R, half == 0);
    if (!full) mask_v<D>(pb_cur, j0, R.n, vh);
    TileWeights w[NA];
    bool open = true;  // every key of the tile visible to every column
#pragma unroll
    for (int nb = 0; nb < NA; ++nb)
      open = open && __all(pos[nb] >= j0 + kTileKeys - 1 && lo[nb] <= j0);
    if (open) {
#pragma unroll
      for (int nb = 0; nb < NA; ++nb)
        w[nb] = tile_softmax<D, false, WIN>(st[nb], acc[nb], j0, pos[nb], lo[nb], P.c);
    } else {
#pragma unroll
      for (int nb = 0; nb < NA; ++nb)
        w[nb] = tile_softmax<D, true, WIN>(st[nb], acc[nb], j0, pos[nb], lo[nb], P.c);
    }
#pragma unroll
    for (int m = 0; m < D / 16; ++m) {
      const u16x8 v0 = cat4(vh[m][0], vh[m][1]), v1 = cat4(vh[m][2], vh[m][3]);
#pragma unroll
      for (int nb = 0; nb < NA; ++nb) tile_pv_block<D>(st[nb], w[nb], m, v0, v1);
    }
#pragma unroll
    for (int nb = 0; nb < NA; ++nb) tile_commit<D>(st[nb], w[nb]);
  }

  if (request_splits(R, window) == 1) {
    // a single split: the merged state is this state; normalise and store
#pragma unroll
    for (int nb = 0; nb < NA; ++nb) {
      if (pos[nb] < 0) continue;
      const int c = cbase + nb * 16 + col;
      store_row<D>(P, st[nb].u, st[nb].m, st[nb].z, R.q0 + c / P.G, g * P.G + c % P.G);
    }
    return;
  }
  if (!WIN && k == pre && folds_prefix(R, pre)) {
    // the left fold of the merge kernels over splits 0 .. k (every row of a
    // member sees all of them), splits 0 .. k - 1 from the partial states,
    // then this item's own state; the row is stored here
#pragma unroll
    for (int nb = 0; nb < NA; ++nb) {
      if (pos[nb] < 0) continue;
      const int c = cbase + nb * 16 + col;
      const int64_t base = ((int64_t)(r * P.hkv + g) * P.ws_cols + c) * MS;
      float M = P.ws_m[base], Z = P.ws_z[base];
      f32x4 W[D / 16];
#pragma unroll
      for (int m = 0; m < D / 16; ++m)
        W[m] = *reinterpret_cast<const f32x4*>(P.ws_u + base * D + 16 * m + 4 * grp);
      for (int j = 1; j <= k; ++j) {
        float mj, zj;
        f32x4 uj[D / 16];
        if (j < k) {
          mj = P.ws_m[base + j];
          zj = P.ws_z[base + j];
#pragma unroll
          for (int m = 0; m < D / 16; ++m)
            uj[m] = *reinterpret_cast<const f32x4*>(P.ws_u + (base + j) * D + 16 * m + 4 * grp);
        } else {
          mj = st[nb].m;
          zj = st[nb].z;
#pragma unroll
          for (int m = 0; m < D / 16; ++m) uj[m] = st[nb].u[m];
        }
        const FoldScalars f = fold_scalars(M, Z, mj, zj);
#pragma unroll
        for (int m = 0; m < D / 16; ++m)
#pragma unroll
          for (int e = 0; e < 4; ++e) W[m][e] = fold_value(W[m][e], uj[m][e], f);
        M = f.M;
        Z = f.Z;
      }
      store_row<D>(P, W, M, Z, R.q0 + c / P.G, g * P.G + c % P.G);
    }
    return;
  }
  // partial state of split k for every column that has a visible key in it
#pragma unroll
  for (int nb = 0; nb < NA; ++nb) {
    const int c = cbase + nb * 16 + col;
    if (pos[nb] < 0 || k > pos[nb] / kSplitKeys || k < lo[nb] / kSplitKeys) continue;
    const int64_t pidx = ((int64_t)(r * P.hkv + g) * P.ws_cols + c) * MS + k;
    if (grp == 0) {
      P.ws_m[pidx] = st[nb].m;
      P.ws_z[pidx] = st[nb].z;
    }
    float* u = P.ws_u + pidx * D + 4 * grp;
#pragma unroll
    for (int m = 0; m < D / 16; ++m) *reinterpret_cast<f32x4*>(u + 16 * m) = st[nb].u[m];
  }
}

// Split items without a plan launch (calls of at most kInWaveMaxSeqs
// requests): every workgroup reads all requests' lengths in one round trip
// (lane l holds requests l, 64 + l, ...) and derives its own item.  Items are
// listed per KV head -- every whole 1024-key split (requests ascending, splits
// ascending), then every last partial split, longest first (tile count 16 down
// to 1, requests ascending) -- and each die (XCD: workgroup id mod the
// die count, 8 on a whole MI355X) takes a contiguous range of the list: with
// 8 KV heads and 8 dies XCD x runs head x, so a page read by several requests
// stays in one L2, and within an XCD the shortest items start last.  (When a
// launch claims its later slots from a counter, only each workgroup's first
// item comes from its die's range; the claimed slots interleave the dies.)
constexpr int kInWaveChunks = 4;
constexpr int kInWaveMaxSeqs = 64 * kInWaveChunks;
// At most this many requests on the chunk path are put in longest-first
// order by the in-wave chunk planner (a pass over them per workgroup).
constexpr int kLongestFirstReqs = 64;

struct SplitRef {
  int r, g, k, half;
  int pre;  // the request's leading splits computed by the shared-prefix kernel
  Req R;
  int per_xcd;  // items each XCD takes (slots b with b / xcds < per_xcd hold one)
};

// Inclusive prefix sum over the 64 lanes with DPP moves: shifts by 1, 2, 4
// and 8 lanes within each row of 16, then the last lane of row 0 (2) added to
// row 1 (3), and lane 31 added to rows 2 and 3.  A lane with no source adds 0.
__device__ __forceinline__ int wave_scan_dpp(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}

__device__ __forceinline__ bool inwave_split_item(const Params& P, int vb, SplitRef& out,
                                                  int* hist) {
  constexpr int C = kInWaveChunks;
  const int lane = __lane_id();
  const unsigned long long below = (1ull << lane) - 1;
  // every load first (indices clamped into [0, num_seqs)), then the arithmetic
  int cq0[C], cq1[C], cn[C], ccs[C];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int rr = min(64 * c + lane, P.num_seqs - 1);
    cq0[c] = P.cu[rr];
    cq1[c] = P.cu[rr + 1];
    cn[c] = P.ctx[rr];
    ccs[c] = P.casc ? P.casc_seq[rr] : 0;  // leading splits run by the shared-prefix kernel
  }
  // per request: whole splits nf from split kfst, the tile count cls of its
  // last partial split (0: none), and its column halves h (an item per split
  // and half: whole-split items nf * h)
  int nf[C], kfst[C], cls[C], hv[C], incl[C];
  int whole = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    nf[c] = 0;
    kfst[c] = 0;
    cls[c] = 0;
    hv[c] = 1;
    incl[c] = 0;
    if (64 * c >= P.num_seqs) continue;  // wave-uniform: no request in this chunk
    if (64 * c + lane < P.num_seqs) {
      const Req R = make_req(P, cq0[c], cq1[c], cn[c]);
      if (R.valid && R.s * P.G <= P.split_cols) {
        const int lo_min = window_lo(R.n - R.s, P.window);
        const int nfull = R.n / kSplitKeys;
        kfst[c] = max(lo_min / kSplitKeys, ccs[c]);
        nf[c] = max(0, nfull - kfst[c]);
        hv[c] = column_halves(P, R);
        if (R.n % kSplitKeys)
          cls[c] = (R.n + kTileKeys - 1) / kTileKeys -
                   max(nfull * kTilesPerSplit, lo_min / kTileKeys);
      }
    }
    incl[c] = wave_scan_dpp(nf[c] * hv[c]);
    whole += __builtin_amdgcn_readlane(incl[c], 63);
  }
  int partial = 0;
#pragma unroll
  for (int c = 0; c < C; ++c)
    partial += __popcll(__ballot(cls[c] > 0)) + __popcll(__ballot(cls[c] > 0 && hv[c] == 2));
  const int per_head = whole + partial;
  const int total = per_head * P.hkv;
  const int per_xcd = (total + P.xcds - 1) >> P.xcd_shift;
  out.per_xcd = per_xcd;
  const int jx = vb >> P.xcd_shift;
  if (jx >= per_xcd) return false;
  const int i = (vb & (P.xcds - 1)) * per_xcd + jx;
  if (i >= total) return false;
  out.g = uni(i / per_head);
  int idx = i - out.g * per_head;
  const bool is_whole = idx < whole;
  int j = -1, cj = 0, kj = 0, hj = 0;
  if (is_whole) {
    int base = 0;
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const int tot = __builtin_amdgcn_readlane(incl[c], 63);
      if (j < 0 && idx < base + tot) {
        // the first request whose inclusive item count passes idx; its items
        // are (split, half), halves adjacent
        j = __builtin_ctzll(__ballot(incl[c] > idx - base));
        cj = c;
        const int h = __builtin_amdgcn_readlane(hv[c], j);
        const int local = idx - base - __builtin_amdgcn_readlane(incl[c] - nf[c] * hv[c], j);
        kj = __builtin_amdgcn_readlane(kfst[c], j) + local / h;
        hj = local % h;
      }
      base += tot;
    }
  } else {
    idx -= whole;
    // Items of each tile count t (1 .. 16) of the last partial splits, in an
    // LDS histogram (the workgroup is this one wavefront); then lane l holds
    // the items of the classes 16 .. 16 - l (longest first), and the first lane
    // whose count passes idx names the item's class.
    if (lane <= kTilesPerSplit) hist[lane] = 0;
    __syncthreads();
#pragma unroll
    for (int c = 0; c < C; ++c)
      if (cls[c] > 0) atomicAdd(&hist[cls[c]], hv[c]);
    __syncthreads();
    const int ht = lane < kTilesPerSplit ? hist[kTilesPerSplit - lane] : 0;
    const int upto = wave_scan_dpp(ht);
    const unsigned long long past = __ballot(upto > idx);
    if (past != 0) {
      const int l = __builtin_ctzll(past);
      const int t = kTilesPerSplit - l;
      idx -= __builtin_amdgcn_readlane(upto - ht, l);  // items of the longer classes
#pragma unroll
      for (int c = 0; c < C; ++c) {
        const unsigned long long m = __ballot(cls[c] == t);
        const unsigned long long m2 = __ballot(cls[c] == t && hv[c] == 2);
        const int cnt = __popcll(m) + __popcll(m2);
        if (j < 0) {
          if (idx < cnt) {
            // the item idx of this class: requests ascending, halves adjacent
            const int before = __popcll(m & below) + __popcll(m2 & below);
            j = __builtin_ctzll(__ballot(cls[c] == t && before <= idx && idx < before + hv[c]));
            cj = c;
            hj = idx - __builtin_amdgcn_readlane(before, j);
          } else {
            idx -= cnt;
          }
        }
      }
    }
  }
  if (j < 0) return false;
  int q0 = 0, q1 = 0, n = 0, cc = 0;
#pragma unroll
  for (int c = 0; c < C; ++c)
    if (c == cj) {
      q0 = __builtin_amdgcn_readlane(cq0[c], j);
      q1 = __builtin_amdgcn_readlane(cq1[c], j);
      n = __builtin_amdgcn_readlane(cn[c], j);
      cc = __builtin_amdgcn_readlane(ccs[c], j);
    }
  out.r = uni(64 * cj + j);
  out.R = make_req(P, q0, q1, n);
  // a whole split found above, or the request's last (partial) split
  out.k = uni(is_whole ? kj : n / kSplitKeys);
  out.half = uni(hj);
  out.pre = uni(cc);
  // the item addresses only the request's own table row, rows and partial
  // states: check that it is one of the request's splits and halves
  return out.r < P.num_seqs && out.g < P.hkv && out.R.valid && out.R.s * P.G <= P.split_cols &&
         out.k >= window_lo(out.R.n - out.R.s, P.window) / kSplitKeys && out.k >= cc &&
         out.k <= (out.R.n - 1) / kSplitKeys && out.half >= 0 &&
         out.half < column_halves(P, out.R);
}

// Chunk items without a plan launch (at most kInWaveMaxSeqs requests): the
// same one-round-trip read of the lengths, and the items of the plan's chunk
// list -- per KV head, every q-tile of 128 query-head rows of every request
// on the chunk path -- with XCD-contiguous ranges.  A workgroup's run time
// grows with its last row's position, so when at most kLongestFirstReqs
// requests are on the chunk path the list takes them longest first
// (decreasing n, ties by index) and a request's q-tiles from its last: the
// blocks of a die are dispatched in that order, which keeps the longest
// items off the end of the launch.  Which workgroup computes a row never
// changes its bits.
__device__ __forceinline__ bool inwave_chunk_item(const Params& P, int& g, int& r, int& qt,
                                                  Req& R) {
  constexpr int C = kInWaveChunks;
  const int lane = __lane_id();
  int cq0[C], cq1[C], cn[C];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int rr = min(64 * c + lane, P.num_seqs - 1);
    cq0[c] = P.cu[rr];
    cq1[c] = P.cu[rr + 1];
    cn[c] = P.ctx[rr];
  }
  int cnt[C], incl[C];
  int per_head = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    cnt[c] = 0;
    incl[c] = 0;
    if (64 * c >= P.num_seqs) continue;
    if (64 * c + lane < P.num_seqs) {
      const Req Rl = make_req(P, cq0[c], cq1[c], cn[c]);
      const int ncols = Rl.s * P.G;
      if (Rl.valid && ncols > P.split_cols) cnt[c] = (ncols + kChunkCols - 1) / kChunkCols;
    }
    incl[c] = wave_scan_dpp(cnt[c]);
    per_head += __builtin_amdgcn_readlane(incl[c], 63);
  }
  const int total = per_head * P.hkv;
  const int per_xcd = (total + P.xcds - 1) >> P.xcd_shift;
  const int jx = (int)(blockIdx.x >> P.xcd_shift);
  if (jx >= per_xcd) return false;
  const int i = (int)(blockIdx.x & (P.xcds - 1)) * per_xcd + jx;
  if (i >= total) return false;
  g = uni(i / per_head);
  const int rem = i - g * per_head;
  // first q-tile of each request in the list: ro
  int ro[C];
  int nreq = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) nreq += __builtin_popcountll(__ballot(cnt[c] > 0));
  const bool longest_first = nreq <= kLongestFirstReqs;
  if (longest_first) {
#pragma unroll
    for (int c = 0; c < C; ++c) ro[c] = 0;
#pragma unroll
    for (int c2 = 0; c2 < C; ++c2) {
      uint64_t mask = __ballot(cnt[c2] > 0);
      while (mask) {
        const int l = __builtin_ctzll(mask);
        mask &= mask - 1;
        const int nl = __builtin_amdgcn_readlane(cn[c2], l);
        const int kl = __builtin_amdgcn_readlane(cnt[c2], l);
#pragma unroll
        for (int c = 0; c < C; ++c) {
          const bool before = nl > cn[c] || (nl == cn[c] && 64 * c2 + l < 64 * c + lane);
          ro[c] += before ? kl : 0;
        }
      }
    }
  } else {
    int base = 0;
#pragma unroll
    for (int c = 0; c < C; ++c) {
      ro[c] = base + incl[c] - cnt[c];
      base += __builtin_amdgcn_readlane(incl[c], 63);
    }
  }
  int j = -1, cj = 0, off = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const uint64_t hit = __ballot(cnt[c] > 0 && ro[c] <= rem && rem < ro[c] + cnt[c]);
    if (j < 0 && hit) {
      j = __builtin_ctzll(hit);
      cj = c;
      const int o = rem - __builtin_amdgcn_readlane(ro[c], j);
      off = longest_first ? __builtin_amdgcn_readlane(cnt[c], j) - 1 - o : o;
    }
  }
  if (j < 0) return false;
  int q0 = 0, q1 = 0, n = 0;
#pragma unroll
  for (int c = 0; c < C; ++c)
    if (c == cj) {
      q0 = __builtin_amdgcn_readlane(cq0[c], j);
      q1 = __builtin_amdgcn_readlane(cq1[c], j);
      n = __builtin_amdgcn_readlane(cn[c], j);
    }
  r = uni(64 * cj + j);
  qt = uni(off);
  R = make_req(P, q0, q1, n);
  const int ncols = R.s * P.G;
  return r < P.num_seqs && g < P.hkv && R.valid && ncols > P.split_cols &&
         qt < (ncols + kChunkCols - 1) / kChunkCols;
}

// The new tokens of the chunk-path requests, written by the split launch's
// last workgroups (calls of at most kInWaveMaxSeqs requests).  Unit u is
// (request, run of its new positions n - s .. n - 1 within one page, KV
// head): units are listed request by request (chunk-path requests only), runs
// ascending, KV heads fastest.  One wavefront per unit, all of its loads in
// flight together: lane l loads the 16-byte pieces q = l, l + 64, ... (row
// q / (D / 8), d from 8 (q % (D / 8))) of the run's K and V rows; K pieces are
// stored as they are; V rows go to the wavefront's LDS rows `lds` (16 x D
// bf16), from which a whole page is stored as 16-byte pieces of its V block
// (2 d x 4 slots each) and a partial run value by value.  Returns false when u
// is past the call's units.  A page id outside the pool is not written.
template <int D>
__device__ __forceinline__ bool append_unit(const Params& P, int u, uint16_t* lds) {
  constexpr int C = kInWaveChunks;
  constexpr int PPR = D / 8;                 // 16-byte pieces per row
  constexpr int NQ = kPage * PPR / 64;       // pieces per lane for a whole page
  const int lane = __lane_id();
  int cq0[C], cq1[C], cn[C];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int rr = min(64 * c + lane, P.num_seqs - 1);
    cq0[c] = P.cu[rr];
    cq1[c] = P.cu[rr + 1];
    cn[c] = P.ctx[rr];
  }
  int cnt[C], incl[C];
  int total = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    cnt[c] = 0;
    incl[c] = 0;
    if (64 * c >= P.num_seqs) continue;
    if (64 * c + lane < P.num_seqs) {
      const Req Rl = make_req(P, cq0[c], cq1[c], cn[c]);
      if (Rl.valid && Rl.s * P.G > P.split_cols)
        cnt[c] = ((Rl.n - 1) / kPage - (Rl.n - Rl.s) / kPage + 1) * P.hkv;
    }
    incl[c] = wave_scan_dpp(cnt[c]);
    total += __builtin_amdgcn_readlane(incl[c], 63);
  }
  if (u >= total) return false;
  int j = -1, cj = 0, rem = 0, base = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int tot = __builtin_amdgcn_readlane(incl[c], 63);
    if (j < 0 && u < base + tot) {
      j = __builtin_ctzll(__ballot(incl[c] > u - base));
      cj = c;
      rem = u - base - __builtin_amdgcn_readlane(incl[c] - cnt[c], j);
    }
    base += tot;
  }
  int q0 = 0, q1 = 0, n = 0;
#pragma unroll
  for (int c = 0; c < C; ++c)
    if (c == cj) {
      q0 = __builtin_amdgcn_readlane(cq0[c], j);
      q1 = __builtin_amdgcn_readlane(cq1[c], j);
      n = __builtin_amdgcn_readlane(cn[c], j);
    }
  const int r = uni(64 * cj + j);
  const Req R = make_req(P, q0, q1, n);
  const int run = uni(rem / P.hkv), h = uni(rem % P.hkv);
  const int p0 = R.n - R.s;
  const int lp = p0 / kPage + run;             // the run's logical page
  const int start = max(p0, lp * kPage), end = min(R.n, lp * kPage + kPage);
  if (!R.valid || r >= P.num_seqs || start >= end) return true;
  const int rows = end - start, slot0 = start % kPage;
  const int32_t page = P.pt[(int64_t)r * P.pt_stride + lp];
  const int64_t t0 = R.q0 + (start - p0);
  u16x8 kv[NQ], vv[NQ];
#pragma unroll
  for (int x = 0; x < NQ; ++x) {
    const int q = 64 * x + lane, i = q / PPR, dc = q % PPR;
    const int64_t src = ((t0 + i) * P.hkv + h) * D + 8 * dc;
    kv[x] = i < rows ? *reinterpret_cast<const u16x8*>(P.knew + src) : zero8();
    vv[x] = i < rows ? *reinterpret_cast<const u16x8*>(P.vnew + src) : zero8();
  }
#pragma unroll
  for (int x = 0; x < NQ; ++x) {
    const int q = 64 * x + lane;
    *reinterpret_cast<u16x8*>(lds + (q / PPR) * D + 8 * (q % PPR)) = vv[x];
  }
  lds_barrier();  // the workgroup is this one wavefront
  if (page < 0 || page >= P.num_pages) return true;
  const int64_t blk = ((int64_t)page * P.hkv + h) * (kPage * D);
  uint16_t* kpool = const_cast<uint16_t*>(P.kpool);
  uint16_t* vpool = const_cast<uint16_t*>(P.vpool);
  // K block: element (slot, d) at ((d / 8) * 16 + slot) * 8 + d % 8
#pragma unroll
  for (int x = 0; x < NQ; ++x) {
    const int q = 64 * x + lane, i = q / PPR, dc = q % PPR;
    if (i < rows) *reinterpret_cast<u16x8*>(kpool + blk + ((int64_t)dc * kPage + slot0 + i) * 8) = kv[x];
  }
  // V block: element (slot, d) at ((d / 16) * 4 + slot / 4) * 64 + (d % 16) * 4 + slot % 4;
  // its 16-byte piece e holds d = 2 (e % 8) + 16 (e / 32) and d + 1 for the
  // slots 4 ((e / 8) % 4) .. + 3
#pragma unroll
  for (int x = 0; x < NQ; ++x) {
    const int e = 64 * x + lane;
    const int d = 16 * (e / 32) + 2 * (e % 8), sg = (e / 8) % 4;
    uint32_t w[4];
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      const int i = 4 * sg + y - slot0;  // the slot's row of the run (rows past it hold zeros)
      w[y] = i >= 0 ? *reinterpret_cast<const uint32_t*>(lds + i * D + d) : 0u;
    }
    uint16_t* dst = vpool + blk + 8 * e;
    if (rows == kPage) {
      const u16x8 o = {(uint16_t)w[0], (uint16_t)w[1], (uint16_t)w[2], (uint16_t)w[3],
                       (uint16_t)(w[0] >> 16), (uint16_t)(w[1] >> 16), (uint16_t)(w[2] >> 16),
                       (uint16_t)(w[3] >> 16)};
      *reinterpret_cast<u16x8*>(dst) = o;
    } else {
#pragma unroll
      for (int y = 0; y < 4; ++y) {
        const int slot = 4 * sg + y;
        if (slot >= slot0 && slot < slot0 + rows) {
          dst[y] = (uint16_t)w[y];
          dst[4 + y] = (uint16_t)(w[y] >> 16);
        }
      }
    }
  }
  return true;
}

// One wavefront per workgroup, 16 columns per item (two wavefronts per SIMD
// at head_dim 128), or with NA = 2 (wide items) 32 columns over one read of
// each tile (one wavefront per SIMD): a finished item frees its slot at once,
// which keeps the end of the launch short when item durations vary.  The grid
// is capped at about twice the wavefronts the chip holds at once; workgroup b
// takes the slots b, b + grid, b + 2 grid, ... (the grid is a multiple of the
// dies, so its slots stay on its XCD) until one is past the items.  NT:
// K/V are streamed with non-temporal loads.
template <int D, bool WIN, bool NT, int NA>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(NA == 1 || D == 64 ? 2 : 1))) void split_kernel(Params P) {
  __shared__ __attribute__((aligned(16))) uint16_t vlds[kMaxNewRows * D];
  __shared__ int hist[kTilesPerSplit + 1];  // the planner's items per last-split tile count
  // The last append_wgs workgroups write the new tokens of the chunk-path
  // requests (units b - grid, b - grid + append_wgs, ...): dispatched after
  // every split workgroup, they run in the launch's tail, when the shortest
  // items leave the memory system room.  (Dispatched first, they delayed the
  // split items: 35 us more for the 8B mixed batch, against 11 us.)
  const int grid = (int)gridDim.x - P.append_wgs;
  if ((int)blockIdx.x >= grid) {
    for (int u = blockIdx.x - grid; append_unit<D>(P, u, vlds); u += P.append_wgs) {
    }
    return;
  }
  const int64_t slots = split_slots(P);  // work-list length
  // Slots b, then (claimed, when the call has more items than workgroups)
  // grid + 0, grid + 1, ...: a workgroup whose die the memory serves faster
  // runs more of the later items.  Claims grow, so the first claimed slot
  // past the last die range ends a workgroup's run.
  bool claims = P.inwave && P.claim != nullptr;
  auto claim = [&]() {
    int c = 0;
    if (__lane_id() == 0) c = atomicAdd(P.claim, 1);
    return grid + uni(c);
  };
  int per_xcd = 0;
  for (int vb = blockIdx.x;;) {
    int r, g, k, half, pre;
    Req R;
    if (P.inwave) {
      SplitRef it;
      const bool found = inwave_split_item(P, vb, it, hist);
      per_xcd = it.per_xcd;
      claims = claims && (per_xcd << P.xcd_shift) > grid;
      if (!found) {
        // a slot with no item: past the last die range, or (claimed slots)
        // one of the last die's unused slots, after which others follow
        if (!claims || (vb >> P.xcd_shift) >= per_xcd) return;
        vb = claim();
        continue;
      }
      r = uni(it.r);
      g = it.g;
      k = uni(it.k);
      half = it.half;
      pre = it.pre;
      R = it.R;
    } else {
      if (vb >= slots) return;
      // the slot's work-list entry: all 8 words in one scalar load, so that
      // the exit test and the item's fields cost a single round trip (the
      // list is read-only for the whole launch)
      typedef int int8v __attribute__((ext_vector_type(8)));
      const int32_t* ep = P.items + (int64_t)uni(vb) * kItemInts;
      int8v ev;
      asm volatile("s_load_dwordx8 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(ev) : "s"(ep) : "memory");
      const int4 e0 = int4{ev[0], ev[1], ev[2], ev[3]}, e1 = int4{ev[4], ev[5], ev[6], ev[7]};
      r = e0.x;
      if (r < 0) return;  // the list's valid entries come first
      g = e0.y;
      k = e0.z;
      R.n = e0.w;
      R.q0 = e1.x;
      R.s = e1.y;
      half = e1.z;
      pre = e1.w;
      R.valid = true;
    }
    split_item<D, NA, WIN, NT>(P, r, g, k, R, vlds, half, pre);
    if (claims) {
      vb = claim();
      if ((vb >> P.xcd_shift) >= per_xcd) return;
    } else {
      if (P.inwave && ((vb + grid) >> P.xcd_shift) >= per_xcd) return;  // no further slot holds an item
      vb += grid;
    }
  }
}

// Zeroes the split launch's slot counter (a kernel rather than a memset, so
// that a captured graph replays it like the launches around it).
__global__ __launch_bounds__(64) void zero_claim_kernel(int32_t* claim) {
  if (threadIdx.x == 0) *claim = 0;
}

// Rows that fold up to this many splits are merged by the short merge kernel.
constexpr int kShortMerge = 16;

// ---------------------------------------------------------------------------
// short merge (rows folding at most KS <= 16 splits: every split of the
// call's contexts, or of a sliding window): one thread per (request, KV
// head, column, 4 consecutive d), folding the partial states in ascending
// split order with fold_scalars / fold_value; KS (4, 8 or 16) sizes the
// registers for the call's split count.
// ---------------------------------------------------------------------------
template <int D, int KS>
__global__ __launch_bounds__(256) void merge_short_kernel(Params P, int cols) {
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int per_rg = cols * (D / 4);
  const int64_t rg = id / per_rg;
  if (rg >= (int64_t)P.num_seqs * P.hkv) return;
  const int rem = (int)(id % per_rg);
  const int c = rem / (D / 4), d = 4 * (rem % (D / 4));
  const int r = (int)(rg / P.hkv), g = (int)(rg % P.hkv);
  const Req R = load_req(P, r);
  if (!R.valid) return;
  const int ncols = R.s * P.G;
  if (ncols > P.split_cols || c >= ncols) return;
  if (request_splits(R, P.window) == 1) return;  // written by the split kernel
  if (P.casc && folds_prefix(R, P.casc_seq[r])) return;  // written by its last split's items
  // the row's splits: from the one holding its window start through its own
  const int pr = R.n - R.s + c / P.G;
  const int klo = window_lo(pr, P.window) / kSplitKeys;
  const int kp = pr / kSplitKeys + 1 - klo;
  const int64_t p0 = ((int64_t)(r * P.hkv + g) * P.ws_cols + c) * P.max_splits + klo;
  // every partial state is loaded first, then folded in ascending split order
  float mk[KS], zk[KS];
  f32x4 uk[KS];
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    if (k < kp) {
      mk[k] = P.ws_m[p0 + k];
      zk[k] = P.ws_z[p0 + k];
      uk[k] = *reinterpret_cast<const f32x4*>(P.ws_u + (p0 + k) * D + d);
    }
  }
  float M = mk[0], Z = zk[0];
  f32x4 W = uk[0];
#pragma unroll
  for (int k = 1; k < KS; ++k) {
    if (k < kp) {
      const FoldScalars f = fold_scalars(M, Z, mk[k], zk[k]);
#pragma unroll
      for (int i = 0; i < 4; ++i) W[i] = fold_value(W[i], uk[k][i], f);
      M = f.M;
      Z = f.Z;
    }
  }
  const float rho = final_scale(Z);
  u16x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = bf16_out(W[i] * rho);
  const int64_t row = (int64_t)(R.q0 + c / P.G) * P.hq + g * P.G + c % P.G;
  *reinterpret_cast<u16x4*>(P.out + row * D + d) = o;
  if (P.lse && d == 0) P.lse[row] = final_lse(M, Z);
}

__device__ __forceinline__ float readlane_f(float v, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

// ---------------------------------------------------------------------------
// long merge (more than 16 splits): one wavefront per (request, KV head,
// column, 64 consecutive d).  The splits are taken in chunks of 64: lane k
// loads split k's (m, z), the running maximum through every split is an exact
// prefix maximum, so both exp2 factors of every fold step are computed in
// parallel; each lane loads its d of all 64 partial U vectors at once, and the
// left fold of fold_scalars / fold_value then runs in ascending split order
// with the factors read from their lanes.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(64) void merge_long_kernel(Params P, int cols) {
  constexpr int CH = 64;
  const int64_t id = blockIdx.x;
  const int per_rg = cols * (D / 64);
  const int64_t rg = id / per_rg;
  if (rg >= (int64_t)P.num_seqs * P.hkv) return;
  const int rem = (int)(id % per_rg);
  const int c = rem / (D / 64), d = 64 * (rem % (D / 64)) + __lane_id();
  const int r = (int)(rg / P.hkv), g = (int)(rg % P.hkv);
  const int lane = __lane_id();
  const Req R = load_req(P, r);
  if (!R.valid) return;
  const int ncols = R.s * P.G;
  if (ncols > P.split_cols || c >= ncols) return;
  if (request_splits(R, P.window) == 1) return;  // written by the split kernel
  if (P.casc && folds_prefix(R, P.casc_seq[r])) return;  // written by its last split's items
  // the row's splits: from the one holding its window start through its own
  const int pr = R.n - R.s + c / P.G;
  const int klo = window_lo(pr, P.window) / kSplitKeys;
  const int kp = pr / kSplitKeys + 1 - klo;
  const int64_t p0 = ((int64_t)(r * P.hkv + g) * P.ws_cols + c) * P.max_splits + klo;
  float carry = -__builtin_inff();  // running maximum before the chunk
  float Z = 0.f, W = 0.f;
  // A chunk's loads are issued while the chunk before it is folded.  Every
  // load reads one of the row's own partial states (indices past its last
  // split are clamped to it; their values are not used), so that no load is
  // issued under a branch.
  float mk_n, zk_n, u_n[CH];
  auto load_chunk = [&](int k0) {
    mk_n = P.ws_m[p0 + min(k0 + lane, kp - 1)];
    zk_n = P.ws_z[p0 + min(k0 + lane, kp - 1)];
#pragma unroll
    for (int j = 0; j < CH; ++j) u_n[j] = P.ws_u[(p0 + min(k0 + j, kp - 1)) * D + d];
  };
  load_chunk(0);
  for (int k0 = 0; k0 < kp; k0 += CH) {
    const bool has = k0 + lane < kp;
    const float mk = has ? mk_n : -__builtin_inff();
    const float zk = has ? zk_n : 0.0f;
    float u[CH];
#pragma unroll
    for (int j = 0; j < CH; ++j) u[j] = u_n[j];
    load_chunk(k0 + CH);
    // inclusive prefix maximum over the chunk: DPP row shifts, then row broadcasts
    const int ninf = __builtin_bit_cast(int, -__builtin_inff());
    int xb = __builtin_bit_cast(int, mk);
    auto mstep = [&](int t) { xb = __builtin_bit_cast(int, fmax_(__builtin_bit_cast(float, xb), __builtin_bit_cast(float, t))); };
    mstep(__builtin_amdgcn_update_dpp(ninf, xb, 0x111, 0xf, 0xf, false));
    mstep(__builtin_amdgcn_update_dpp(ninf, xb, 0x112, 0xf, 0xf, false));
    mstep(__builtin_amdgcn_update_dpp(ninf, xb, 0x114, 0xf, 0xf, false));
    mstep(__builtin_amdgcn_update_dpp(ninf, xb, 0x118, 0xf, 0xf, false));
    mstep(__builtin_amdgcn_update_dpp(ninf, xb, 0x142, 0xa, 0xf, false));
    mstep(__builtin_amdgcn_update_dpp(ninf, xb, 0x143, 0xc, 0xf, false));
    const float pm = __builtin_bit_cast(float, xb);
    const float Mk = fmax_(carry, pm);  // M after split k0 + lane
    // M before it: lane l - 1's (wave shift right), the carry in lane 0
    const float Mp = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
        __builtin_bit_cast(int, carry), __builtin_bit_cast(int, Mk), 0x138, 0xf, 0xf, false));
    const float a = ex2(Mp - Mk), b = ex2(mk - Mk);
    // one fold step: split k0 + j (the first split of the row starts the state)
    auto step = [&](int j) {
      if (k0 + j == 0) {
        W = u[0];
        Z = readlane_f(zk, 0);
      } else {
        const float aj = readlane_f(a, j), bj = readlane_f(b, j);
        Z = Z * aj + readlane_f(zk, j) * bj;
        W = fold_value(W, u[j], FoldScalars{0.f, 0.f, aj, bj});
      }
    };
    if (k0 + CH <= kp) {
      // a whole chunk: no test between the steps
#pragma unroll
      for (int j = 0; j < CH; ++j) step(j);
    } else {
#pragma unroll
      for (int j = 0; j < CH; ++j)
        if (k0 + j < kp) step(j);
    }
    carry = readlane_f(Mk, CH - 1);
  }
  const int64_t row = (int64_t)(R.q0 + c / P.G) * P.hq + g * P.G + c % P.G;
  P.out[row * D + d] = bf16_out(W * final_scale(Z));
  if (P.lse && d == 0) P.lse[row] = final_lse(carry, Z);  // carry: the maximum over every split
}

// Issue order of a tile's LDS reads against its matrix instructions in the
// chunk and shared-prefix kernels (scheduling hints only: every accumulator's
// chain of instructions, and so every bit, is the same).  Without them the
// compiler keeps two K reads ahead of Q.K and one d-block's V reads ahead of
// P.V, and waits on each.  Q.K: four of the tile's kPagesPerTile * D / 32 K
// reads first, then one read per NB matrix instructions.  P.V: the V reads of
// two d-blocks first, then one d-block's (four reads) per d-block of matrix
// instructions (2 NB).
template <int D, int NB>
__device__ __forceinline__ void order_qk_reads() {
  constexpr int R = kPagesPerTile * (D / 32), A = 4;
  __builtin_amdgcn_sched_group_barrier(0x100, A, 0);  // DS reads
#pragma unroll
  for (int i = A; i < R; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, NB, 0);  // matrix instructions
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, NB * A, 0);
}
template <int D, int NB>
__device__ __forceinline__ void order_pv_reads() {
  constexpr int MB = D / 16;  // d-blocks, four V reads and 2 NB matrix instructions each
  __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
  for (int m = 2; m < MB; ++m) {
    __builtin_amdgcn_sched_group_barrier(0x008, 2 * NB, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 4 * NB, 0);
}

// ---------------------------------------------------------------------------
// chunk kernel: one workgroup (4 wavefronts x 32 columns) per
// (request, KV head, 128 query-head rows).  The request's K/V tiles stream
// through an LDS ring (kChunkStages tiles) filled by direct global-to-LDS
// loads: while the wavefronts compute tile t, the loads of the next tiles are
// in flight.  The splits are folded in registers as each one ends.
// ---------------------------------------------------------------------------
// Depth of the chunk kernel's LDS ring: tiles t + 1 .. t + kChunkStages - 1 are
// in flight while tile t is computed.
#ifndef VD_CHUNK_STAGES
#define VD_CHUNK_STAGES 2
#endif
constexpr int kChunkStages = VD_CHUNK_STAGES;

// Entries lp0 .. lp0 + NE - 1 of a page-table row into spid (every thread of
// a 256-thread workgroup takes part; the caller synchronises): the page id,
// or -1 for an entry at or past npages or outside the pool.  Only entries
// below npages are read.  The shared-prefix kernel stages a split's page ids
// this way, so that a tile's page lookups are LDS reads, not dependent scalar
// loads between the tile's barrier and its copies.
template <int NE>
__device__ __forceinline__ void load_pid_window(const Params& P, const int32_t* ptrow, int lp0,
                                                int npages, int32_t* spid) {
  static_assert(NE % 256 == 0 || NE < 256, "window size");
#pragma unroll
  for (int e0 = 0; e0 < NE; e0 += 256) {
    const int e = e0 + (int)threadIdx.x;
    if (NE >= 256 || e < NE) {
      const int lp = lp0 + e;
      int page = lp < npages ? ptrow[lp] : -1;
      spid[e] = (page < 0 || page >= P.num_pages) ? -1 : page;
    }
  }
}

// Two workgroups per CU (waves_per_eu 2: at most 256 registers per lane, and
// two LDS rings of kChunkStages tiles): while one wavefront of a SIMD waits on
// its softmax chain, the other issues matrix-core work.  WIN: the handle has a
// sliding window; without one every window term is the constant 0 and
// compiles away (the kernel is at its register budget).
template <int D, bool WIN>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void chunk_kernel(Params P) {
  constexpr int NB = 2;
  constexpr int BLK = kPage * D;                   // elements of one page block
  constexpr int NBLK = 2 * kPagesPerTile;          // 4 K blocks then 4 V blocks
  constexpr int TILE = NBLK * BLK;                 // elements of one staged tile
  constexpr int WCH = TILE / (4 * 512);            // 1 KB copies per wavefront per tile
  constexpr int STAGES = kChunkStages;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];  // [STAGES][NBLK][BLK]
  const int wave = uni(threadIdx.x >> 6);
  const int lane = __lane_id();
  const int col = lane & 15;
  const int window = WIN ? P.window : 0;
  // Items are ordered (KV head, request, q-tile) and blocks of one XCD (block
  // id mod the die count) take a contiguous range of them: the q-tiles of one
  // (request, KV head) share that XCD's L2, and with 8 KV heads on 8 dies each
  // XCD takes one head of every request, so long and short requests spread
  // over all XCDs.  (The in-wave planner lists the requests longest first.)
  int g, r, qt;
  Req R;
  if (P.inwave) {
    if (!inwave_chunk_item(P, g, r, qt, R)) return;
  } else {
    const int per_head = P.off_chunk[P.num_seqs];
    const int total = per_head * P.hkv;
    const int per_xcd = (total + P.xcds - 1) >> P.xcd_shift;
    const int jx = (int)(blockIdx.x >> P.xcd_shift);
    if (jx >= per_xcd) return;
    const int i = uni((int)(blockIdx.x & (P.xcds - 1)) * per_xcd + jx);
    if (i >= total) return;
    g = uni(i / per_head);
    const int rem = i - g * per_head;
    r = find_req(P.off_chunk, P.num_seqs, rem);
    R = load_req(P, r);
    qt = uni(rem - P.off_chunk[r]);
  }
  const int ncols = R.s * P.G;
  const int c0 = qt * kChunkCols;
  const int cend = min(ncols, c0 + kChunkCols);
  const int pmax = R.n - R.s + (cend - 1) / P.G;  // last position of the block

  int pos[NB], lo[NB];  // visible keys of the column: lo .. pos
  u16x8 qf[NB][D / 32];
  State<D> st[NB];
  float M[NB], Z[NB];
  f32x4 W[NB][D / 16];
  int wave_pmax = -1;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int c = c0 + wave * 32 + nb * 16 + col;
    const bool v = c < cend;
    pos[nb] = v ? R.n - R.s + c / P.G : -1;
    lo[nb] = window_lo(pos[nb], window);
    load_q<D>(P, qf[nb], R.q0 + (v ? c / P.G : 0), g * P.G + (v ? c % P.G : 0), v);
    const int cb = c0 + wave * 32 + nb * 16;
    const int clast = min(cend, cb + 16) - 1;
    if (clast >= cb) wave_pmax = max(wave_pmax, R.n - R.s + clast / P.G);
    M[nb] = 0.f;
    Z[nb] = 0.f;
#pragma unroll
    for (int m = 0; m < D / 16; ++m) W[nb][m] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int32_t* ptrow = P.pt + (int64_t)r * P.pt_stride;
  const int ntiles = pmax / kTileKeys + 1;
  // the block's first row has the smallest window start: earlier tiles hold
  // no visible key for any column of the block (identity steps)
  const int kt_first = window_lo(R.n - R.s + c0 / P.G, window) / kTileKeys;
  // this wavefront's smallest window start (its first valid column)
  const int wave_lo = window_lo(R.n - R.s + min(c0 + wave * 32, cend - 1) / P.G, window);
  const int npages = (R.n + kPage - 1) / kPage;
  // whether every page id of the request's table row lies in the pool: then
  // a tile is full (needs no masking) when it lies below n, without looking
  // its pages up again
  bool bad = false;
  for (int e = lane; e < npages; e += 64) {
    const int32_t pg = ptrow[e];
    bad = bad || pg < 0 || pg >= P.num_pages;
  }
  const bool pages_ok = !__any(bad);
  // The page blocks of tile kt (-1: past the request's pages or outside the
  // pool); a tile below the request's last page takes its 4 table entries in
  // one scalar load.
  auto tile_blocks = [&](int kt, int64_t (&pb)[kPagesPerTile]) {
    const int lp0 = kt * kPagesPerTile;
    if (lp0 + kPagesPerTile <= npages) {
      typedef __attribute__((address_space(4))) const int32_t const_i32;
      const const_i32* e = (const const_i32*)(ptrow + lp0);
      const int32_t pg[kPagesPerTile] = {e[0], e[1], e[2], e[3]};
#pragma unroll
      for (int b = 0; b < kPagesPerTile; ++b)
        pb[b] = (pg[b] < 0 || pg[b] >= P.num_pages) ? -1 : (int64_t)pg[b] * P.hkv + g;
    } else {
#pragma unroll
      for (int b = 0; b < kPagesPerTile; ++b) pb[b] = page_block(P, ptrow, lp0 + b, R.n, g);
    }
  };
  // Issues this wavefront's WCH direct loads of tile kt into stage buf: copy
  // q = wave * WCH + w moves 1 KB of page block q / (BLK / 512); a wavefront's
  // copies cover whole page blocks, whose 1 KB parts share one M0 setting.
  constexpr int SUBS = BLK / 512;  // 1 KB copies per page block
  static_assert(WCH % SUBS == 0, "whole page blocks per wavefront");
  auto fetch = [&](int kt, int buf) {
    int64_t pb[kPagesPerTile];
    tile_blocks(kt, pb);
#pragma unroll
    for (int w = 0; w < WCH; w += SUBS) {
      const int blk = (wave * WCH + w) / SUBS;
      const int b = blk % kPagesPerTile;
      const int64_t pbb = pb[b] < 0 ? 0 : pb[b];
      const uint16_t* src = block_ptr<D>(blk < kPagesPerTile ? P.kpool : P.vpool, pbb) + 8 * lane;
      const uint32_t dst = (uint32_t)(uintptr_t)(lds + (buf * NBLK + blk) * BLK);
      lds_dma16_run<SUBS>(src, uni((int)dst));
    }
  };
  // Zeroes, in stage buf, the K rows and V entries of keys >= n or of
  // invalid pages (a request's last, ragged tile only).
  auto mask_stage = [&](int kt, int buf) {
    const int j0 = kt * kTileKeys;
    bool pvalid[kPagesPerTile];
#pragma unroll
    for (int b = 0; b < kPagesPerTile; ++b)
      pvalid[b] = page_block(P, ptrow, kt * kPagesPerTile + b, R.n, g) >= 0;
    for (int ch = threadIdx.x; ch < TILE / 8; ch += 256) {
      const int blk = ch / (BLK / 8), off = (ch % (BLK / 8)) * 8;
      const int b = blk % kPagesPerTile;
      const int kbase = j0 + 16 * b;
      const bool pok = pvalid[b];
      u16x8* p = reinterpret_cast<u16x8*>(lds + (buf * NBLK + blk) * BLK + off);
      u16x8 v = *p;
      if (blk < kPagesPerTile) {
        const int slot = (off / 8) % 16;  // K block: [D/8][16][8]
        if (!pok || kbase + slot >= R.n) v = zero8();
      } else {
        const int sg = (off / 64) % 4;  // V block: [D/16][4][16][4]
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (pok && kbase + 4 * sg + (e % 4) < R.n) ? v[e] : (uint16_t)0;
      }
      *p = v;
    }
  };
  auto tile_is_full = [&](int kt) {
    if ((kt + 1) * kTileKeys > R.n) return false;
    if (pages_ok) return true;
#pragma unroll
    for (int b = 0; b < kPagesPerTile; ++b)
      if (page_block(P, ptrow, kt * kPagesPerTile + b, R.n, g) < 0) return false;
    return true;
  };

  wait_vmcnt<0>();  // the Q operands are in registers before any tile copy is issued
#pragma unroll
  for (int t = 0; t < STAGES - 1; ++t)
    if (kt_first + t < ntiles) fetch(kt_first + t, (kt_first + t) % STAGES);
  for (int kt = kt_first; kt < ntiles; ++kt) {
    const int j0 = kt * kTileKeys;
    const int k = kt / kTilesPerSplit;
    const int buf = kt % STAGES;
    // tile kt has landed once at most the later tiles' loads are outstanding
    const int later = min(STAGES - 2, ntiles - 1 - kt);
    static_assert(STAGES >= 2 && STAGES <= 5, "ring depth");
    if (later >= 3)
      wait_vmcnt<3 * WCH>();
    else if (later == 2)
      wait_vmcnt<2 * WCH>();
    else if (later == 1)
      wait_vmcnt<WCH>();
    else
      wait_vmcnt<0>();
    lds_barrier();  // every wavefront's part of tile kt is in LDS; tile kt - 1 is consumed
    if (!tile_is_full(kt)) {
      mask_stage(kt, buf);
      lds_barrier();
    }
    if (kt + STAGES - 1 < ntiles) fetch(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
    if (kt % kTilesPerSplit == 0 || kt == kt_first) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) state_init(st[nb]);
    }
    const uint16_t* T = lds + buf * NBLK * BLK;
    if (wave_pmax >= j0 && j0 + kTileKeys - 1 >= wave_lo) {
      f32x4 acc[NB][kPagesPerTile];
      // The two wavefronts of a SIMD belong to different workgroups; the one
      // issuing matrix-core work gets the higher issue priority, the other's
      // softmax fills the vector ALU around it.
      __builtin_amdgcn_s_setprio(2);
      tile_scores<D, NB>(
          [&](int b, int ks) { return *reinterpret_cast<const u16x8*>(T + b * BLK + 512 * ks + 8 * lane); },
          qf, acc);
      order_qk_reads<D, NB>();
      __builtin_amdgcn_s_setprio(0);
      TileWeights w[NB];
      bool open = true;  // every key of the tile visible to every column
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        open = open && __all(pos[nb] >= j0 + kTileKeys - 1 && lo[nb] <= j0);
      if (open) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          w[nb] = tile_softmax<D, false, WIN>(st[nb], acc[nb], j0, pos[nb], lo[nb], P.c);
      } else {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          w[nb] = tile_softmax<D, true, WIN>(st[nb], acc[nb], j0, pos[nb], lo[nb], P.c);
      }
      __builtin_amdgcn_s_setprio(2);
#pragma unroll
      for (int m = 0; m < D / 16; ++m) {
        const int o = 256 * m + 4 * lane;
        const u16x8 v0 = cat4(lds_read8<u16x4>(T + 4 * BLK + o), lds_read8<u16x4>(T + 5 * BLK + o));
        const u16x8 v1 = cat4(lds_read8<u16x4>(T + 6 * BLK + o), lds_read8<u16x4>(T + 7 * BLK + o));
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) tile_pv_block<D>(st[nb], w[nb], m, v0, v1);
      }
      order_pv_reads<D, NB>();
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) tile_commit<D>(st[nb], w[nb]);
      __builtin_amdgcn_s_setprio(0);
    }
    if (kt % kTilesPerSplit == kTilesPerSplit - 1 || kt == ntiles - 1) {
      // split k ends: fold it into the running merge for columns that have it
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        // the column's splits run from the one holding its window start
        const int klo = lo[nb] / kSplitKeys;
        if (pos[nb] < 0 || k > pos[nb] / kSplitKeys || k < klo) continue;
        if (k == klo) {
          M[nb] = st[nb].m;
          Z[nb] = st[nb].z;
#pragma unroll
          for (int m = 0; m < D / 16; ++m) W[nb][m] = st[nb].u[m];
        } else {
          const FoldScalars f = fold_scalars(M[nb], Z[nb], st[nb].m, st[nb].z);
#pragma unroll
          for (int m = 0; m < D / 16; ++m)
#pragma unroll
            for (int e = 0; e < 4; ++e) W[nb][m][e] = fold_value(W[nb][m][e], st[nb].u[m][e], f);
          M[nb] = f.M;
          Z[nb] = f.Z;
        }
      }
    }
  }

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (pos[nb] < 0) continue;
    const int c = c0 + wave * 32 + nb * 16 + col;
    store_row<D>(P, W[nb], M[nb], Z[nb], R.q0 + c / P.G, g * P.G + c % P.G);
  }
}

// Dynamic LDS bytes of the chunk kernel: kChunkStages stages of 8 page blocks.
template <int D>
constexpr size_t chunk_lds_bytes() {
  return (size_t)kChunkStages * 2 * kPagesPerTile * kPage * D * sizeof(uint16_t);
}

// ... and of the shared-prefix kernel: the same ring, then the page ids of an
// item's split.
template <int D>
constexpr size_t prefix_lds_bytes() {
  return chunk_lds_bytes<D>() + (size_t)(kSplitKeys / kPage) * sizeof(int32_t);
}

// ---------------------------------------------------------------------------
// shared-prefix kernel: one workgroup (4 wavefronts x 32 columns) per (KV
// head, listed group, 128 query-head rows of the group's query rows, shared
// split k).  Split k is read once for all these rows: its K/V tiles stream
// through the LDS ring as in the chunk kernel (page ids from the first
// member's table row, which every member shares), and each column runs the
// same per-tile operations as the split item (request, KV head, k) of its own
// request would (every key of a shared split is visible to it) and stores the
// same partial state; the merge folds it with the request's other splits.
// Rows of requests in the group's range that are not members are padding
// columns (zero queries, never stored).
// ---------------------------------------------------------------------------
// One item i of the list (per_head items per KV head); every value read from
// the list is checked before it addresses memory.  NB = 2: the item's 128
// query-head rows (32 per wavefront); NB = 1: half of them, rows 64 half ..
// 64 half + 63 (16 per wavefront).
template <int D, int NB>
__device__ __forceinline__ void prefix_item(const Params& P, int i, int half, int ngroups,
                                            int per_head, uint16_t* lds, int* scu) {
  static_assert(NB == 1 || NB == 2, "column blocks per wavefront");
  constexpr int BLK = kPage * D;
  constexpr int NBLK = 2 * kPagesPerTile;
  constexpr int TILE = NBLK * BLK;
  constexpr int WCH = TILE / (4 * 512);
  constexpr int STAGES = kChunkStages;
  const int wave = uni(threadIdx.x >> 6);
  const int lane = __lane_id();
  const int col = lane & 15, grp = lane >> 4;
  const int g = uni(i / per_head);
  const int rem = i - g * per_head;
  const int li = find_req(P.casc_off, ngroups, rem);
  const int4 gr = P.casc_grp[li];
  const int first = uni(gr.x), end = uni(gr.y), cg = uni(gr.z);
  if (first < 0 || end > P.num_seqs || end - first < 2 || cg < 1 || cg > kCascMaxSplits ||
      cg > P.max_splits)
    return;
  const int t0 = P.cu[first];
  const int x = uni(rem - P.casc_off[li]);  // (tile, split) of the group
  const int c0 = (x / cg) * kChunkCols + half * 64 * NB, k = x % cg;
  const int ncols = (P.cu[end] - t0) * P.G;
  if (c0 < 0 || c0 >= ncols) return;
  // the requests of the item's rows: consecutive, from the one holding its
  // first row (a group's requests are valid, so cu is increasing over it)
  const int r0 = first + find_req(P.cu + first, end - first, t0 + c0 / P.G);
  const int nr = min(end - r0, kChunkCols);  // the rows reach requests r0 .. r0 + nr - 1
  if ((int)threadIdx.x <= nr) scu[threadIdx.x] = P.cu[r0 + threadIdx.x];
  const int32_t* ptrow = P.pt + (int64_t)first * P.pt_stride;
  // 1024 cg <= nh: every shared page is in the first member's table row
  const int nh = (int)min<int64_t>(P.ctx[first], (int64_t)P.pt_stride * kPage);
  const int kt0 = k * kTilesPerSplit, ntiles = kTilesPerSplit;
  // the split's page ids (kSplitKeys / kPage entries from kt0's first) in LDS
  int32_t* spid = reinterpret_cast<int32_t*>(lds + STAGES * TILE);
  load_pid_window<kSplitKeys / kPage>(P, ptrow, kt0 * kPagesPerTile, (nh + kPage - 1) / kPage, spid);
  __syncthreads();

  bool live[NB];
  int64_t pidx[NB];  // the column's partial state of split k
  u16x8 qf[NB][D / 32];
  State<D> st[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int c = c0 + wave * 16 * NB + nb * 16 + col;
    bool v = c < ncols;
    int t = 0, hh = 0;
    pidx[nb] = 0;
    if (v) {
      t = t0 + c / P.G;
      hh = c % P.G;
      int lo = 0, hi = nr;  // scu[lo] <= t < scu[hi]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (scu[mid] <= t) lo = mid; else hi = mid;
      }
      const int r = r0 + lo;
      const int cl = (t - scu[lo]) * P.G + hh;  // the column's index among its request's
      // a member (its rows are on the split path), and the row is its own
      v = P.casc_seq[r] == cg && t >= scu[lo] && t < scu[lo + 1] && cl < P.ws_cols;
      pidx[nb] = ((int64_t)(r * P.hkv + g) * P.ws_cols + cl) * P.max_splits + k;
    }
    live[nb] = v;
    load_q<D>(P, qf[nb], v ? t : 0, g * P.G + (v ? hh : 0), v);
    state_init(st[nb]);
  }
  bool any_live = false;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) any_live = any_live || live[nb];
  const bool wave_live = __any(any_live);

  // the page ids of tile kt (-1: no page), one broadcast LDS read
  auto tile_pages = [&](int kt) {
    return *reinterpret_cast<const int4*>(spid + (kt - kt0) * kPagesPerTile);
  };
  // a wavefront's copies cover whole page blocks, whose 1 KB parts share one
  // M0 setting
  constexpr int SUBS = BLK / 512;
  static_assert(WCH % SUBS == 0, "whole page blocks per wavefront");
  auto fetch = [&](int kt, int buf) {
    const int4 pg = tile_pages(kt);
    const int pages[kPagesPerTile] = {pg.x, pg.y, pg.z, pg.w};
#pragma unroll
    for (int w = 0; w < WCH; w += SUBS) {
      const int blk = (wave * WCH + w) / SUBS;
      const int page = uni(pages[blk % kPagesPerTile]);
      const int64_t pbb = page < 0 ? 0 : (int64_t)page * P.hkv + g;
      const uint16_t* src = block_ptr<D>(blk < kPagesPerTile ? P.kpool : P.vpool, pbb) + 8 * lane;
      const uint32_t dst = (uint32_t)(uintptr_t)(lds + (buf * NBLK + blk) * BLK);
      lds_dma16_run<SUBS>(src, uni((int)dst));
    }
  };
  // a page id outside the pool reads as zeros, as on the split path
  auto pages_ok = [&](int kt) {
    const int4 pg = tile_pages(kt);
    return min(min(pg.x, pg.y), min(pg.z, pg.w)) >= 0;
  };
  auto zero_pages = [&](int kt, int buf) {
    const int4 pg = tile_pages(kt);
    const bool pvalid[kPagesPerTile] = {pg.x >= 0, pg.y >= 0, pg.z >= 0, pg.w >= 0};
    for (int ch = threadIdx.x; ch < TILE / 8; ch += 256) {
      const int blk = ch / (BLK / 8);
      if (!pvalid[blk % kPagesPerTile])
        *reinterpret_cast<u16x8*>(lds + (buf * NBLK + blk) * BLK + (ch % (BLK / 8)) * 8) = zero8();
    }
  };

  wait_vmcnt<0>();  // the Q operands are in registers before any tile copy is issued
#pragma unroll
  for (int t = 0; t < STAGES - 1; ++t) fetch(kt0 + t, t % STAGES);
  for (int it = 0; it < ntiles; ++it) {
    const int kt = kt0 + it;
    const int j0 = kt * kTileKeys;
    const int buf = it % STAGES;
    const int later = min(STAGES - 2, ntiles - 1 - it);
    if (later >= 3)
      wait_vmcnt<3 * WCH>();
    else if (later == 2)
      wait_vmcnt<2 * WCH>();
    else if (later == 1)
      wait_vmcnt<WCH>();
    else
      wait_vmcnt<0>();
    lds_barrier();  // every wavefront's part of tile kt is in LDS; tile kt - 1 is consumed
    if (!pages_ok(kt)) {
      zero_pages(kt, buf);
      lds_barrier();
    }
    if (it + STAGES - 1 < ntiles) fetch(kt + STAGES - 1, (it + STAGES - 1) % STAGES);
    const uint16_t* T = lds + buf * NBLK * BLK;
    if (wave_live) {
      f32x4 acc[NB][kPagesPerTile];
      tile_scores<D, NB>(
          [&](int b, int ks) { return *reinterpret_cast<const u16x8*>(T + b * BLK + 512 * ks + 8 * lane); },
          qf, acc);
      order_qk_reads<D, NB>();
      __builtin_amdgcn_sched_barrier(0);  // Q.K, the softmax and P.V are scheduled apart
      // every key of a shared split is visible to every member column
      TileWeights w[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) w[nb] = tile_softmax<D, false, false>(st[nb], acc[nb], j0, 0, 0, P.c);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int m = 0; m < D / 16; ++m) {
        const int o = 256 * m + 4 * lane;
        const u16x8 v0 = cat4(lds_read8<u16x4>(T + 4 * BLK + o), lds_read8<u16x4>(T + 5 * BLK + o));
        const u16x8 v1 = cat4(lds_read8<u16x4>(T + 6 * BLK + o), lds_read8<u16x4>(T + 7 * BLK + o));
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) tile_pv_block<D>(st[nb], w[nb], m, v0, v1);
      }
      order_pv_reads<D, NB>();
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) tile_commit<D>(st[nb], w[nb]);
    }
  }

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (!live[nb]) continue;
    if (grp == 0) {
      P.ws_m[pidx[nb]] = st[nb].m;
      P.ws_z[pidx[nb]] = st[nb].z;
    }
    float* u = P.ws_u + pidx[nb] * D + 4 * grp;
#pragma unroll
    for (int m = 0; m < D / 16; ++m) *reinterpret_cast<f32x4*>(u + 16 * m) = st[nb].u[m];
  }
}

// Items: KV head major, then listed group, then (tile, split).  Each XCD
// (workgroup id mod the die count) takes a contiguous share of the list, which its
// workgroups run in turn: the grid is sized to the chip, not to the list.  When
// the share's last round would fill at most half of the die's workgroups, each
// of its items runs as two halves of 64 query-head rows on two workgroups: the
// same per-column operations, on twice as many compute units.
template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void prefix_kernel(Params P) {
  // [STAGES][8 page blocks], then the page ids of an item's split
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  __shared__ int scu[kChunkCols + 1];  // cu of the requests an item's rows may belong to
  const int ngroups = P.casc_hdr[0], per_head = P.casc_hdr[1];
  if (ngroups < 1 || ngroups > P.num_seqs / 2 || per_head < 1 || per_head > (1 << 24)) return;
  const int total = per_head * P.hkv;
  const int per_xcd = (total + P.xcds - 1) >> P.xcd_shift;
  const int slots = (int)(gridDim.x >> P.xcd_shift);  // workgroups of a die
  const int base = (per_xcd - 1) / slots * slots;       // items before the last round
  const int last = per_xcd - base;
  const bool halve = 2 * last <= slots;
  const int entries = halve ? base + 2 * last : per_xcd;
  for (int e = (int)(blockIdx.x >> P.xcd_shift); e < entries; e += slots) {
    const bool part = halve && e >= base;
    const int j = part ? base + (e - base) / 2 : e;
    const int i = uni((int)(blockIdx.x & (P.xcds - 1)) * per_xcd + j);
    if (i >= total) break;
    if (part)
      prefix_item<D, 1>(P, i, (e - base) % 2, ngroups, per_head, lds, scu);
    else
      prefix_item<D, 2>(P, i, 0, ngroups, per_head, lds, scu);
    __syncthreads();  // LDS (ring, scu) is free for the next item
  }
}

// ---------------------------------------------------------------------------
// Opt-in check of a batch's device-side data: one wavefront per request
// writes the bit mask of the preconditions the request violates (the
// status codes of vd_attn_validate).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void validate_kernel(const int32_t* cu, const int32_t* ctx,
                                                      const int32_t* pt, int32_t pt_stride,
                                                      int64_t num_pages, int64_t T, int32_t max_q,
                                                      int32_t max_ctx, int32_t num_seqs,
                                                      int32_t* status) {
  const int r = blockIdx.x;
  if (r >= num_seqs) return;
  const int lane = __lane_id();
  const int q0 = cu[r], q1 = cu[r + 1], n = ctx[r];
  const int64_t s = (int64_t)q1 - q0;
  int st = 0;
  if (s < 1 || s > n) st |= 1;
  if (s > max_q || n > max_ctx) st |= 2;
  const int64_t npages = n > 0 ? ((int64_t)n + kPage - 1) / kPage : 0;
  if (npages > pt_stride) st |= 4;
  if (q0 < 0 || (int64_t)q1 > T) st |= 8;
  // page ids of the table entries the request reads (within its row)
  const int ne = (int)(npages < pt_stride ? npages : pt_stride);
  bool bad = false;
  for (int e = lane; e < ne; e += 64) {
    const int32_t pg = pt[(int64_t)r * pt_stride + e];
    bad = bad || pg < 0 || pg >= num_pages;
  }
  if (__any(bad)) st |= 16;
  if (lane == 0) status[r] = st;
}

// ---------------------------------------------------------------------------
// KV write: one thread per (token, KV head, 8 consecutive d)
template <int D>
__global__ __launch_bounds__(256) void kv_write_kernel(const uint16_t* knew, const uint16_t* vnew,
                                                       const int64_t* slots, int64_t ntok,
                                                       uint16_t* kpool, uint16_t* vpool,
                                                       int64_t num_pages, int hkv) {
  kv_write_one<D>(knew, vnew, slots, ntok, kpool, vpool, num_pages, hkv,
                  (int64_t)blockIdx.x * blockDim.x + threadIdx.x);
}

}  // namespace

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
struct vd_attn {
  int32_t hq, hkv, d, page_size, group;
  int32_t window;  // sliding window in keys, 0 = none
  float scale;
  float c;  // scale * log2(e) in fp32
};

namespace {

size_t round_up(size_t x) { return (x + 255) & ~(size_t)255; }


// The split launch's slot counter: an int32 of the workspace header's 256
// bytes, after the shared-prefix plan's two.
constexpr int kClaimWord = 16;

struct WsLayout {
  size_t off_full, off_part, off_chunk, casc_hdr, casc_seq, casc_off, casc_grp, items, m_off,
      z_off, u_off, total;
};

// Query-head rows per (request, KV head) that can hold split partial states:
// those of a request on the split path, at most min(max_q_len * G, 32).
int ws_cols(const vd_attn* h, int32_t max_q_len) {
  return (int)std::min<int64_t>((int64_t)std::max(max_q_len, 1) * h->group, kSplitCols);
}

// Workspace: three offset arrays of num_seqs + 1 int32, the shared-prefix
// plan (a header, one int32 per request, and per listed group -- at most
// num_seqs / 2 -- an item offset and 4 int32), the split work list (8 int32
// per (request, KV head, split, column half)), then the split partial states
// (m, z, U) for every (request, KV head, column < ws_cols, split).
WsLayout ws_layout(const vd_attn* h, int32_t num_seqs, int32_t max_q_len,
                   int32_t max_context_len) {
  const int64_t ms = ((int64_t)max_context_len + kSplitKeys - 1) / kSplitKeys;
  const int64_t n = (int64_t)num_seqs * h->hkv * ws_cols(h, max_q_len) * (ms < 1 ? 1 : ms);
  const size_t offs = round_up((size_t)(num_seqs + 1) * sizeof(int32_t));
  const size_t groups = (size_t)num_seqs / 2 + 1;
  WsLayout L;
  L.off_full = 0;
  L.off_part = offs;
  L.off_chunk = 2 * offs;
  L.casc_hdr = 3 * offs;
  L.casc_seq = L.casc_hdr + 256;
  L.casc_off = L.casc_seq + offs;
  L.casc_grp = L.casc_off + round_up((groups + 1) * sizeof(int32_t));
  L.items = L.casc_grp + round_up(groups * 4 * sizeof(int32_t));
  L.m_off = L.items + round_up((size_t)num_seqs * h->hkv * (ms < 1 ? 1 : ms) * 2 * kItemInts * sizeof(int32_t));
  L.z_off = L.m_off + round_up(n * sizeof(float));
  L.u_off = L.z_off + round_up(n * sizeof(float));
  L.total = L.u_off + round_up((size_t)n * h->d * sizeof(float));
  return L;
}

// p is a multiple of a bytes (a null pointer is).
bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int check_batch(const vd_attn* h, const vd_attn_batch* b) {
  if (!h || !b) return VD_ERR_INVALID_ARG;
  if (b->num_seqs < 0 || b->total_q_tokens < 0) return VD_ERR_INVALID_ARG;
  if (b->num_seqs == 0 || b->total_q_tokens == 0) return VD_OK;
  if (!b->q || !b->cu_q_lens || !b->context_lens || !b->page_table || !b->k_pool || !b->v_pool)
    return VD_ERR_INVALID_ARG;
  if (b->pt_stride < 1 || b->num_pages < 1 || b->max_q_len < 1 || b->max_context_len < 1)
    return VD_ERR_INVALID_ARG;
  if (b->max_q_len > b->max_context_len) return VD_ERR_INVALID_ARG;
  if (b->total_q_tokens > INT32_MAX) return VD_ERR_INVALID_ARG;
  if ((b->k_new == nullptr) != (b->v_new == nullptr)) return VD_ERR_INVALID_ARG;
  // the kernels read and write these buffers with aligned vector accesses
  // (16 bytes for bf16 data, 4 for int32 and fp32 entries)
  if (!aligned(b->q, 16) || !aligned(b->k_pool, 16) || !aligned(b->v_pool, 16) ||
      !aligned(b->k_new, 16) || !aligned(b->v_new, 16) || !aligned(b->cu_q_lens, 4) ||
      !aligned(b->context_lens, 4) || !aligned(b->page_table, 4) || !aligned(b->lse, 4))
    return VD_ERR_INVALID_ARG;
  return VD_OK;
}

// The output (16-byte aligned, like the other bf16 buffers) and the workspace
// (16-byte aligned: its fields are read and written as 16-byte vectors, and
// its offsets are multiples of 256 bytes from its start).
int check_out_ws(const void* out, bool need_out, const void* ws) {
  if (need_out && !out) return VD_ERR_INVALID_ARG;
  if (!aligned(out, 16) || !aligned(ws, 16)) return VD_ERR_INVALID_ARG;
  return VD_OK;
}

bool needs_chunks(const vd_attn* h, const vd_attn_batch* b) {
  return (int64_t)b->max_q_len * h->group > kSplitCols;
}

// The same from a call's parameters.
bool needs_chunks_params(const Params& P) { return (int64_t)P.max_q * P.G > kSplitCols; }

// Calls of at most kInWaveMaxSeqs requests need no work lists: the split and
// chunk workgroups derive their items from the lengths.
bool plans_inwave(const vd_attn_batch* b) { return b->num_seqs <= kInWaveMaxSeqs; }

// The split launch writes the call's new tokens when its workgroups plan for
// themselves and no split-path request has more than kMaxNewRows query rows
// (s * G <= 32 keeps s <= 16 for groups of two or more query heads): the
// split items those of their own requests, the launch's last workgroups
// those of the chunk-path requests.
bool fuses_write(const vd_attn* h, const vd_attn_batch* b) {
  return b->k_new != nullptr && plans_inwave(b) &&
         (h->group >= 2 || b->max_q_len <= kMaxNewRows);
}

// The shared-prefix pass runs for calls with the shared_pages hint: at most
// kCascMaxSeqs requests, no sliding window, contexts of more than one split.
bool cascades(const vd_attn* h, const vd_attn_batch* b) {
  return b->shared_pages != 0 && h->window == 0 && b->num_seqs >= 2 &&
         b->num_seqs <= kCascMaxSeqs && b->max_context_len > kSplitKeys &&
         b->total_q_tokens * h->group <= INT32_MAX;
}

// The plan launch runs for the work lists of a call with more requests, for
// new tokens the split items do not write, and for the shared-prefix plan.
bool needs_plan(const vd_attn* h, const vd_attn_batch* b) {
  return !plans_inwave(b) || (b->k_new != nullptr && !fuses_write(h, b)) || cascades(h, b);
}

int split_nb(const vd_attn* h, int32_t max_q_len) {
  return (int64_t)max_q_len * h->group <= 16 ? 1 : 2;
}

Params make_params(const vd_attn* h, const vd_attn_batch* b, void* out, const void* ws) {
  Params P;
  P.q = static_cast<const uint16_t*>(b->q);
  P.cu = b->cu_q_lens;
  P.ctx = b->context_lens;
  P.pt = b->page_table;
  P.kpool = static_cast<const uint16_t*>(b->k_pool);
  P.vpool = static_cast<const uint16_t*>(b->v_pool);
  P.out = static_cast<uint16_t*>(out);
  const WsLayout L = ws_layout(h, b->num_seqs, b->max_q_len, b->max_context_len);
  char* w = static_cast<char*>(const_cast<void*>(ws));
  P.off_full = reinterpret_cast<int32_t*>(w + L.off_full);
  P.off_part = reinterpret_cast<int32_t*>(w + L.off_part);
  P.off_chunk = reinterpret_cast<int32_t*>(w + L.off_chunk);
  P.items = reinterpret_cast<int32_t*>(w + L.items);
  P.ws_m = reinterpret_cast<float*>(w + L.m_off);
  P.ws_z = reinterpret_cast<float*>(w + L.z_off);
  P.ws_u = reinterpret_cast<float*>(w + L.u_off);
  P.T = b->total_q_tokens;
  P.num_pages = (int32_t)(b->num_pages > INT32_MAX ? INT32_MAX : b->num_pages);
  P.num_seqs = b->num_seqs;
  P.pt_stride = b->pt_stride;
  P.max_q = b->max_q_len;
  P.max_ctx = b->max_context_len;
  P.max_splits = (b->max_context_len + kSplitKeys - 1) / kSplitKeys;
  P.split_cols = 16 * split_nb(h, b->max_q_len);
  P.ws_cols = ws_cols(h, b->max_q_len);
  // wide items when every request is on the split path and some may have
  // more than 16 rows (max_q G in 17 .. 32); a call with chunk-path rows keeps
  // 16-row items, whose kernel holds two wavefronts per SIMD
  P.wide = (int64_t)b->max_q_len * h->group > 16 && (int64_t)b->max_q_len * h->group <= kSplitCols;
  P.hq = h->hq;
  P.hkv = h->hkv;
  P.G = h->group;
  const Geometry geo = device_geometry();
  P.xcds = geo.xcds;
  P.xcd_shift = geo.xcd_shift;
  P.window = h->window;
  P.c = h->c;
  P.knew = static_cast<const uint16_t*>(b->k_new);
  P.vnew = static_cast<const uint16_t*>(b->v_new);
  P.inwave = plans_inwave(b);
  P.lse = b->lse;
  P.fuse_write = fuses_write(h, b);
  P.append_wgs = 0;  // set by the split launch
  P.casc = cascades(h, b);
  P.casc_hdr = reinterpret_cast<int32_t*>(w + L.casc_hdr);
  P.casc_seq = reinterpret_cast<int32_t*>(w + L.casc_seq);
  P.casc_off = reinterpret_cast<int32_t*>(w + L.casc_off);
  P.casc_grp = reinterpret_cast<int4*>(w + L.casc_grp);
  return P;
}

int launched() { return hipGetLastError() == hipSuccess ? VD_OK : VD_ERR_LAUNCH; }



template <int D>
int run_plan(const Params& P, hipStream_t s) {
  // workgroup 0 plans (unless the workgroups plan for themselves); then one
  // wavefront per query row when the call's new tokens are written here
  const int64_t blocks = 1 + (P.knew && !P.fuse_write ? (P.T + 15) / 16 : 0);
  if (blocks > INT32_MAX) return VD_ERR_INVALID_ARG;
  hipLaunchKernelGGL((plan_kernel<D>), dim3((unsigned)blocks), dim3(1024), 0, s, P);
  return launched();
}

// Kernel launches go through hipExtLaunchKernelGGL, which records the
// optional timing events e0 / e1 with the dispatch itself.
template <int D, bool NT>
auto split_kernel_for(const Params& P) {
  // a handle's window is fixed at creation: one kernel per handle
  if (P.wide) return P.window > 0 ? &split_kernel<D, true, NT, 2> : &split_kernel<D, false, NT, 2>;
  return P.window > 0 ? &split_kernel<D, true, NT, 1> : &split_kernel<D, false, NT, 1>;
}

template <int D>
int run_splits(const Params& P0, bool stream_kv, hipStream_t s, hipEvent_t e0 = nullptr,
               hipEvent_t e1 = nullptr) {
  Params P = P0;
  // upper bound of the split items (the work-list length); a workgroup stops
  // at its first slot past the call's items.  Workgroups that plan for
  // themselves take XCD-contiguous ranges of the items (their first items
  // only, when the later ones are claimed).
  const int64_t items = split_slots(P);
  if (items > INT32_MAX - 8) return VD_ERR_INVALID_ARG;
  // at most about twice the wavefronts the chip holds at once (4 SIMDs per
  // compute unit, two wavefronts each -- one for wide items at head dim
  // 128); a multiple of the dies
  const Geometry geo = device_geometry();
  const int64_t cap = (P.wide && D == 128 ? 8 : 16) * (int64_t)geo.cus;
  const int64_t split_wgs = (std::min(items, cap) + geo.xcds - 1) / geo.xcds * geo.xcds;
  // the chunk-path requests' new tokens: a workgroup per unit up to the cap
  // (an upper bound of the units: every request's page runs number at most
  // s / 16 + 2, times the KV heads), dispatched after the split workgroups
  int64_t append = 0;
  if (P.fuse_write && needs_chunks_params(P)) {
    const int64_t units = ((P.T + kPage - 1) / kPage + 2 * (int64_t)P.num_seqs) * P.hkv;
    append = (std::min(units, cap) + geo.xcds - 1) / geo.xcds * geo.xcds;
  }
  P.append_wgs = (int)append;
  // Calls that can have more items than workgroups take the later ones from
  // a counter in the workspace header, when the items derive their own slots
  // and the K/V stream past the caches (with shared pages, each die keeps its
  // own KV head's range, whose pages stay in its L2).  The items of a request
  // and KV head: its splits from the one holding its first row's window
  // start (at most (window + s - 2) / 1024 + 2 of them), times its column
  // halves.
  const int64_t req_splits =
      P.window > 0 ? std::min<int64_t>(P.max_splits, ((int64_t)P.window + P.max_q - 2) / kSplitKeys + 2)
                   : P.max_splits;
  const int64_t item_bound = (int64_t)P.num_seqs * P.hkv * req_splits *
                             (!P.wide && (int64_t)P.max_q * P.G > 16 ? 2 : 1);
  P.claim = nullptr;
  if (P.inwave && stream_kv && !P.casc && item_bound > split_wgs) {
    P.claim = P.casc_hdr + kClaimWord;
    hipLaunchKernelGGL(zero_claim_kernel, dim3(1), dim3(64), 0, s, P.claim);
  }
  const dim3 grid((unsigned)(split_wgs + append)), block(64);
  const auto kern = stream_kv ? split_kernel_for<D, true>(P) : split_kernel_for<D, false>(P);
  hipExtLaunchKernelGGL(kern, grid, block, 0, s, e0, e1, 0, P);
  return launched();
}

template <int D>
int run_prefix(const Params& P, hipStream_t s, hipEvent_t e0 = nullptr) {
  // Two workgroups per CU, or fewer for fewer items: an upper bound of the
  // items is Hkv (ceil(T G / 128) + B / 2) tiles (the members' query rows of
  // different groups are disjoint, and a listed group has at least two
  // requests) times the shared splits, at most max_splits - 1.  A multiple
  // of the dies.
  const int64_t bound = (int64_t)P.hkv *
                        ((P.T * P.G + kChunkCols - 1) / kChunkCols + P.num_seqs / 2) *
                        std::min(kCascMaxSplits, std::max(P.max_splits - 1, 1));
  const Geometry geo = device_geometry();
  const int64_t blocks =
      (std::min<int64_t>(bound, 2 * (int64_t)geo.cus) + geo.xcds - 1) / geo.xcds * geo.xcds;
  constexpr size_t lds = prefix_lds_bytes<D>();
  static std::atomic<unsigned char> lds_set[kMaxDevices];
  if (set_lds_limit(reinterpret_cast<const void*>(&prefix_kernel<D>), (int)lds, lds_set) != hipSuccess)
    return VD_ERR_LAUNCH;
  hipExtLaunchKernelGGL((prefix_kernel<D>), dim3((unsigned)blocks), dim3(256), (uint32_t)lds, s, e0,
                        nullptr, 0, P);
  return launched();
}

// The splits phase: the shared-prefix kernel (calls with the shared_pages
// hint), then the split kernel; e0 / e1 are recorded by the first and the last
// launch.
template <int D>
int run_split_phase(const Params& P, bool stream_kv, hipStream_t s, hipEvent_t e0 = nullptr,
                    hipEvent_t e1 = nullptr) {
  if (P.casc) {
    const int rc = run_prefix<D>(P, s, e0);
    if (rc != VD_OK) return rc;
    return run_splits<D>(P, stream_kv, s, nullptr, e1);
  }
  return run_splits<D>(P, stream_kv, s, e0, e1);
}

template <int D>
int run_merge(const Params& P, hipStream_t s) {
  const int64_t cols = P.ws_cols;  // = min(max_q * G, split_cols)
  // the most splits a row folds: every split through the longest context, or
  // with a window of w keys the splits from the one holding p - w + 1 to the
  // one holding p, at most floor((w - 1) / 1024) + 2
  const int fold = P.window > 0 ? std::min(P.max_splits, (P.window - 1) / kSplitKeys + 2)
                                : P.max_splits;
  if (fold <= kShortMerge) {
    const int64_t threads = (int64_t)P.num_seqs * P.hkv * cols * (D / 4);
    const int64_t blocks = (threads + 255) / 256;
    if (blocks > INT32_MAX) return VD_ERR_INVALID_ARG;
    // registers for the rows' split count: 4, 8 or 16 partial states
    const auto kern = fold <= 4   ? &merge_short_kernel<D, 4>
                      : fold <= 8 ? &merge_short_kernel<D, 8>
                                  : &merge_short_kernel<D, 16>;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), 0, s, P, (int)cols);
    return launched();
  }
  const int64_t blocks = (int64_t)P.num_seqs * P.hkv * cols * (D / 64);
  if (blocks > INT32_MAX) return VD_ERR_INVALID_ARG;
  hipLaunchKernelGGL((merge_long_kernel<D>), dim3((unsigned)blocks), dim3(64), 0, s, P, (int)cols);
  return launched();
}

template <int D>
int run_chunks(const Params& P, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr) {
  // upper bound of sum_r Hkv * ceil(s_r G / 128) <= Hkv (ceil(T G / 128) + B),
  // rounded up to a multiple of the dies
  int64_t blocks = (int64_t)P.hkv * ((P.T * P.G + kChunkCols - 1) / kChunkCols + P.num_seqs);
  blocks = (blocks + P.xcds - 1) / P.xcds * P.xcds;
  if (blocks > INT32_MAX) return VD_ERR_INVALID_ARG;
  constexpr size_t lds = chunk_lds_bytes<D>();
  // a handle's window is fixed at creation: one kernel per handle
  const auto kern = P.window > 0 ? &chunk_kernel<D, true> : &chunk_kernel<D, false>;
  static std::atomic<unsigned char> lds_set[2][kMaxDevices];
  if (set_lds_limit(reinterpret_cast<const void*>(kern), (int)lds, lds_set[P.window > 0]) != hipSuccess)
    return VD_ERR_LAUNCH;
  hipExtLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), (uint32_t)lds, s, e0, e1, 0, P);
  return launched();
}

// The workspace of vd_attn_forward_noalloc, for callers that cannot allocate:
// the library's own device array, one copy on every device the library runs
// on, held until the process ends.  On the host, `scratch` names a stand-in,
// not device memory: host code uses only the address scratch_address()
// obtains for the current device.
static_assert(VD_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size");
static __device__ __align__(256) unsigned char scratch[VD_NOALLOC_SCRATCH_BYTES];

// The current device's copy of `scratch` (hipGetSymbolAddress with the device
// current, once per device), or nullptr when it cannot be had.
void* scratch_address() {
  static std::atomic<void*> addr[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void* p = addr[dev].load(std::memory_order_acquire);
  if (p) return p;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
  addr[dev].store(p, std::memory_order_release);
  return p;
}

bool ws_ok(const vd_attn* h, const vd_attn_batch* b, const void* ws, size_t bytes) {
  return ws && bytes >= ws_layout(h, b->num_seqs, b->max_q_len, b->max_context_len).total;
}

}  // namespace

extern "C" {

int vd_attn_create(const vd_attn_desc* desc, vd_attn** out) {
  if (out) *out = nullptr;
  if (!desc || !out) return VD_ERR_INVALID_ARG;
  if (desc->abi_version != VD_ABI_VERSION) return VD_ERR_INVALID_ARG;
  if (desc->num_q_heads < 1 || desc->num_kv_heads < 1 || desc->head_dim < 1 ||
      desc->page_size < 1)
    return VD_ERR_INVALID_ARG;
  if (!(desc->softmax_scale == desc->softmax_scale)) return VD_ERR_INVALID_ARG;  // NaN
  if (desc->window < 0) return VD_ERR_INVALID_ARG;
  if (desc->dtype != VD_DTYPE_BF16) return VD_ERR_UNSUPPORTED;
  if (desc->head_dim != 64 && desc->head_dim != 128) return VD_ERR_UNSUPPORTED;
  if (desc->page_size != kPage) return VD_ERR_UNSUPPORTED;
  if (desc->num_q_heads % desc->num_kv_heads != 0) return VD_ERR_UNSUPPORTED;
  if (desc->num_q_heads / desc->num_kv_heads > kSplitCols) return VD_ERR_UNSUPPORTED;
  vd_attn* h = new (std::nothrow) vd_attn;
  if (!h) return VD_ERR_INVALID_ARG;
  h->hq = desc->num_q_heads;
  h->hkv = desc->num_kv_heads;
  h->d = desc->head_dim;
  h->page_size = desc->page_size;
  h->group = desc->num_q_heads / desc->num_kv_heads;
  h->window = desc->window;
  const double scale = desc->softmax_scale > 0.0f ? (double)desc->softmax_scale
                                                  : 1.0 / std::sqrt((double)desc->head_dim);
  h->scale = (float)scale;
  h->c = (float)(scale * 1.4426950408889634073599246810019);  // log2(e)
  *out = h;
  return VD_OK;
}

void vd_attn_destroy(vd_attn* h) { delete h; }

int vd_attn_workspace_size(const vd_attn* h, int32_t num_seqs, int32_t max_q_len,
                           int32_t max_context_len, size_t* bytes) {
  if (!h || !bytes || num_seqs < 0 || max_q_len < 0 || max_context_len < 0)
    return VD_ERR_INVALID_ARG;
  *bytes = ws_layout(h, num_seqs, max_q_len, max_context_len).total;
  return VD_OK;
}

int vd_attn_forward_plan(const vd_attn* h, const vd_attn_batch* b, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  int rc = check_batch(h, b);
  if (rc != VD_OK || b->num_seqs == 0 || b->total_q_tokens == 0) return rc;
  if ((rc = check_out_ws(nullptr, false, workspace)) != VD_OK) return rc;
  if (!ws_ok(h, b, workspace, workspace_bytes)) return VD_ERR_WORKSPACE;
  if (!needs_plan(h, b)) return VD_OK;  // the split workgroups plan for themselves
  const Params P = make_params(h, b, nullptr, workspace);
  return h->d == 64 ? run_plan<64>(P, stream) : run_plan<128>(P, stream);
}

int vd_attn_forward_splits(const vd_attn* h, const vd_attn_batch* b, void* out, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  int rc = check_batch(h, b);
  if (rc != VD_OK || b->num_seqs == 0 || b->total_q_tokens == 0) return rc;
  if ((rc = check_out_ws(out, true, workspace)) != VD_OK) return rc;
  if (!ws_ok(h, b, workspace, workspace_bytes)) return VD_ERR_WORKSPACE;
  const Params P = make_params(h, b, out, workspace);
  // with the shared-prefix pass, the shared splits are read (cached) by the
  // shared-prefix kernel and the split items stream the requests' own pages
  const bool nt = b->shared_pages == 0 || P.casc;
  return h->d == 64 ? run_split_phase<64>(P, nt, stream) : run_split_phase<128>(P, nt, stream);
}

int vd_attn_forward_chunks(const vd_attn* h, const vd_attn_batch* b, void* out,
                           const void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int rc = check_batch(h, b);
  if (rc != VD_OK || b->num_seqs == 0 || b->total_q_tokens == 0) return rc;
  if ((rc = check_out_ws(out, true, workspace)) != VD_OK) return rc;
  if (!ws_ok(h, b, workspace, workspace_bytes)) return VD_ERR_WORKSPACE;
  if (!needs_chunks(h, b)) return VD_OK;
  const Params P = make_params(h, b, out, workspace);
  return h->d == 64 ? run_chunks<64>(P, stream) : run_chunks<128>(P, stream);
}

// Events of a phase that launches nothing: recorded back to back.
static int record_pair(hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (e0 && hipEventRecord(e0, s) != hipSuccess) return VD_ERR_LAUNCH;
  if (e1 && hipEventRecord(e1, s) != hipSuccess) return VD_ERR_LAUNCH;
  return VD_OK;
}

int vd_attn_forward_splits_timed(const vd_attn* h, const vd_attn_batch* b, void* out,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream,
                                 hipEvent_t start, hipEvent_t stop) {
  int rc = check_batch(h, b);
  if (rc != VD_OK) return rc;
  if (b->num_seqs == 0 || b->total_q_tokens == 0) return record_pair(stream, start, stop);
  if ((rc = check_out_ws(out, true, workspace)) != VD_OK) return rc;
  if (!ws_ok(h, b, workspace, workspace_bytes)) return VD_ERR_WORKSPACE;
  const Params P = make_params(h, b, out, workspace);
  // with the shared-prefix pass, the shared splits are read (cached) by the
  // shared-prefix kernel and the split items stream the requests' own pages
  const bool nt = b->shared_pages == 0 || P.casc;
  return h->d == 64 ? run_split_phase<64>(P, nt, stream, start, stop)
                    : run_split_phase<128>(P, nt, stream, start, stop);
}

int vd_attn_forward_chunks_timed(const vd_attn* h, const vd_attn_batch* b, void* out,
                                 const void* workspace, size_t workspace_bytes,
                                 hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
  int rc = check_batch(h, b);
  if (rc != VD_OK) return rc;
  if (b->num_seqs == 0 || b->total_q_tokens == 0) return record_pair(stream, start, stop);
  if ((rc = check_out_ws(out, true, workspace)) != VD_OK) return rc;
  if (!ws_ok(h, b, workspace, workspace_bytes)) return VD_ERR_WORKSPACE;
  if (!needs_chunks(h, b)) return record_pair(stream, start, stop);
  const Params P = make_params(h, b, out, workspace);
  return h->d == 64 ? run_chunks<64>(P, stream, start, stop)
                    : run_chunks<128>(P, stream, start, stop);
}

int vd_attn_forward_merge(const vd_attn* h, const vd_attn_batch* b, void* out,
                          const void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int rc = check_batch(h, b);
  if (rc != VD_OK || b->num_seqs == 0 || b->total_q_tokens == 0) return rc;
  if ((rc = check_out_ws(out, true, workspace)) != VD_OK) return rc;
  if (!ws_ok(h, b, workspace, workspace_bytes)) return VD_ERR_WORKSPACE;
  const Params P = make_params(h, b, out, workspace);
  return h->d == 64 ? run_merge<64>(P, stream) : run_merge<128>(P, stream);
}

int vd_attn_forward(const vd_attn* h, const vd_attn_batch* b, void* out, void* workspace,
                    size_t workspace_bytes, hipStream_t stream) {
  int rc = check_batch(h, b);
  if (rc != VD_OK || b->num_seqs == 0 || b->total_q_tokens == 0) return rc;
  if ((rc = check_out_ws(out, true, workspace)) != VD_OK) return rc;
  if (!ws_ok(h, b, workspace, workspace_bytes)) return VD_ERR_WORKSPACE;
  rc = vd_attn_forward_plan(h, b, workspace, workspace_bytes, stream);
  if (rc != VD_OK) return rc;
  rc = vd_attn_forward_splits(h, b, out, workspace, workspace_bytes, stream);
  if (rc != VD_OK) return rc;
  rc = vd_attn_forward_chunks(h, b, out, workspace, workspace_bytes, stream);
  if (rc != VD_OK) return rc;
  return vd_attn_forward_merge(h, b, out, workspace, workspace_bytes, stream);
}

int vd_attn_forward_noalloc(const vd_attn* h, const vd_attn_batch* b, void* out,
                            hipStream_t stream) {
  int rc = check_batch(h, b);
  if (rc != VD_OK || b->num_seqs == 0 || b->total_q_tokens == 0) return rc;
  if ((rc = check_out_ws(out, true, nullptr)) != VD_OK) return rc;
  if (ws_layout(h, b->num_seqs, b->max_q_len, b->max_context_len).total > VD_NOALLOC_SCRATCH_BYTES)
    return VD_ERR_WORKSPACE;
  void* ws = scratch_address();
  if (!ws) return VD_ERR_LAUNCH;
  // the same phases as vd_attn_forward; nothing in them allocates
  return vd_attn_forward(h, b, out, ws, VD_NOALLOC_SCRATCH_BYTES, stream);
}

int vd_attn_validate(const vd_attn* h, const vd_attn_batch* b, int32_t* status,
                     hipStream_t stream) {
  int rc = check_batch(h, b);
  if (rc != VD_OK || b->num_seqs == 0) return rc;
  if (!status || !b->cu_q_lens || !b->context_lens || !b->page_table || b->pt_stride < 1 ||
      !aligned(status, 4))
    return VD_ERR_INVALID_ARG;
  hipLaunchKernelGGL(validate_kernel, dim3((unsigned)b->num_seqs), dim3(64), 0, stream,
                     b->cu_q_lens, b->context_lens, b->page_table, b->pt_stride, b->num_pages,
                     b->total_q_tokens, b->max_q_len, b->max_context_len, b->num_seqs, status);
  return launched();
}

int vd_pool_bytes(const vd_attn* h, int64_t num_pages, size_t* bytes) {
  if (!h || !bytes || num_pages < 0) return VD_ERR_INVALID_ARG;
  *bytes = (size_t)num_pages * h->hkv * kPage * h->d * sizeof(uint16_t);
  return VD_OK;
}

int vd_kv_write(const vd_attn* h, const void* k_new, const void* v_new,
                const int64_t* slot_mapping, int64_t num_tokens, void* k_pool, void* v_pool,
                int64_t num_pages, hipStream_t stream) {
  if (!h || num_tokens < 0 || num_pages < 0) return VD_ERR_INVALID_ARG;
  if (num_tokens == 0) return VD_OK;
  if (!k_new || !v_new || !slot_mapping || !k_pool || !v_pool) return VD_ERR_INVALID_ARG;
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(slot_mapping, 8) ||
      !aligned(k_pool, 16) || !aligned(v_pool, 16))
    return VD_ERR_INVALID_ARG;
  const int64_t threads = num_tokens * h->hkv * (h->d / 8);
  const dim3 grid((unsigned)((threads + 255) / 256)), block(256);
  const uint16_t* kn = static_cast<const uint16_t*>(k_new);
  const uint16_t* vn = static_cast<const uint16_t*>(v_new);
  uint16_t* kp = static_cast<uint16_t*>(k_pool);
  uint16_t* vp = static_cast<uint16_t*>(v_pool);
  if (h->d == 64)
    hipLaunchKernelGGL((kv_write_kernel<64>), grid, block, 0, stream, kn, vn, slot_mapping,
                       num_tokens, kp, vp, num_pages, h->hkv);
  else
    hipLaunchKernelGGL((kv_write_kernel<128>), grid, block, 0, stream, kn, vn, slot_mapping,
                       num_tokens, kp, vp, num_pages, h->hkv);
  return launched();
}

const char* vd_status_string(int status) {
  switch (status) {
    case VD_OK: return "ok";
    case VD_ERR_INVALID_ARG: return "invalid argument";
    case VD_ERR_UNSUPPORTED: return "unsupported configuration";
    case VD_ERR_WORKSPACE: return "workspace missing or too small";
    case VD_ERR_LAUNCH: return "kernel launch failed";
    default: return "unknown status";
  }
}

int vd_attn_tiling(const vd_attn* h, int32_t* tile_keys, int32_t* split_keys, int32_t* page_size) {
  if (!h) return VD_ERR_INVALID_ARG;
  if (tile_keys) *tile_keys = kTileKeys;
  if (split_keys) *split_keys = kSplitKeys;
  if (page_size) *page_size = kPage;
  return VD_OK;
}

}  // extern "C"
