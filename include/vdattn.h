/*
 * vdattn.h -- batch-invariant paged causal attention for AMD MI355X (gfx950).
 *
 * C ABI of libvdattn.so.  Plain pointers and sizes only.
 *
 * What the library computes
 * -------------------------
 * The paper's problem statement (Appendix A.1, "Properties and Logical
 * Inputs") and causal contract (Section 5.3): an invocation packs the query
 * rows of num_seqs requests.  Request r has query length s_r and key length
 * n_r with 0 < s_r <= n_r; its query row i (0 <= i < s_r) stands for logical
 * position p = n_r - s_r + i.  Logical keys and values are read through the
 * request's page table pi_r: K[j] = Kphys[pi_r(floor(j / P)), slot j mod P].
 * Query head h reads KV head floor(h / (Hq / Hkv)).  The output row is softmax
 * attention of the query over keys 0..p (causal prefix), computed with the
 * tiled online-softmax update of Appendix A.2 ("A Simplified Tile IR") in
 * fp32 with bf16 inputs and a bf16 output.
 *
 * Guarantee (the causal contract of Section 5.3 / Appendix A.1): the output
 * bits of a row depend only on (p, the row's query, K/V at positions 0..p,
 * the handle); with a sliding window of w keys (Appendix A.5), only on K/V
 * at positions max(0, p - w + 1)..p.  They do not depend on s_r, n_r, the row index, the other
 * requests of the call, their order, the page table (physical placement,
 * stride, sharing of pages between requests), num_pages, the hints, the
 * workspace contents or the stream.  Keys are processed in tiles of 64
 * logical positions and in splits of 1024 logical positions whose partial
 * states are merged in ascending split order; both sizes are fixed by the
 * handle, never by the batch.
 *
 * Ownership and threading
 * -----------------------
 * Every buffer is caller-owned device memory (except the descriptor and the
 * hints, which are host values).  The library never allocates or frees
 * device memory, never synchronises the device, and keeps no mutable global
 * state.  A handle is immutable after creation and may be used from several
 * host threads and streams at once; concurrent calls must not share a
 * workspace.
 *
 * Errors
 * ------
 * Every entry point returns VD_OK (0) or a negative vd_status.  Arguments the
 * host can see are checked before anything is launched; on such an error no
 * output is touched.  Among them, alignment (VD_ERR_INVALID_ARG otherwise):
 * the bf16 buffers (q, k_pool, v_pool, k_new, v_new, the output) and the
 * workspace start at a multiple of 16 bytes, the int32 and fp32 arrays
 * (cu_q_lens, context_lens, page_table, lse, a validator's status) at a
 * multiple of 4, vd_kv_write's slot_mapping at a multiple of 8; the kernels
 * access them with aligned vector loads and stores.  Device-side data
 * (lengths, page ids) is not read by the host; the kernels never access
 * memory outside the buffers described below:
 * a request whose lengths violate 0 < s <= n, whose page count exceeds the
 * table stride, whose lengths exceed the hints, or whose rows fall outside
 * total_q_tokens is skipped (its output rows are left unwritten), and a page
 * id outside [0, num_pages) reads as zeros.
 */
#ifndef VDATTN_H
#define VDATTN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VD_ABI_VERSION 4

typedef enum {
  VD_OK = 0,
  VD_ERR_INVALID_ARG = -1, /* null pointer, negative or oversized size, bad descriptor field */
  VD_ERR_UNSUPPORTED = -2, /* head_dim not in {64, 128}, page_size != 16, dtype != bf16,
                              Hq not a multiple of Hkv, group size > 32; the paper's
                              "reject a missing configuration" (Section 1) */
  VD_ERR_WORKSPACE = -3,   /* workspace missing or smaller than vd_attn_workspace_size */
  VD_ERR_LAUNCH = -4       /* a kernel launch failed (hipGetLastError) */
} vd_status;

#define VD_DTYPE_BF16 1

/* Fixed per-model configuration, bound once (Section 4.1, "Fixed kernel
 * choices": tiles and specialisations are chosen at initialisation and never
 * from the batch). */
typedef struct {
  int32_t abi_version;  /* VD_ABI_VERSION */
  int32_t num_q_heads;  /* Hq  >= 1 */
  int32_t num_kv_heads; /* Hkv >= 1, divides Hq, Hq / Hkv <= 32 */
  int32_t head_dim;     /* D in {64, 128} */
  int32_t page_size;    /* P, must be 16 */
  int32_t dtype;        /* VD_DTYPE_BF16: Q, K, V and the output are bf16 */
  float softmax_scale;  /* <= 0 selects 1 / sqrt(head_dim) */
  int32_t window;       /* sliding-window attention (Appendix A.5, "Relational Alignment and
                           Composition"): w > 0 restricts the row at position p to the keys
                           p - w < j <= p; 0 selects the full causal prefix.  Like the scale,
                           it is fixed by the handle (a model's layer), never by the batch */
} vd_attn_desc;

typedef struct vd_attn vd_attn; /* opaque, immutable after creation */

/* Creates a handle.  *out receives it on success (and NULL on error). */
int vd_attn_create(const vd_attn_desc* desc, vd_attn** out);

/* Destroys a handle (NULL is accepted). */
void vd_attn_destroy(vd_attn* h);

/* One call's packed inputs.  Pointers are device memory unless noted. */
typedef struct {
  int32_t num_seqs;             /* B >= 0 */
  int64_t total_q_tokens;       /* T = cu_q_lens[B] >= 0 */
  const void* q;                /* [T, Hq, D] bf16, rows packed by request, i ascending */
  const int32_t* cu_q_lens;     /* [B + 1], cu[0] = 0, s_r = cu[r + 1] - cu[r] */
  const int32_t* context_lens;  /* [B], n_r (counts this call's own query tokens) */
  const int32_t* page_table;    /* [B * pt_stride]; entries 0 .. ceil(n_r / 16) - 1 of row r used */
  int32_t pt_stride;            /* >= 1 */
  const void* k_pool;           /* pools in the library layout (see vd_kv_write), */
  const void* v_pool;           /*   num_pages pages of Hkv page blocks each */
  int64_t num_pages;            /* >= 1 */
  int32_t max_q_len;            /* HOST hint: >= every s_r (launch sizing only) */
  int32_t max_context_len;      /* HOST hint: >= every n_r (launch sizing only) */
  /* Optional (NULL: none): the K and V of the call's own query rows, each [T, Hkv, D] bf16,
   * row t belonging to query row t.  Before any key is read, row t is written into the pool
   * at the slot that its logical position p has in its request's page table (the engine
   * writes new tokens to their private slots before attention reads them, Section 4.1:
   * append + attend in one call).  Rows of a skipped request, or whose page id is outside
   * [0, num_pages), are not written.  Two requests of one call must not hold the same slot
   * for their query rows, and no request of the call may read another request's query-row
   * slot as a key (the slots of new tokens are private, Section 4.1). */
  const void* k_new;
  const void* v_new;
  /* HOST hint, never value-relevant: nonzero when some pages are read by several requests
   * of the call (a shared prefix, Section 4.1's prefix cache).  It turns on the shared-prefix
   * pass: the plan launch compares the page tables of adjacent requests and finds groups of
   * requests whose tables start with the same pages (requests r - 1 and r share 1024-key
   * split k when their entries of splits 0 .. k are equal; a group shares the splits all its
   * neighbours share, at most 32).  Each shared split is then read once for the query rows
   * of every member (a request of the group with s_r * (Hq / Hkv) <= 32 whose rows all lie
   * past the shared splits), with the same operations per row as the request's own split
   * item, so the output bits do not change; the rest of each request's splits are read by
   * its own split items.  Not with a sliding window, nor for more than 1024 requests.
   * Zero: every split is read by its request's items, K/V streamed past the caches with
   * non-temporal loads (the faster choice when each page is read once). */
  int32_t shared_pages;
  /* Optional output (NULL: not written): [T, Hq] fp32, row t's log-sum-exp in natural log,
   * ln sum_j exp(scale * q.k_j) over the keys the row sees.  The tile update of Appendix A.2
   * carries it as the state (m, z); the paper does not export it.  It is what a caller needs
   * to merge this attention with attention over other keys, and it is bit-invariant like
   * the output (it depends only on the row's final (m, z)). */
  float* lse;
} vd_attn_batch;

/* Bytes of workspace one call needs for the given host-side sizes: the plan
 * (int32 arrays of about 3 num_seqs, the shared-prefix list, the split work
 * list and the split launch's slot counter) and, for every (request, KV head, query-head row < min(max_q_len *
 * Hq / Hkv, 32), 1024-key split < ceil(max_context_len / 1024)), a partial
 * state of head_dim + 2 floats. */
int vd_attn_workspace_size(const vd_attn* h, int32_t num_seqs, int32_t max_q_len,
                           int32_t max_context_len, size_t* bytes);

/* Paged causal attention for every row of the batch (Appendix A.2 update,
 * Section 5.3 contract).  `out` is device [T, Hq, D] bf16.  The K/V of this
 * call's own tokens must be in the pool (vd_kv_write) or be handed over in
 * k_new / v_new.  The workspace holds the plan and the split partial states;
 * its prior contents do not matter.  Launches on `stream` and returns without
 * waiting. */
int vd_attn_forward(const vd_attn* h, const vd_attn_batch* batch, void* out, void* workspace,
                    size_t workspace_bytes, hipStream_t stream);

/* vd_attn_forward without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same launches, same output bits; the
 * workspace is the library's own static device array of
 * VD_NOALLOC_SCRATCH_BYTES (128 MiB), one on every device the library runs
 * on, held until the process ends.  A call whose vd_attn_workspace_size
 * exceeds it returns VD_ERR_WORKSPACE before any launch (e.g. 64 requests of
 * up to 4,096 keys need 4 MB; 8 of up to 131,072 keys 17 MB; a call with prefill
 * rows or 4-token verify rows of a group of 8 query heads needs 32 partial
 * states per (request, KV head, 1024-key split): 256 such requests of up to
 * 2,560 keys 102 MB).  It allocates nothing and calls no allocating routine.
 * Every call on one device uses that device's one array, which keeps the last
 * call's contents (no call reads what it did not write first): calls that may
 * overlap on one device -- other streams, other threads -- race, and the
 * caller must order them; calls on one stream are ordered by the stream. */
#define VD_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
int vd_attn_forward_noalloc(const vd_attn* h, const vd_attn_batch* batch, void* out,
                            hipStream_t stream);

/* The four phases vd_attn_forward runs, in this order, for callers that time
 * or schedule them separately (same batch, same output, same stream, same
 * workspace; their composition is bit-identical to vd_attn_forward):
 *   plan:   only for calls with more than 256 requests, with k_new / v_new
 *           that the split launch does not write (Hq / Hkv = 1 and
 *           max_q_len > 16), or with the shared_pages hint; otherwise it
 *           launches nothing.  Writes k_new / v_new into the pool (when the
 *           split launch does not) and, reading the per-request lengths and
 *           page tables on the device, the work lists of the split and
 *           shared-prefix phases into the workspace (no device-to-host
 *           synchronisation);
 *   splits: rows of requests with s_r * (Hq / Hkv) <= 32 -- one work item
 *           per (request, KV head, 1024-key split, 16 query-head rows; 32 in
 *           a call whose max_q_len * (Hq / Hkv) is 17..32), after
 *           the shared-prefix items (shared_pages hint) -- one per (group, KV
 *           head, 128 query-head rows of its members, shared split).  Without
 *           a plan launch, every workgroup derives its items from the lengths
 *           and the call's new tokens are written by this launch: the items
 *           write their own requests' rows, and further workgroups, after
 *           the items', those of the requests of the chunks phase.  When the
 *           call can have more items than the launch has workgroups (and its
 *           K/V stream past the caches: no shared_pages hint), a one-wavefront
 *           launch first zeroes a counter in the workspace, from which the
 *           workgroups claim the items past their first.  A request with one
 *           split writes its output rows directly; otherwise each item writes
 *           a partial state;
 *   chunks: rows of requests with s_r * (Hq / Hkv) > 32 -- one work item per
 *           (request, KV head, 128 query-head rows); folds the splits in
 *           registers and writes their output rows;
 *   merge:  folds the partial states of the split-phase rows of requests
 *           with more than one split, in ascending split order, and writes
 *           their output rows. */
int vd_attn_forward_plan(const vd_attn* h, const vd_attn_batch* batch, void* workspace,
                         size_t workspace_bytes, hipStream_t stream);
int vd_attn_forward_splits(const vd_attn* h, const vd_attn_batch* batch, void* out,
                           void* workspace, size_t workspace_bytes, hipStream_t stream);
int vd_attn_forward_chunks(const vd_attn* h, const vd_attn_batch* batch, void* out,
                           const void* workspace, size_t workspace_bytes, hipStream_t stream);
int vd_attn_forward_merge(const vd_attn* h, const vd_attn_batch* batch, void* out,
                          const void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The splits and chunks phases with their kernels timed: identical launches
 * and results, and in addition `start` and `stop` (hipEvent_t the caller
 * created with timing enabled, or NULL) are recorded by the kernel dispatches
 * themselves (hipExtLaunchKernel): `start` at the start of the phase's first
 * kernel (the shared-prefix kernel when it runs), `stop` at the end of its
 * last, with no separate marker packet in the stream.  When the phase
 * launches no kernel (no such rows), both events are recorded back to back
 * on `stream`. */
int vd_attn_forward_splits_timed(const vd_attn* h, const vd_attn_batch* batch, void* out,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream,
                                 hipEvent_t start, hipEvent_t stop);
int vd_attn_forward_chunks_timed(const vd_attn* h, const vd_attn_batch* batch, void* out,
                                 const void* workspace, size_t workspace_bytes,
                                 hipStream_t stream, hipEvent_t start, hipEvent_t stop);

/* Opt-in check of the batch's device-side data, the preconditions the host cannot see
 * (Appendix A.1: 0 < s_r <= n_r; page ids within the pool).  One kernel on `stream`; reads
 * only.  status: device int32 [num_seqs]; status[r] receives the bit mask of what request r
 * violates (0: nothing):
 *    1  s_r < 1 or s_r > n_r (cu_q_lens, context_lens);
 *    2  s_r > max_q_len or n_r > max_context_len (the host hints);
 *    4  ceil(n_r / 16) > pt_stride;
 *    8  cu_q_lens[r] < 0 or cu_q_lens[r + 1] > total_q_tokens;
 *   16  a page id among the entries 0 .. ceil(n_r / 16) - 1 of its table row (those
 *       within the stride) lies outside [0, num_pages).
 * vd_attn_forward skips a request with any of bits 1, 2, 4, 8 (its output rows are left
 * unwritten) and reads a page with bit 16's ids as zeros.  Host-visible errors as for
 * vd_attn_forward; a batch with no request returns VD_OK without a launch. */
int vd_attn_validate(const vd_attn* h, const vd_attn_batch* batch, int32_t* status,
                     hipStream_t stream);

/* Bytes of ONE pool (K or V) holding num_pages pages. */
int vd_pool_bytes(const vd_attn* h, int64_t num_pages, size_t* bytes);

/* KV-cache write (the engine writes new tokens' K/V to private slots before
 * attention reads them, Section 4.1 "Separate cache reuse from generation").
 *
 * k_new, v_new: device [num_tokens, Hkv, D] bf16 rows (16-byte aligned).
 * slot_mapping: device [num_tokens] int64 (8-byte aligned), slot = page * 16 + offset; a
 *               negative slot skips the token; slots outside
 *               [0, num_pages * 16) are skipped too.
 * k_pool, v_pool: device pools of vd_pool_bytes(num_pages) bytes each (16-byte aligned).
 *
 * Pool layout (one "page block" per (page, KV head), 16 * D bf16 elements at
 * element offset (page * Hkv + kv_head) * 16 * D):
 *   K block: element (slot, d) at ((d / 8) * 16 + slot) * 8 + d % 8
 *   V block: element (slot, d) at ((d / 16) * 4 + slot / 4) * 64 + (d % 16) * 4 + slot % 4
 * so that the matrix-core operand of each wavefront is one contiguous load.
 * Two tokens written to the same slot in one call race (either may win). */
int vd_kv_write(const vd_attn* h, const void* k_new, const void* v_new,
                const int64_t* slot_mapping, int64_t num_tokens, void* k_pool, void* v_pool,
                int64_t num_pages, hipStream_t stream);

/* Batch-invariant linear layer (the matmul contract of Section 5.4, Fig. 3: the output
 * row of a token depends only on that token's input row and on the weights):
 *   c[m][n] = bf16_RNE( sum_k a[m][k] * b[n][k] )   for 0 <= m < M, 0 <= n < N
 * a: device [M rows of lda] bf16 activations (the first K values of a row used);
 * b: device [N rows of ldb] bf16 weights, one row per output feature (the layout a
 *    linear layer stores, [out_features, in_features]); the first K values used;
 * c: device [M rows of ldc] bf16 output (the first N values of a row written).
 * Each output element is one fp32 accumulation chain of v_mfma_f32_16x16x32_bf16 over K
 * in ascending 32-wide chunks starting from +0, cast to bf16 round-to-nearest-even: row m
 * of c is bit-identical for any M, any position of the row in a, and any strides.  The
 * tiling is fixed (it depends on nothing but the build); there is no split over K.
 * Requirements (else VD_ERR_UNSUPPORTED for K, VD_ERR_INVALID_ARG otherwise): K a multiple
 * of 64; when K > 0, lda, ldb >= K and multiples of 8 with a and b 16-byte aligned (K = 0:
 * a and b are not read and every output is +0); ldc >= N; c 2-byte aligned; M, N, K >= 0
 * (M = 0 or N = 0: nothing to do).  Launches on `stream` and
 * returns without waiting; allocates nothing.  Strides are in elements. */
int vd_linear(const void* a, int64_t lda, const void* b, int64_t ldb, void* c, int64_t ldc,
              int64_t M, int32_t N, int32_t K, hipStream_t stream);

/* Static description of a status code (never NULL). */
const char* vd_status_string(int status);

/* Fixed tiling constants of a handle (host query, for reports and tests):
 * tile_keys = 64, split_keys = 1024, page_size = 16. */
int vd_attn_tiling(const vd_attn* h, int32_t* tile_keys, int32_t* split_keys,
                   int32_t* page_size);

#ifdef __cplusplus
}
#endif

#endif /* VDATTN_H */
