/*
 * cowa.h -- C ABI of the CoWindow Attention (CoWA) library for AMD MI355X (gfx950).
 *
 * CoWA is causal attention in which every KV head sees a shared prefix-sink
 * window and a shared near-diagonal window, while complementary long-range
 * windows split the remaining causal distances across the KV heads so that
 * together they cover the whole causal prefix (paper Sec. 2.1, Eq. fwa_support,
 * Eq. fwa_collective_coverage).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All functions are extern "C", never throw, and return a cowa_status.  On a
 *   negative status nothing has been launched and no output has been written;
 *   cowa_last_error() then returns a message for the calling thread.
 * - Device pointers are plain addresses of memory the caller allocated on the
 *   current HIP device.  The library allocates no memory, never synchronises,
 *   and enqueues its kernels on the given stream (a hipStream_t passed as
 *   void*; NULL is the default stream).  Asynchronous kernel faults surface at
 *   the caller's next synchronisation of that stream.
 * - Tensors are dense, contiguous and head-major (Sec. 2.3, forward
 *   execution): Q, O, dQ, dO are [B, H_q, N_q, d]; K, V, dK, dV are
 *   [B, H_k, N_k, d]; LSE is [B, H_q, N_q] float32 holding the natural-log
 *   log-sum-exp of each row (Alg. 1, final step).  Element type is bfloat16 or
 *   float32 per cowa_params.dtype; q/k/v/o/do/dq/dk/dv must be 16-byte aligned
 *   and lse 4-byte aligned.
 * - Queries and keys are bottom-right aligned: query i_q and key i_k are at
 *   causal distance delta = i_q + (N_k - N_q) - i_k (Eq. fwa_distance); N_q <= N_k.
 * - QO head h uses KV head floor(h * H_k / H_q) (Sec. 2.1, grouped-query attention).
 * - Window breakpoints use the global KV-head index h_k_offset + h_local and the
 *   global head count h_k_total (Eq. fwa_global_head); a single device holding
 *   all heads passes h_k_total = h_k and h_k_offset = 0.
 */
#ifndef COWA_H_
#define COWA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  COWA_OK = 0,
  COWA_ERR_INVALID_ARG = -1,       /* a size, window, pointer or alignment is invalid */
  COWA_ERR_UNSUPPORTED = -2,       /* valid but not built: head_dim, tile or dtype combination */
  COWA_ERR_WORKSPACE = -3,         /* workspace pointer missing or smaller than required */
  COWA_ERR_SCHEDULE_MISMATCH = -4, /* schedule built for different shapes or windows */
  COWA_ERR_NO_DEVICE = -5,         /* no HIP device, or the current device is not gfx950 */
  COWA_ERR_HIP = -6                /* a HIP call or kernel launch failed */
} cowa_status;

typedef enum { COWA_BF16 = 0, COWA_FP32 = 1 } cowa_dtype;

/* Per-KV-head window four-tuple of Sec. 2.1 (the interface of Alg. 1 and
 * Alg. 2): sink width, near width, gap after the near window, long-range
 * width.  KV head h sees key i_k from query i_q iff, with the causal distance
 * delta = i_q + (N_k - N_q) - i_k >= 0,
 *     delta < near,  or  i_k < sink,  or  near + gap <= delta < near + gap + width.
 * The default pattern (Eq. fwa_long_range_span) is (w_sink, w_near, b_h,
 * b_{h+1} - b_h) with L = max(N_k - w_sink - w_near, 0), b_h = floor(h L / H_k)
 * over the global KV-head index; Sec. 2.1 notes that the same interface
 * permits head-specific widths and gaps, e.g. the m-window layouts of the
 * collective-coverage ablation (App. A.1, Table 1).  All fields >= 0. */
typedef struct {
  int32_t sink, near, gap, width;
} cowa_window;

/* Shapes and windows of one forward/backward call.
 *
 * Fixed lengths (cu_seqlens_q == NULL): B sequences of N_q queries and N_k
 * keys; tensors [B, H, N, d] as described above.
 *
 * Ragged batch (cu_seqlens_q and cu_seqlens_k non-NULL; Eq. fwa_distance
 * aligns each sequence's queries to the end of its own keys, which is what
 * variable-length prefill needs): sequence b has queries
 * [cu_seqlens_q[b], cu_seqlens_q[b+1]) and keys [cu_seqlens_k[b],
 * cu_seqlens_k[b+1]) of the packed tensors Q, O, dO, dQ [H_q, N_q, d] and K,
 * V, dK, dV [H_k, N_k, d] (LSE [H_q, N_q]), where n_q = cu_seqlens_q[B] and
 * n_k = cu_seqlens_k[B] are the packed totals.  Both arrays are host int32
 * [batch + 1], start at 0, never decrease, and 0 <= N_q(b) <= N_k(b) for every
 * sequence; a query of sequence b never sees a key of another sequence.
 *
 * Windows: windows == NULL takes the default rule from w_sink, w_near,
 * h_k_total and h_k_offset (per sequence from its own N_k when ragged);
 * otherwise windows points to h_k host tuples, one per local KV head, used
 * as given for every sequence (w_sink, w_near, h_k_total, h_k_offset are then
 * not used for the windows).
 *
 * The host arrays are read by the call that receives them and not kept, except
 * that a schedule records a digest of their values (see cowa_schedule_t). */
typedef struct {
  int32_t batch;          /* B >= 0; B = 0 is a no-op */
  int32_t n_q, n_k;       /* fixed: 1 <= N_q <= N_k < 2^30; ragged: the packed totals (< 2^30) */
  int32_t h_q, h_k;       /* local heads on this device; H_q % H_k == 0 */
  int32_t head_dim;       /* 64 or 128 */
  int32_t w_sink, w_near; /* >= 0 */
  int32_t h_k_total;      /* global KV heads (>= h_k_offset + h_k) */
  int32_t h_k_offset;     /* global index of local KV head 0 */
  int32_t tile_q, tile_k; /* block sizes B_q, B_k: 32, 64 or 128 */
  float softmax_scale;    /* > 0, multiplies Q K^T (1/sqrt(d) for the standard scale) */
  int32_t dtype;          /* cowa_dtype */
  const cowa_window* windows;    /* NULL (default rule) or h_k host tuples */
  const int32_t* cu_seqlens_q;   /* NULL (fixed lengths) or host int32 [batch + 1] */
  const int32_t* cu_seqlens_k;   /* NULL iff cu_seqlens_q is NULL */
} cowa_params;

/* Block schedule (Sec. 2.3): for every local KV head h and QO block i the KV
 * blocks J_h(i) that hold at least one legal pair, and its inverse I_h(j).
 * A caller-owned plain struct; the device buffer `buf` of `bytes` bytes is
 * caller-allocated and filled by cowa_schedule().  Layout of buf (each array
 * starts at a 256-byte aligned offset given below):
 *   fwd_row_ptr  int32 [h_k * n_qt + 1]   row r = h * n_qt + i
 *   bwd_col_ptr  int32 [h_k * n_kt + 1]   column c = h * n_kt + j
 *   fwd_ent      uint32[nnz]  (j << 1) | partial, j descending in a row (Alg. 1)
 *   bwd_ent      uint32[nnz]  (i << 1) | partial, i ascending in a column (Alg. 2)
 *   then internal tables (resolved windows; sequence table and block-to-
 *   sequence maps of a ragged batch) at off_windows .. bytes.
 * In a ragged batch i and j count the blocks over the whole batch (the blocks
 * of sequence b follow those of sequence b - 1; each sequence starts a new
 * block), while the entries hold blocks within the sequence.  partial = 0
 * (FULL) iff all B_q * B_k element pairs of the tile lie inside the sequence
 * and are legal; only partial tiles are masked element-wise.
 * `p` is a copy of the sizing parameters: its pointer fields must still hold
 * the same values when cowa_schedule is called (checked against `digest`),
 * and cowa_fwd / cowa_bwd compare the digest of their own parameters. */
typedef struct {
  cowa_params p;          /* the parameters it was sized for */
  int32_t n_qt, n_kt;     /* QO / KV blocks: ceil(N / B) per sequence, or summed over a ragged batch */
  int32_t max_row;        /* longest J_h(i) */
  int32_t max_col;        /* longest I_h(j) */
  int64_t nnz;            /* listed tiles over the local KV heads (and sequences, when ragged) */
  size_t off_fwd_row_ptr, off_bwd_col_ptr, off_fwd_ent, off_bwd_ent; /* byte offsets in buf */
  size_t off_windows, off_seqs, off_qt_seq, off_kt_seq;            /* internal tables */
  int32_t max_qt, max_kt; /* QO / KV blocks of the longest sequence */
  uint64_t digest;        /* of the window tuples and sequence lengths it was sized for */
  size_t bytes;           /* size of buf */
  void* buf;              /* device buffer, set by the caller */
} cowa_schedule_t;

/* Shapes of one decoding step (Sec. 2.3, decoding execution). */
typedef struct {
  int32_t batch;          /* sequences B >= 0 */
  int32_t h_q, h_k;       /* local heads; H_q % H_k == 0 */
  int32_t head_dim;       /* 64 or 128 */
  int32_t n_max;          /* KV-cache capacity (row stride) per sequence and head */
  int32_t w_sink, w_near; /* >= 0 */
  int32_t h_k_total, h_k_offset;
  int32_t split_keys;     /* visible keys per split program (a multiple of 64); 0 = library
                             default: ~1024 programs in total, each >= 256 keys */
  float softmax_scale;    /* > 0 */
  int32_t dtype;          /* COWA_BF16 */
  const cowa_window* windows;  /* NULL: default rule from each sequence's N_k; else h_k host
                                  tuples (at most 256 local KV heads), the same for every sequence */
} cowa_decode_params;

/* Library version string. */
const char* cowa_version(void);

/* Message for the last non-OK status returned on the calling thread. */
const char* cowa_last_error(void);

/* Window tuples of the h_k local KV heads for key length n_k (Sec. 2.1,
 * Eq. fwa_long_range_span, Eq. fwa_global_head).  Host only; out_host has
 * p->h_k entries.  Computed in 64-bit integers.  With explicit windows they
 * are returned as given; for a ragged batch under the default rule each
 * sequence has its own tuples (from its N_k): this returns those of key
 * length p->n_k. */
cowa_status cowa_windows(const cowa_params* p, cowa_window* out_host);

/* Size the schedule of `p` (Sec. 2.3; tile sets are the paper's J_h(i) and
 * I_h(j)): fills every field of *out except buf.  Host only, O(h_k (n_qt + n_kt)).
 * Validates the windows and sequence lengths (COWA_ERR_INVALID_ARG). */
cowa_status cowa_schedule_size(const cowa_params* p, cowa_schedule_t* out);

/* Work accounting (host only): the number of legal (query, key) pairs of
 * Eq. fwa_support summed over the batch and every QO head.  Attention FLOPs
 * follow from it (App. A.2 and A.3: 4d per pair forward, 10d backward). */
cowa_status cowa_legal_pairs(const cowa_params* p, int64_t* pairs);

/* Work accounting of one decoding step (host only): visible keys summed over
 * the sequences (seqlens_host: host int32 [batch]) and the local KV heads;
 * each is one K row and one V row read.  Invalid lengths count zero. */
cowa_status cowa_decode_visible_keys(const cowa_decode_params* p, const int32_t* seqlens_host, int64_t* keys);

/* Build the schedule into s->buf on the device: the window (and sequence)
 * tables, then three small kernels: per-row counts, prefix sums, entry fill.
 * The host arrays of s->p are read during the call (they are copied into the
 * kernels' arguments), so they may be freed as soon as it returns. */
cowa_status cowa_schedule(const cowa_schedule_t* s, void* stream);

/* Forward (Alg. 1): O and LSE of masked softmax attention over each query's
 * visible-key set.  q [B,H_q,N_q,d], k/v [B,H_k,N_k,d] -> o [B,H_q,N_q,d],
 * lse [B,H_q,N_q] float32.  `s` must have been sized for the same n_q, n_k,
 * h_k, windows, global head indexing and tiles, and built.  The bf16 path
 * takes tile_q and tile_k in {64, 128} (COWA_ERR_UNSUPPORTED otherwise) and
 * keeps one schedule row in LDS: COWA_ERR_UNSUPPORTED (before any launch)
 * when ceil(N_k / tile_k) exceeds 8188 (head_dim 128, tile_k 128; 24572 for
 * tile_k 64 or head_dim 64 with tile_k 128; 32764 for head_dim 64, tile_k
 * 64), i.e. 1M key tokens at 128. */
cowa_status cowa_fwd(const cowa_params* p, const cowa_schedule_t* s,
                     const void* q, const void* k, const void* v,
                     void* o, float* lse, void* stream);

/* Workspace bytes cowa_bwd needs: per query row, the float32 -D with
 * D = rowsum(O * dO) (the term of Alg. 2) and -LSE log2(e) (the row's
 * exponent offset in base 2): two arrays in the row layout of LSE; then, when
 * the KV blocks holding sink keys have query lists much longer than every
 * other KV block (every query sees the sink, Eq. fwa_support), float32 dK/dV
 * partials of those blocks, which the dK/dV stage walks in several parts and
 * sums in a fixed order (at most 16 parts per block and 256 MB in total; the
 * split depends only on the parameters, so results stay deterministic). */
cowa_status cowa_bwd_workspace_size(const cowa_params* p, size_t* bytes);

/* Backward (Alg. 2): exact gradients of <dO, O> w.r.t. the unscaled Q, K and
 * V, using the saved O and LSE of the forward.  dq like q; dk/dv like k/v
 * (keys that no query sees get zero).  bf16 only; tile_q and tile_k in
 * {64, 128}.  Equivalent to cowa_bwd_prepare, cowa_bwd_main and cowa_bwd_dq in
 * that order on the same workspace.  Deterministic: no atomics.
 * Each pass keeps one schedule row or column in LDS, which bounds the shape:
 * COWA_ERR_UNSUPPORTED (before any launch) when ceil(N_q / tile_q) exceeds
 * 16000 (head_dim 128; 28288 for 64) or ceil(N_k / tile_k) exceeds 8192
 * (head_dim 128, tile_k 128; 24576 for tile_k 64; 24576 and 32768 for
 * head_dim 64): 2M query and 1M key tokens at the 128 x 128 tiles.  All
 * three backward entry points apply these checks. */
cowa_status cowa_bwd(const cowa_params* p, const cowa_schedule_t* s,
                     const void* q, const void* k, const void* v,
                     const void* o, const float* lse, const void* d_o,
                     void* dq, void* dk, void* dv,
                     void* workspace, size_t ws_bytes, void* stream);

/* Backward stage 1: the per-row values of Alg. 2 into the workspace -- -D with
 * D = rowsum(O * dO) (subtracted from dP), and -LSE log2(e) from the saved
 * natural-log LSE of the forward (the offset that rebuilds P = exp(S - LSE)). */
cowa_status cowa_bwd_prepare(const cowa_params* p, const void* o, const void* d_o, const float* lse,
                             void* workspace, size_t ws_bytes, void* stream);

/* Backward stage 2, dK and dV (the loop of Alg. 2 over QO blocks): for every
 * local KV head and KV block, over every QO head of its group and every QO
 * block of I_h(j) in ascending order, recompute P from LSE, form dS, and
 * accumulate dK and dV of the block, written once without atomics.  Needs
 * the workspace filled by cowa_bwd_prepare. */
cowa_status cowa_bwd_main(const cowa_params* p, const cowa_schedule_t* s,
                          const void* q, const void* k, const void* v,
                          const void* d_o, void* dk, void* dv,
                          void* workspace, size_t ws_bytes, void* stream);

/* Backward stage 3, dQ: for every QO head and QO block, over the KV blocks of
 * J_h(i), recompute P and dS and accumulate dQ = scale dS K, written once.
 * (Alg. 2 adds these contributions with atomics inside stage 2; a separate
 * pass avoids them.)  Needs the workspace filled by cowa_bwd_prepare. */
cowa_status cowa_bwd_dq(const cowa_params* p, const cowa_schedule_t* s,
                        const void* q, const void* k, const void* v,
                        const void* d_o, void* dq,
                        void* workspace, size_t ws_bytes, void* stream);

/* Workspace bytes of one decoding step (Sec. 2.3, decoding execution): the
 * visible keys of each (sequence, KV head) are split into ranges processed in
 * parallel, and each range leaves a partial softmax state per QO head -- its
 * running maximum m, its sum l and its unnormalised output O (float32) --
 * that a second kernel merges.  Depends on batch, h_q, head_dim, n_max, the
 * windows and split_keys. */
cowa_status cowa_decode_workspace_size(const cowa_decode_params* p, size_t* bytes);

/* One decoding step (Sec. 2.3): the forward with N_q = 1 for every sequence b,
 * N_k = seqlens_k[b] (cached tokens plus the current one, already appended;
 * 1 <= N_k <= n_max), breakpoints recomputed from that N_k.  q [B,H_q,d],
 * k_cache/v_cache [B,H_k,n_max,d], seqlens_k device int32 [B] -> o [B,H_q,d],
 * lse [B,H_q].  A seqlens_k value outside [1, n_max] yields O = 0 and
 * LSE = -inf for that sequence. */
cowa_status cowa_decode(const cowa_decode_params* p, const void* q,
                        const void* k_cache, const void* v_cache,
                        const int32_t* seqlens_k, void* o, float* lse,
                        void* workspace, size_t ws_bytes, void* stream);

/* cowa_decode without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): the same kernels and results as cowa_decode, with the
 * split partials in a device array inside the library (32 MiB per GPU, held
 * until the process ends; looked up once per device).  Allocates nothing.
 * Returns COWA_ERR_UNSUPPORTED (before any launch) when cowa_decode_workspace_size
 * of `p` exceeds 32 MiB (e.g. 64 sequences x 32 QO heads x d = 128 use 2 MiB at
 * the default split size).  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (different streams or host threads) race and
 * must be serialised by the caller.  Nothing in the array needs clearing: each
 * call overwrites every partial it reads. */
cowa_status cowa_decode_noalloc(const cowa_decode_params* p, const void* q,
                                const void* k_cache, const void* v_cache,
                                const int32_t* seqlens_k, void* o, float* lse, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* COWA_H_ */
