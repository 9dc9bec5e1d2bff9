/*
 * msparse -- vertical-slash dynamic sparse attention for long-context training
 * on one AMD Instinct MI355X (gfx950).  C ABI of libmsparse.so.
 *
 * The library implements the single-GPU hot path of MTraining (arXiv
 * 2510.18830): per-head pattern estimation from the last queries (Algorithm 1,
 * Section 4.1), conversion of the selected vertical and slash lines into a
 * 64 x 64 block index plus a token-level column index (Section 4.1 (ii),
 * convert_index of Algorithms 1 and 2), and a sparse FlashAttention forward
 * (out + LSE) and backward (dQ, dK, dV) over only the selected blocks and
 * columns (block_bar_sparse_attention_forward of Algorithm 2; gradients by
 * Eq. softmax_gradient and Eq. attention_backward).  A ring worker's share
 * (Section 4.2, Algorithm 2) is one call per ring step with a msparse_ring
 * descriptor, and partial results are combined by msparse_merge_out_lse
 * (merge_out_and_lse of Algorithm 2).
 *
 * Conventions shared by every entry point
 *   - Tensors are device pointers to contiguous row-major arrays, 16-byte
 *     aligned: Q, O, dO bf16 [B, Hq, Nq, d]; K, V bf16 [B, Hkv, Nk, d];
 *     lse fp32 [B, Hq, Nq] (natural log); dQ fp32 [B, Hq, Nq, d];
 *     dK, dV fp32 [B, Hkv, Nk, d].  A tensor off 16-byte alignment is
 *     rejected with MSPARSE_ERR_INVALID.
 *   - GQA: query head h reads KV head h / (Hq / Hkv) (contiguous groups).
 *   - Causal attention with 64-token blocks only.  scale <= 0 selects
 *     1 / sqrt(head_dim).
 *   - The caller owns every buffer, including the workspace; the library
 *     allocates no device memory and keeps no state besides its loaded code.
 *     Calls are re-entrant.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *     returns before it finishes.  Only msparse_index_count waits for the GPU.
 *     Setting MSPARSE_SYNC_CHECK=1 in the environment makes every call wait
 *     for its kernels and report asynchronous faults as MSPARSE_ERR_HIP
 *     (except on a stream under graph capture, whose work runs at replay).
 *   - Arguments are validated on the host before anything is launched, so a
 *     call that returns an error has enqueued no work.
 */
#ifndef MSPARSE_H
#define MSPARSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#ifndef MSPARSE_API
#define MSPARSE_API __attribute__((visibility("default")))
#endif

typedef enum {
    MSPARSE_OK = 0,
    MSPARSE_ERR_INVALID = -1,     /* null pointer, k or last_q outside [1, N], Hq % Hkv != 0, bad ring */
    MSPARSE_ERR_UNSUPPORTED = -2, /* head_dim not 64/128, N % 64 != 0, non-causal, block != 64, last_q > 64 */
    MSPARSE_ERR_CAPACITY = -3,    /* index capacities below what the call must write */
    MSPARSE_ERR_WORKSPACE = -4,   /* workspace missing or smaller than the *_workspace query */
    MSPARSE_ERR_HIP = -5          /* a HIP launch or runtime call failed */
} msparse_status;

/* Problem shape.  seq_q and seq_k are the local lengths (equal for a whole
 * sequence; in ring mode the worker's query shard and one KV shard, both
 * N_global / world). */
typedef struct {
    int32_t batch;
    int32_t seq_q;
    int32_t seq_k;
    int32_t heads_q;
    int32_t heads_kv;
    int32_t head_dim; /* 64 or 128 */
    int32_t block;    /* must be 64 */
    int32_t causal;   /* must be 1 */
    float scale;      /* <= 0: 1 / sqrt(head_dim) */
} msparse_dims;

enum { MSPARSE_LAYOUT_STRIPED = 0, MSPARSE_LAYOUT_ZIGZAG = 1 };

/* One step of a ring (Section 4.2).  The global sequence of world * seq_q
 * tokens is split into 64-token blocks; block g belongs to
 *   STRIPED: worker g mod world;
 *   ZIGZAG:  worker c if c < world else 2 world - 1 - c, c = g / (nb / (2 world)).
 * A worker keeps its blocks in ascending global order.  At step t worker
 * `rank` holds the KV shard of worker (rank - t) mod world (the flat ring).
 * With inner > 1 dividing world (and below it), the steps follow the
 * hierarchical order of Section 4.3 / Algorithm 2 instead: the world / inner
 * nodes of `inner` cards (rank = node * inner + card) run an outer ring over
 * nodes and, within each outer step, an inner ring over the node's cards, so
 * at step t = i * inner + j worker rank holds the shard of worker
 *   ((node - i) mod (world / inner)) * inner + (card - j) mod inner
 * (msparse_ring_shard).  inner = 0, 1 or world is the flat ring.  Passing NULL
 * instead of a descriptor means the whole sequence (world = 1). */
typedef struct {
    int32_t world;
    int32_t rank;
    int32_t step;
    int32_t layout;
    int32_t inner; /* cards per node for the hierarchical order; 0 = flat ring */
} msparse_ring;

/* The sparse index of one call (whole sequence or one ring step).  All arrays
 * are device memory owned by the caller; bh = b * Hq + h.
 *   blk_ptr  int64 [B*Hq*nqb + 1]  blk_idx[blk_ptr[bh*nqb+i] .. blk_ptr[bh*nqb+i+1])
 *                                  are the ascending local key blocks of local
 *                                  query block i (nqb = seq_q / 64)
 *   col_ptr  int64 [B*Hq*nqb + 1]  col_idx: ascending local key token offsets of
 *                                  the vertical columns of query block i that no
 *                                  selected block already covers
 *   kblk_ptr int64 [B*Hq*nkb + 1]  kblk_idx: the transpose of the block lists
 *                                  (ascending local query blocks per local key
 *                                  block, nkb = seq_k / 64); same length as blk_idx
 *   vcol_ptr int64 [B*Hq + 1]      vcol_idx: ascending local key offsets of the
 *                                  head's verticals that lie in this KV shard
 *   diag_bits uint32 [B*Hq*ceil(nb/32)]  bit x set when block-diagonal x (query
 *                                  block - key block, global) is selected;
 *                                  nb = global blocks
 *   q_blk_global int32 [nqb], k_blk_global int32 [nkb]: global block numbers
 *   overflow int32 [1] (may be NULL): set to 1 by msparse_build_index when a
 *                                  capacity was too small, else 0.  The build
 *                                  then writes nothing out of bounds, but the
 *                                  lists are incomplete (an entry range that
 *                                  crosses a capacity is left unwritten), so
 *                                  the attention calls read this flag first and,
 *                                  when it is set, return from every kernel
 *                                  without reading the lists or writing any
 *                                  output: out, lse, out_f32, o_acc, lse_acc,
 *                                  dq, dk and dv keep their previous contents.
 *                                  Check the flag (or size the index with
 *                                  msparse_index_count) before using them.
 *   world    host-side: ring workers the index was built for (1 for a whole
 *            sequence), so nb = world * seq_q / 64
 * blk_cap, col_cap, vcol_cap are host-side element capacities of blk_idx (and
 * kblk_idx), col_idx and vcol_idx. */
typedef struct {
    int64_t* blk_ptr;
    int32_t* blk_idx;
    int64_t blk_cap;
    int64_t* col_ptr;
    int32_t* col_idx;
    int64_t col_cap;
    int64_t* kblk_ptr;
    int32_t* kblk_idx;
    int64_t* vcol_ptr;
    int32_t* vcol_idx;
    int64_t vcol_cap;
    uint32_t* diag_bits;
    int32_t* q_blk_global;
    int32_t* k_blk_global;
    int32_t* overflow;
    int32_t world;
} msparse_index;

/* The worker whose KV shard `rank` holds at ring step `step` (host only, no
 * GPU work), for the flat (inner = 0, 1, world) or hierarchical order above;
 * -1 when the arguments are outside 0 <= rank, step < world or inner does not
 * divide world. */
MSPARSE_API int32_t msparse_ring_shard(int32_t world, int32_t inner, int32_t rank, int32_t step);

/* Human-readable name of a status code (static storage). */
MSPARSE_API const char* msparse_strerror(msparse_status status);

/* Detail of the last error returned on the calling host thread. */
MSPARSE_API const char* msparse_last_error(void);

/* ------------------------------------------------------------------------ */
/* Pattern estimation (Algorithm 1 on one GPU).  For every (b, h): the last
 * last_q query rows n attend causally to all keys m <= n with logits
 * scale * q_n . k_m; P is their row-wise softmax over the whole sequence;
 * v_score[m] = sum_n P[n, m] (vertical scores, sum_v) and
 * s_score[delta] = sum_n P[n, n - delta] (slash scores along n - m = delta,
 * sum_s).  v_idx receives the k_v largest vertical scores and s_idx the k_s
 * largest slash scores (argtopk with a fixed budget; equal scores go to the
 * lower index), each list ascending.
 *   q, k      bf16 [B, Hq, N, d] and [B, Hkv, N, d], N = seq_q = seq_k
 *   v_idx     int32 [B, Hq, k_v];  s_idx int32 [B, Hq, k_s]
 *   v_score, s_score  fp32 [B, Hq, N], or NULL to keep them in the workspace
 * Requires 1 <= last_q <= min(64, N), 1 <= k_v, k_s <= N. */
MSPARSE_API size_t msparse_estimate_workspace(const msparse_dims* dims, int32_t last_q, int32_t k_v, int32_t k_s);
MSPARSE_API msparse_status msparse_estimate(const msparse_dims* dims, const void* q, const void* k, int32_t last_q,
                                int32_t k_v, int32_t k_s, int32_t* v_idx, int32_t* s_idx, float* v_score,
                                float* s_score, void* workspace, size_t workspace_bytes, void* stream);

/* Pattern estimation with the online top-p budget (score_cover of Algorithm 1,
 * Section 4.1 (i)).  The scores are those of msparse_estimate.  For each list
 * the budget is the smallest k whose k largest scores (ties to the lower index)
 * sum to at least p times the list's total mass (L for both lists: every
 * observed softmax row sums to 1), capped at kmax; then argtopk with that k.
 * Masses are summed exactly in fixed point (score * 2^40, truncated), so the
 * budget does not depend on the order of the additions.
 *   p_v, p_s      fractions in (0, 1) (the paper prints no value)
 *   kmax_v/_s     capacities, 1 <= kmax <= N
 *   v_idx         int32 [B, Hq, kmax_v]: the v_cnt[b, h] selected positions
 *                 ascending, then -1 in every unused slot; s_idx alike
 *   v_cnt, s_cnt  int32 [B, Hq] (device): the budgets after the cap
 * The padded lists go to msparse_index_count / msparse_build_index unchanged,
 * with k_v = kmax_v and k_s = kmax_s: negative entries are ignored there.
 * Errors as msparse_estimate, plus MSPARSE_ERR_INVALID for p outside (0, 1)
 * or NULL budget outputs.  The workspace is msparse_estimate's. */
MSPARSE_API size_t msparse_estimate_topp_workspace(const msparse_dims* dims, int32_t last_q, int32_t kmax_v,
                                                   int32_t kmax_s);
MSPARSE_API msparse_status msparse_estimate_topp(const msparse_dims* dims, const void* q, const void* k,
                                                 int32_t last_q, double p_v, double p_s, int32_t kmax_v,
                                                 int32_t kmax_s, int32_t* v_idx, int32_t* s_idx, int32_t* v_cnt,
                                                 int32_t* s_cnt, float* v_score, float* s_score, void* workspace,
                                                 size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Index construction (Section 4.1 (ii); convert_index of Algorithms 1, 2).
 * v_idx [B, Hq, k_v] and s_idx [B, Hq, k_s] are in global token coordinates:
 * vertical positions and slash offsets delta = n - m.  Each slash offset is
 * executed as the 64 x 64 block-diagonals floor(delta/64) and ceil(delta/64)
 * (D); query block i gets the key blocks i - x for x in D, x <= i, and the
 * verticals v <= 64 i + 63 whose block-diagonal i - v/64 is not in D.  With a
 * ring descriptor, the lists are restricted to the step's KV shard and written
 * in local coordinates.  Duplicate entries in v_idx or s_idx count once;
 * negative entries (the unused slots of a top-p list) are ignored.
 *
 * msparse_index_count returns the exact element counts the build will write
 * (it waits for the GPU).  msparse_build_index writes them asynchronously,
 * never past blk_cap / col_cap / vcol_cap.  With an overflow flag, a capacity
 * that turns out too small sets *overflow on the GPU (see msparse_index: the
 * attention calls then leave their outputs untouched).  Without one, every
 * capacity must cover the worst case for the budgets (B Hq nqb min(nkb,
 * 2 k_s, nb) block entries, B Hq nqb min(k_v, seq_k) column entries, B Hq
 * min(k_v, seq_k) vertical entries), else MSPARSE_ERR_CAPACITY before any
 * launch.  The exact sizes come from msparse_index_count. */
MSPARSE_API size_t msparse_index_workspace(const msparse_dims* dims, int32_t k_v, int32_t k_s, const msparse_ring* ring);
MSPARSE_API msparse_status msparse_index_count(const msparse_dims* dims, const int32_t* v_idx, int32_t k_v,
                                   const int32_t* s_idx, int32_t k_s, const msparse_ring* ring,
                                   int64_t* blk_nnz, int64_t* col_nnz, int64_t* vcol_nnz, void* workspace,
                                   size_t workspace_bytes, void* stream);
MSPARSE_API msparse_status msparse_build_index(const msparse_dims* dims, const int32_t* v_idx, int32_t k_v,
                                   const int32_t* s_idx, int32_t k_s, const msparse_ring* ring,
                                   const msparse_index* index, void* workspace, size_t workspace_bytes,
                                   void* stream);

/* Count and build in one call: the work of msparse_index_count followed by
 * msparse_build_index without running the vertical / diagonal preparation
 * and the counts twice.  Waits for the GPU once (to read the counts back),
 * then writes the exact element counts to blk_nnz, col_nnz, vcol_nnz.  When
 * every capacity of `index` covers them, the lists are filled asynchronously
 * on `stream` and MSPARSE_OK is returned; otherwise nothing is filled, the
 * index's overflow flag is set (so the attention calls leave their outputs
 * untouched) and MSPARSE_ERR_CAPACITY is returned with the needed sizes
 * written back: grow the index and call again.  index->overflow must not be
 * NULL.  Errors otherwise as msparse_build_index; the workspace is that of
 * msparse_index_workspace. */
MSPARSE_API msparse_status msparse_index_count_build(const msparse_dims* dims, const int32_t* v_idx, int32_t k_v,
                                                     const int32_t* s_idx, int32_t k_s, const msparse_ring* ring,
                                                     const msparse_index* index, int64_t* blk_nnz, int64_t* col_nnz,
                                                     int64_t* vcol_nnz, void* workspace, size_t workspace_bytes,
                                                     void* stream);

/* msparse_build_index without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, results and errors as
 * msparse_build_index, whose kernels it runs; their scratch (the
 * msparse_index_workspace(dims, k_v, k_s, ring) bytes) lives instead in a
 * fixed device array of 64 MiB inside the library, one per GPU, held from
 * the library's loading on that GPU until the process ends (28 heads at 1M
 * tokens need about 28 MB).  A larger need is MSPARSE_ERR_WORKSPACE before
 * any launch.  The call allocates nothing; its first call on a device looks
 * up that device's array (the calling thread's current device must be the
 * device of `stream` and of the buffers).  Every call on one GPU shares the
 * array: calls that overlap on a GPU (other streams, other threads) race and
 * must be serialised by the caller.  Nothing in the array needs clearing
 * between calls: each build writes what it reads. */
MSPARSE_API msparse_status msparse_build_index_noalloc(const msparse_dims* dims, const int32_t* v_idx, int32_t k_v,
                                                       const int32_t* s_idx, int32_t k_s, const msparse_ring* ring,
                                                       const msparse_index* index, void* stream);

/* Ring workload matrix (Section 4.2; the workload balance analysis of Section 5).
 * For a ring of `world` workers with the given layout over the whole sequence
 * (dims: seq_q = seq_k = N, the global length), counts, summed over all heads,
 * the selected tiles and the column entries of worker r's query blocks whose
 * keys lie in worker s's shard:
 *   tiles, cols  int64 [world * world] (device), entry r * world + s, overwritten.
 * Any step order (flat or hierarchical, msparse_ring_shard) is a permutation of
 * each row; work in tile-equivalents is tiles + cols / 64.  Integer counts,
 * identical to the sizes msparse_index_count reports per ring step.
 * Requires 1 <= world <= 4096 and N / 64 divisible by world (striped) or by
 * 2 world (zigzag); otherwise as msparse_index_count.  The workspace is that
 * of msparse_index_workspace for (dims, k_v, k_s, NULL). */
MSPARSE_API msparse_status msparse_ring_work(const msparse_dims* dims, const int32_t* v_idx, int32_t k_v,
                                             const int32_t* s_idx, int32_t k_s, int32_t world, int32_t layout,
                                             int64_t* tiles, int64_t* cols, void* workspace,
                                             size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Sparse attention forward (block_bar_sparse_attention_forward, Algorithm 2).
 * For each query row n of local query block i, softmax attention over the
 * keys of the selected blocks and columns of i that are causally visible
 * (global key position <= global query position):
 *   out_n = sum_m P[n, m] v_m,  lse_n = log sum_m exp(scale q_n . k_m).
 * A row that sees no key gets out = 0 and lse = -inf.  out is bf16 (round to
 * nearest even), lse fp32.  out_f32 (fp32 [B, Hq, Nq, d], may be NULL) also
 * receives the unrounded output; msparse_attn_bwd computes
 * Delta = dO . O more accurately from it, and ring steps merge it.  out may be
 * NULL when out_f32 is given.  Workspace: msparse_attn_fwd_workspace(dims)
 * bytes (it holds an fp16 copy of v times a power of two, B * Hkv * seq_k *
 * d * 2 bytes, and a few words). */
MSPARSE_API size_t msparse_attn_fwd_workspace(const msparse_dims* dims);
MSPARSE_API msparse_status msparse_attn_fwd(const msparse_dims* dims, const void* q, const void* k, const void* v,
                                const msparse_index* index, void* out, float* lse, float* out_f32,
                                void* workspace, size_t workspace_bytes, void* stream);

/* One ring step's forward merged straight into the running result
 * (block_bar_sparse_attention_forward followed by merge_out_and_lse,
 * Algorithm 2): the forward above (same arguments up to index), then the
 * merge of msparse_merge_out_lse below, without storing the step's partial.
 * A row that neither the running result nor this step has seen stays at
 * O = 0, lse = -inf.
 *   o_acc fp32 [B, Hq, Nq, d], lse_acc fp32 [B, Hq, Nq]: the running (O, lse);
 *   read and updated unless `first`, which writes the step's own result
 *   out_bf16 bf16 [B, Hq, Nq, d] or NULL: also stores the merged O as bf16
 *   (pass it on the last step).
 * Each query row is merged by the workgroup that computes it.  Workspace:
 * msparse_attn_fwd_workspace(dims) bytes.  Errors as msparse_attn_fwd. */
MSPARSE_API msparse_status msparse_attn_fwd_merge(const msparse_dims* dims, const void* q, const void* k, const void* v,
                                      const msparse_index* index, float* o_acc, float* lse_acc, void* out_bf16,
                                      int32_t first, void* workspace, size_t workspace_bytes, void* stream);

/* Log-sum-exp merge of one ring step's partial result into a running one
 * (merge_out_and_lse, Algorithm 2): lse = logaddexp(lse_acc, lse_part),
 * o_acc = exp(lse_acc - lse) o_acc + exp(lse_part - lse) o_part.
 *   o_part fp32 [B, Hq, Nq, d], lse_part fp32 [B, Hq, Nq]: the step's out_f32
 *   and lse from msparse_attn_fwd
 *   o_acc fp32 [B, Hq, Nq, d], lse_acc fp32 [B, Hq, Nq]: read unless `first`,
 *   which copies the partial instead
 *   out_bf16 bf16 [B, Hq, Nq, d] or NULL: also stores the merged O as bf16. */
MSPARSE_API msparse_status msparse_merge_out_lse(const msparse_dims* dims, const float* o_part, const float* lse_part,
                                     float* o_acc, float* lse_acc, void* out_bf16, int32_t first, void* stream);

/* ------------------------------------------------------------------------ */
/* Sparse attention backward over the same index (Eq. softmax_gradient,
 * Eq. attention_backward; the index is a constant).  With
 * P = exp(scale q k^T - lse) on the executed entries and Delta_n = dO_n . O_n:
 *   dV = P^T dO,  dZ = P o (dO V^T - Delta),  dQ = scale dZ K,  dK = scale dZ^T Q,
 * dK and dV summed over the query heads of each KV head.  out (bf16) and lse
 * are the forward's final (merged) results; out_f32 (may be NULL) is the same
 * output unrounded and is used for Delta when given (recommended: Delta from
 * a bf16-rounded O moves large gradients by about 2^-9 of their size).
 * dq, dk, dv are fp32 and overwritten, with two flags:
 *   MSPARSE_BWD_ACCUMULATE_DQ  add into dq instead (ring steps after the first);
 *   MSPARSE_BWD_REUSE_QROWS    the workspace still holds the query-side data of
 *                              the previous msparse_attn_bwd call, made with the
 *                              same dims, q, out, out_f32, dout and lse and the
 *                              same workspace (the previous ring step of the
 *                              same worker; only k, v and the index differ):
 *                              Delta, max |dO| and the fp16 copies of q and dO
 *                              are not recomputed.  Results are undefined if
 *                              that does not hold.
 * Other flag bits are MSPARSE_ERR_INVALID.
 * Range: the fp16 operands are scaled by powers of two chosen per call from
 * max |q|, |k|, |v| and |dO| (dZ by t with t head_dim max|v| in
 * [2^9, 2^10)), so no input scale makes them overflow, and inputs multiplied
 * by powers of two (within the bf16 range) give exactly the correspondingly
 * scaled results; every finite bf16 input is accepted.  Accuracy depends on
 * the logits' magnitude, not on the inputs' scale: the forward and backward
 * recompute P from fp32 logits and the fp32 lse, whose absolute rounding
 * grows with |logit|, and rows with nearly all their weight on one key
 * amplify it in dQ.  Measured: key rows up to 2^4 times the rest (logits up
 * to about +-290) keep every output within 2e-2 of the exact result (row-wise,
 * in units of the row's RMS); key rows 2^8 times larger (logits up to about
 * +-4600) reach 3.7e-2 in dQ.
 * Workspace: msparse_attn_bwd_workspace(dims, vcol_cap) bytes; it holds
 * fp16 copies of q, k, v and dO (each times a power of two), Delta, the scaled
 * row values, and the column pass's work list and per-item partials (its size
 * grows with vcol_cap). */
enum { MSPARSE_BWD_ACCUMULATE_DQ = 1, MSPARSE_BWD_REUSE_QROWS = 2 };
MSPARSE_API size_t msparse_attn_bwd_workspace(const msparse_dims* dims, int64_t vcol_cap);
MSPARSE_API msparse_status msparse_attn_bwd(const msparse_dims* dims, const void* q, const void* k, const void* v,
                                const void* out, const float* out_f32, const void* dout, const float* lse,
                                const msparse_index* index, float* dq, float* dk, float* dv,
                                int32_t flags, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Kernel-level tracing for measurement.  While enabled, every kernel the
 * library launches is bracketed by two HIP events on its stream.
 * msparse_trace_read waits for the recorded events, writes up to `cap`
 * per-kernel totals (launch count and summed milliseconds) into `out`, clears
 * the record and returns the number of distinct kernels.  Host-side state,
 * shared by all threads; do not enable it around graph capture. */
typedef struct {
    char name[32];
    int32_t launches;
    double total_ms;
} msparse_trace_entry;

MSPARSE_API void msparse_trace_enable(int32_t on);
MSPARSE_API int32_t msparse_trace_read(msparse_trace_entry* out, int32_t cap);

/* Achievable MFMA rate (measurement, not part of the attention path): one
 * launch of (CUs x waves_per_simd) workgroups of 256 threads on `stream`,
 * each wave running `iters` rounds of four independent 32x32x16 fp16 MFMA
 * chains (4 x 32768 FLOPs per round) with no memory traffic in the loop; the
 * caller times it with HIP events.  random_operands = 0: one constant operand
 * pair; otherwise eight pairs of random fp16 values cycled from MFMA to MFMA
 * (the power, and so the clock, of the matrix cores depends on the operand
 * data).  `out` (device) receives one float per thread: CUs x waves_per_simd
 * x 256 floats.  MSPARSE_ERR_INVALID for waves_per_simd outside [1, 8],
 * iters < 1 or not a multiple of 8, or a NULL out. */
MSPARSE_API int32_t msparse_mfma_peak_probe(int32_t waves_per_simd, int32_t iters, int32_t random_operands, float* out,
                                void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MSPARSE_H */
