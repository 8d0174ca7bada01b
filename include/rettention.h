/*
 * rettention.h — C ABI of the MI355X (gfx950) Re-ttention attention library.
 *
 * Re-ttention (arXiv 2505.22918) runs block-sparse softmax attention at very
 * high sparsity and corrects each query row with statistics cached at an
 * earlier full-attention denoising step: the sparse softmax is scaled by the
 * ratio rho of the sparse to the full softmax denominator (Eq.8, Eq.9) and the
 * cached residual R of the masked tokens is added (Eq.10, App. A.3).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Q, K, V, O and R are bf16 tensors [B, H, T, D], contiguous, row-major
 *    (D fastest).  D is the real head width d_h; supported D: 64, 72.
 *  - Scores are A^pre = Q K^T / sqrt(D) with the real D (Eq.2).
 *  - Row statistics are fp32 [B, H, T]: row_max m = max_j A^pre_ij and
 *    row_sum l = sum_j exp(A^pre_ij - m) over the keys the call attends to,
 *    so l * exp(m) is the softmax denominator of Eq.4 (dense) or Eq.5 (sparse).
 *  - rho is fp32 [B, H, T]; one value per batch element, head and query row.
 *  - The block mask is a CSR over blocks of `block` tokens, shared by every
 *    (batch, head) or given per head (rt_bsr): block b covers tokens
 *    [b*block, min((b+1)*block, T)),
 *    n_qblk = n_kblk = ceil(T / block).  row_ptr has n_qblk+1 entries, col_idx
 *    lists the kept key blocks of each query block in ascending order.  A key
 *    past T is never attended to.
 *  - Tensor pointers marked "device" are device memory owned by the caller; the
 *    library allocates nothing and keeps no state except a thread-local error
 *    string.  Every call that takes `stream` (a hipStream_t passed as void*)
 *    only enqueues work on it and returns; results are ready after the caller
 *    synchronises that stream.
 *  - Argument errors are found on the host before anything is enqueued, and
 *    the call then returns a non-zero rt_status and enqueues nothing.  A launch
 *    failure returns RT_EHIP.  rt_last_error() describes the last failure on
 *    the calling thread.
 *  - An output buffer must not overlap any input buffer or another output of
 *    the same call (RT_EINVAL): every work item reads all of a head's K and V
 *    while others write their output rows.
 *  - A call with B*H*T == 0 checks its arguments and enqueues nothing.
 *  - Every call launches on the calling thread's current HIP device (and the
 *    allocation-free build uses that device's copy of its workspace): the
 *    device pointers and the stream must belong to it.
 */
#ifndef RETTENTION_H
#define RETTENTION_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RT_OK = 0,
    RT_EINVAL = 1,       /* a null pointer, a negative or inconsistent size  */
    RT_EUNSUPPORTED = 2, /* a head width or block size the library lacks    */
    RT_ECAPACITY = 3,    /* an output buffer smaller than the result needs   */
    RT_EHIP = 4          /* the HIP runtime refused a launch                 */
} rt_status;

/* Shape of Q, K, V, O, R: [B, H, T, D]. */
typedef struct {
    int32_t B, H, T, D;
} rt_dims;

/* A block CSR on the device: one mask shared by all (batch, head), or one per
 * head, or one per (batch, head) (Eq.5 indexes the kept set by head).
 * row_ptr [n_masks][n_qblk + 1] and col_idx [nnz] are device int32 arrays;
 * row_ptr entries are absolute offsets into col_idx (mask m's rows start at
 * row_ptr[m][0]).  Head h of batch b uses mask 0 (n_masks 0 or 1), mask h
 * (n_masks == H) or mask b*H + h (n_masks == B*H).  Every query block must
 * keep at least one key block: Eq.5 normalises over the kept keys, so an empty
 * kept set has no softmax.  rt_bsr_check verifies a host copy of the CSR (the
 * Python binding runs it on every CSR it copies to the device) and the index
 * builder never emits an empty row.  The attention calls do not read the device
 * arrays on the host; for a CSR the host has not checked, the kernels clamp
 * row_ptr entries to [0, nnz] and skip column indices outside [0, n_qblk), so a
 * malformed CSR cannot make them read out of bounds, and a query block left
 * with no kept key block comes out as NaN rows (rt_attn_cache: rho = 0). */
typedef struct {
    const int32_t* row_ptr;
    const int32_t* col_idx;
    int32_t block;   /* 32 or 64 */
    int32_t n_qblk;  /* must equal ceil(T / block) */
    int32_t nnz;     /* entries in col_idx */
    int32_t n_masks; /* 0 or 1 (shared), H or B*H */
} rt_bsr;

/* Host only.  Checks a host copy of a block CSR before it is used on the
 * device: host_row_ptr [n_masks][n_qblk + 1] and host_col_idx [nnz] mirror
 * mask->row_ptr / mask->col_idx (the device pointers are not read).  Returns
 * RT_EINVAL when a row is empty (Eq.5 needs a kept key), when offsets leave
 * [0, nnz] or decrease, when a column index leaves [0, n_qblk) or a row is
 * not strictly ascending, or when nnz differs from the largest last offset
 * (row_ptr[n_qblk] for a single mask); RT_EUNSUPPORTED for a block size other
 * than 32 or 64. */
rt_status rt_bsr_check(const rt_bsr* mask, const int32_t* host_row_ptr, const int32_t* host_col_idx);

/* Static mask patterns (Sec.3 static masks; App. A.4 local windows). */
enum {
    RT_PAT_EXPLICIT = 0, /* given 0/1 block matrix                              */
    RT_PAT_LOCAL2D = 1,  /* image latent grid_h x grid_w, spatial window        */
    RT_PAT_VIDEO3D = 2   /* n_text text tokens then frames x grid_h x grid_w    */
};

typedef struct {
    int32_t kind;
    const uint8_t* mask;      /* EXPLICIT, device: n_qblk x n_qblk row-major 0/1  */
    const uint8_t* host_mask; /* EXPLICIT, host copy read by rt_index_size only  */
    int32_t grid_h, grid_w;   /* LOCAL2D and VIDEO3D latent grid                 */
    int32_t frames;           /* VIDEO3D latent frames                           */
    int32_t n_text;           /* VIDEO3D leading text tokens                     */
    int32_t keep;             /* LOCAL2D: key blocks kept per query block;
                                 VIDEO3D: video key blocks kept per video query
                                 block (text key blocks are always kept)         */
    int32_t n_masks;          /* EXPLICIT: masks stacked in mask / host_mask
                                 (n_masks x n_qblk x n_qblk; 0 means 1); the
                                 built CSR holds n_masks row_ptr arrays.  The
                                 window patterns are the same for every head
                                 and take 0 or 1.                                */
} rt_pattern;

/*
 * Block-index rule (the paper names local windows, App. A.4, but no block
 * rule).  A block's centroid is the mean latent position of its tokens; image
 * token t sits at (t / grid_w, t % grid_w); video token n_text + v sits at
 * (v / (grid_h*grid_w), (v / grid_w) % grid_h, v % grid_w).  Candidate key
 * blocks are ranked by (squared centroid distance, |kb - qb|, kb) ascending and
 * the first ones kept; each row is stored in ascending kb.  LOCAL2D keeps
 * min(keep, n_qblk) blocks.  VIDEO3D: a block with any text token is a text
 * block; text query blocks keep all text key blocks only; video query blocks
 * keep all text key blocks plus the min(keep, #video blocks) highest-ranked
 * video key blocks.  The result is exact (integer arithmetic) and unique.
 */

/* Host only.  Writes the exact number of CSR entries rt_index_build produces.
 * EXPLICIT reads pattern->host_mask (host, n_masks x n_qblk x n_qblk) and
 * returns RT_EINVAL for a row without a kept block (Eq.5).  Needs T >= 1,
 * block in {32, 64}, grid sizes matching T (LOCAL2D: grid_h*grid_w == T;
 * VIDEO3D: n_text + frames*grid_h*grid_w == T), keep >= 1, n_qblk <= 4096. */
rt_status rt_index_size(const rt_pattern* pattern, int32_t T, int32_t block, int32_t* nnz_out);

/* Builds the CSR on the device: row_ptr [n_masks][ceil(T/block)+1] (absolute
 * offsets), col_idx [capacity]; EXPLICIT with several masks needs
 * n_masks * ceil(T/block) <= 32768.
 * For LOCAL2D / VIDEO3D the size is known on the host and a capacity below it
 * is RT_ECAPACITY.  EXPLICIT reads pattern->mask (device) and writes at most
 * `capacity` entries; when pattern->host_mask is given it is checked as in
 * rt_index_size (RT_EINVAL for an empty row, RT_ECAPACITY when it needs more
 * than capacity), otherwise the caller must size capacity to the mask and keep
 * every row non-empty. */
rt_status rt_index_build(const rt_pattern* pattern, int32_t T, int32_t block, int32_t* row_ptr,
                         int32_t* col_idx, int32_t capacity, void* stream);

/* Dynamic block mask, chosen from the step's own Q and K (the run-time masks
 * Sec.6 and App. A.2 name as future work, by the block-pooled Q K^T with top-k
 * selection Sec.2 describes).  Per (batch, head) and query block qb:
 *   score(qb, kb) = sum_d Qsum_qb[d] * Kmean_kb[d]
 * Qsum: the fp32 sum of qb's rows, one addition per row in ascending order;
 * Kmean: kb's rows summed the same way, divided by its token count; the dot
 * product accumulates in fp32 over ascending d, product and sum each rounded
 * (no fused multiply-add).  qb keeps itself (Eq.5 needs a non-empty kept set)
 * and the keep - 1 best other blocks (higher score first, ties to the lower
 * index; a NaN score ranks as -inf, after every other score), stored
 * ascending, so every row holds exactly
 * kk = min(keep, n_qblk) blocks.  The result is one mask per (batch, head):
 * row_ptr [B*H][n_qblk + 1] (absolute offsets, row (bh, qb) starting at
 * (bh*n_qblk + qb)*kk) and col_idx [B*H*n_qblk*kk], for an rt_bsr with
 * n_masks = B*H and nnz = B*H*n_qblk*kk.
 * q, k: device bf16 [B,H,T,D]; row_ptr, col_idx: device int32 (written);
 * capacity: entries col_idx can hold (RT_ECAPACITY below nnz); workspace:
 * caller-owned device memory of at least the bytes rt_dynamic_index_workspace
 * reports (RT_ECAPACITY otherwise), overwritten; outputs and workspace must not
 * overlap the inputs or each other.  Needs block in {32, 64}, keep >= 1 and
 * n_qblk <= 4096. */
rt_status rt_dynamic_index_workspace(rt_dims dims, int32_t block, int32_t keep, int64_t* bytes);
rt_status rt_dynamic_index(const void* q, const void* k, rt_dims dims, int32_t block, int32_t keep,
                           int32_t* row_ptr, int32_t* col_idx, int32_t capacity, void* workspace,
                           int64_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): rt_dynamic_index
 * with its workspace taken from a library-owned device array of 16 MiB per
 * GPU instead of an argument; nothing is allocated.  The shape's workspace
 * (2*B*H*n_qblk*D fp32) must fit it, else RT_ECAPACITY.  The array's address
 * is looked up on the first call on each device (RT_EHIP if that fails).
 * Every call on one GPU shares that GPU's array: calls that overlap on one GPU
 * (on different streams or threads) race; calls on one stream do not.  Nothing
 * in it needs clearing between calls. */
rt_status rt_dynamic_index_noalloc(const void* q, const void* k, rt_dims dims, int32_t block, int32_t keep,
                                   int32_t* row_ptr, int32_t* col_idx, int32_t capacity, void* stream);

/* Dense attention with row statistics, Eq.1 with the Eq.4 denominator.
 * q, k, v: device bf16 [B,H,T,D]; o: device bf16 [B,H,T,D] (written);
 * row_max, row_sum: device fp32 [B,H,T] (written, either may be NULL).
 * The query tiling uses `block` rows (32 or 64). */
rt_status rt_attn_full(const void* q, const void* k, const void* v, rt_dims dims, int32_t block,
                       void* o, float* row_max, float* row_sum, void* stream);

/* Sparse attention over a block mask, Eq.5: each row's softmax runs over the
 * tokens of its query block's kept key blocks only.  Same buffers as
 * rt_attn_full; row statistics are over the kept keys. */
rt_status rt_attn_sparse(const void* q, const void* k, const void* v, rt_dims dims,
                         const rt_bsr* mask, void* o, float* row_max, float* row_sum,
                         void* stream);

/* One-pass caching step (App. A.3): dense attention over every key block,
 * with the keys split by the mask into the kept set S and the rest, so that
 * one walk gives the step's full output and the statistics cache:
 *   O_full = softmax over all keys (Eq.1)                  -> o
 *   rho    = sum_{j in S} e^{s_j} / sum_j e^{s_j}  (Eq.8)  -> rho
 *   R      = sum_{j not in S} A_j v_j = O_full - rho O_S   -> resid (Eq.10)
 * The kept blocks are walked first (their normalised output passes through o,
 * which is then overwritten), the others after, against one running max.
 * q, k, v: device bf16 [B,H,T,D]; o, resid: device bf16 [B,H,T,D] (written,
 * must not alias q, k, v or each other); rho: device fp32 [B,H,T] (written);
 * row_max / row_sum: device fp32 [B,H,T], the full-attention statistics, or
 * NULL.  Rows whose query block keeps every key block get rho = 1, R = 0; a
 * query block with no kept block gets rho = 0, R = O_full.
 * rho may be NULL: the cache of the ablation without the statistical reshape
 * (Eq.10 with the ratio fixed at one, the window-attention-plus-caching scheme
 * the paper compares against in Sec.5 and App. A.4) is then written instead,
 * resid = O_full - O_S (O_full where the query block keeps no block). */
rt_status rt_attn_cache(const void* q, const void* k, const void* v, rt_dims dims, const rt_bsr* mask,
                        void* o, float* row_max, float* row_sum, float* rho, void* resid, void* stream);

/* Post-softmax masking, Eq.7 (the Sec.3 toy operation, an ablation, not a
 * speedup): O = (A o M) V, the full softmax A of Eq.4 with the masked entries
 * zeroed and the full denominator kept, so each row sums to rho < 1.  Runs the
 * caching walk (every key block) and writes only o: device bf16 [B,H,T,D]
 * (must not alias q, k, v).  Equals rho * SparseAttention(Q,K,V) of the same
 * step (Eq.8). */
rt_status rt_attn_postmask(const void* q, const void* k, const void* v, rt_dims dims, const rt_bsr* mask,
                           void* o, void* stream);

/* Statistics cache at a caching (full-attention) step, Eq.8 and Eq.10:
 *   rho = (l_sparse / l_full) * exp(m_sparse - m_full)      (Eq.8)
 *   R   = O_full - rho * O_sparse                           (Eq.10)
 * o_full, o_sparse: device bf16 [B,H,T,D]; m_*, l_*: device fp32 [B,H,T];
 * rho: device fp32 [B,H,T] (written); resid: device bf16 [B,H,T,D] (written,
 * rounded to nearest even).  With rho NULL (the ablation without the reshape)
 * R = O_full - O_sparse is written and m_*, l_* are not read (may be NULL). */
rt_status rt_cache_build(const void* o_full, const float* m_full, const float* l_full,
                         const void* o_sparse, const float* m_sparse, const float* l_sparse,
                         rt_dims dims, float* rho, void* resid, void* stream);

/* Fused sparse attention + statistical reshape, Eq.5 then Eq.9 with the ramp
 * of Sec.4.2 and the residual of Eq.10:
 *   O = min(1, rho + rho_delta) * SparseAttention(Q,K,V) + R
 * rho_delta = lambda * (t - c) is the ramp accumulated since the caching step
 * c (0 for no ramp).  rho: device fp32 [B,H,T]; resid: device bf16 [B,H,T,D];
 * o: device bf16 [B,H,T,D] (written); row_max / row_sum: device fp32 [B,H,T],
 * the sparse statistics of this step, or NULL to skip writing them.
 * rho may be NULL: the ablation without the statistical reshape then computes
 * O = SparseAttention(Q,K,V) + R (no Eq.9 scaling; rho_delta is ignored), with R
 * the ratio-free cache of rt_attn_cache / rt_cache_build. */
rt_status rt_attn_sparse_reshape(const void* q, const void* k, const void* v, rt_dims dims,
                                 const rt_bsr* mask, const float* rho, const void* resid,
                                 float rho_delta, void* o, float* row_max, float* row_sum,
                                 void* stream);

/* The same reshape applied to an already computed sparse output (unfused):
 * Eq.9 scales the sparse softmax output by the cached ratio, ramped by
 * rho_delta as in Sec.4.2 and clamped to 1, and Eq.10 adds the cached residual:
 *   O = min(1, rho + rho_delta) * o_sparse + R
 * o_sparse, resid, o: device bf16 [B,H,T,D]; rho: device fp32 [B,H,T], or NULL
 * for the ablation without the reshape (O = o_sparse + R). */
rt_status rt_reshape_apply(const void* o_sparse, const float* rho, const void* resid,
                           float rho_delta, rt_dims dims, void* o, void* stream);

/* Static description of a status code. */
const char* rt_status_str(rt_status status);

/* The message of the last failing call on this thread ("" if none). */
const char* rt_last_error(void);

/* Library version, major*10000 + minor*100 + patch. */
int32_t rt_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RETTENTION_H */
