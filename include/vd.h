/*
 * vd.h -- C ABI of the ValueDiff eviction pass on MI355X (gfx950).
 *
 * What is computed (per unit = one (sequence, layer, KV head) of a KV cache):
 *   v_bar = (1/n) sum_{i<n} v_i over the n cached tokens, the block just
 *           appended included (Sec. 3.2, Eq. vd; Sec. 2.2, Eq. block_processing);
 *   score s_j (Sec. 3.2):
 *     VD_SCORE_L2    s_j = ||v_j - v_bar||                 (Eq. vd)
 *     VD_SCORE_DIR   s_j = 1 - cos(v_j, v_bar), with cos := 0 when
 *                    ||v_j|| or ||v_bar|| is zero           (direction-only variant)
 *     VD_SCORE_NORM  s_j = ||v_j||, larger kept            (magnitude-only variant)
 *   the key-side scores of Sec. 4 (Baselines, key geometry) are the same three
 *   forms on the key rows: VD_SCORE_KEY_L2 (ManifoldKV), VD_SCORE_KEY_DIR
 *   (KeyDiff) and VD_SCORE_KEY_NORM (KeyNorm, which keeps the SMALLEST norms);
 *   whenever n exceeds the budget N, the N highest scores are kept (the N
 *   lowest for KeyNorm) (Sec. 2.1, Eq. eviction); equal scores go to the
 *   lower slot index;
 *   K and V are gathered onto the kept set with the slot-reuse layout:
 *   the evicted slots below N, ascending, receive the kept slots at or above
 *   N, ascending, so that afterwards the kept tokens occupy slots [0, N),
 *   surviving tokens below N never move, and K, V (and pos) rows stay paired.
 *
 * Cache layout.  K and V share one descriptor.  Element (seq s, layer l,
 * KV head h, slot j, channel c) lives at
 *     base + s*stride_seq + l*stride_layer + h*stride_head + j*stride_slot + c
 * (strides in elements; the channel stride is 1).  The usual "HND" layout
 * [seq][layer][kv_head][slot][head_dim] and per-layer "NHD" layouts are both
 * strides.  Rows (head_dim contiguous elements) must be 16-byte aligned.
 * Units are numbered u = (s*num_layers + l)*num_kv_heads + h; every per-unit
 * array below ([U][...], U = num_seqs*num_layers*num_kv_heads) is indexed so.
 * Query heads are never read; num_q_heads is only checked for the GQA shape.
 *
 * Memory.  Every array pointer is a DEVICE pointer owned by the caller unless
 * stated otherwise; n_valid and budget are HOST arrays of num_seqs entries
 * (all units of a sequence share n and N).  The library allocates nothing
 * and keeps no state between calls; work is queued on the caller's stream and
 * nothing synchronizes the host.
 *
 * Errors.  Arguments are validated on the host before anything is queued; a
 * rejected call returns VD_ERR_INVALID_ARG or VD_ERR_UNSUPPORTED and queues
 * no work.  A failed launch returns VD_ERR_HIP (the HIP error stays
 * queryable).  Device faults surface at the caller's next synchronization.
 * Inputs must be finite; non-finite values give unspecified rankings.
 *
 * Precision.  Means are accumulated in fp64; scores are computed and returned
 * in fp32, and the selection ranks exactly the fp32 values returned, so the
 * separate and the fused paths keep the same sets.
 */
#ifndef VD_H
#define VD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

struct ihipStream_t;
/* The HIP stream type (hipStream_t); NULL is the default stream. */
typedef struct ihipStream_t *vd_stream;

typedef enum {
    VD_OK = 0,
    VD_ERR_INVALID_ARG = 1,  /* a null, negative, inconsistent or misaligned argument */
    VD_ERR_UNSUPPORTED = 2,  /* a valid shape this build does not handle (see limits) */
    VD_ERR_WORKSPACE = 3,    /* workspace missing or smaller than the size query says */
    VD_ERR_HIP = 4           /* the HIP runtime refused a launch */
} vd_status;

typedef enum { VD_DTYPE_BF16 = 0, VD_DTYPE_F32 = 1 } vd_dtype;

/* Scores (Sec. 3.2 for the value side; Sec. 4, Baselines, for the key side
 * and for FastCAOTE).  The key-side scores are the same three geometric
 * scores taken on the key rows instead of the value rows. */
typedef enum {
    VD_SCORE_L2 = 0,         /* ||v_j - v_bar||, largest kept (ValueDiff) */
    VD_SCORE_DIR = 1,        /* 1 - cos(v_j, v_bar), largest kept */
    VD_SCORE_NORM = 2,       /* ||v_j||, largest kept */
    VD_SCORE_KEY_L2 = 3,     /* ||k_j - k_bar||, largest kept (ManifoldKV) */
    VD_SCORE_KEY_DIR = 4,    /* 1 - cos(k_j, k_bar), largest kept (KeyDiff) */
    VD_SCORE_KEY_NORM = 5,   /* ||k_j||, SMALLEST kept (KeyNorm) */
    VD_SCORE_FASTCAOTE = 6   /* a_j / (1 - a_j) * ||v_j - v_bar|| with a_j the
                                observed attention weight; only in the fused
                                decode step (App. A, Eq. app_fastcaote) */
} vd_variant;

/* Limits of this build. */
#define VD_MAX_CAPACITY 16384  /* slots per unit */

typedef struct {
    void *k;               /* device; may be NULL, then only V (and pos) is gathered */
    void *v;               /* device; never NULL */
    int32_t dtype;         /* vd_dtype; K and V share it */
    int32_t num_seqs;      /* >= 1 */
    int32_t num_layers;    /* >= 1 */
    int32_t num_kv_heads;  /* >= 1 */
    int32_t num_q_heads;   /* multiple of num_kv_heads (GQA); otherwise unused */
    int32_t head_dim;      /* 64, 128 or 256 */
    int32_t capacity;      /* slots per unit, 1 .. VD_MAX_CAPACITY, >= every n_valid */
    int64_t stride_seq, stride_layer, stride_head, stride_slot; /* elements, >= 0 */
} vd_cache_desc;

/*
 * vd_score -- mean and scores of every unit (Sec. 3.2, Eq. vd and variants).
 *   n_valid[s]  host; cached tokens of sequence s, 0 <= n <= capacity
 *   scores      device float [U][capacity]; entries j < n written
 *   variant     VD_SCORE_L2 .. VD_SCORE_KEY_NORM
 *   mean_out    device float [U][head_dim] or NULL; the mean of the scored rows
 *               of units with n > 0 (rounded to fp32)
 * Reads V, or K for a key-side variant (desc->k then required).  Units with
 * n = 0 are left untouched.  scores[j] is the score itself (for KeyNorm the
 * norm, of which the smallest are kept).
 */
vd_status vd_score(const vd_cache_desc *desc, const int32_t *n_valid, vd_variant variant,
                   float *scores, float *mean_out, vd_stream stream);

/*
 * vd_select_topn -- the kept set of every unit (Sec. 2.1, Eq. eviction).
 *   scores      device float [U][capacity], finite; first n entries read
 *   budget[s]   host; N >= 1
 *   keep_mask   device uint8 [U][capacity]; entry j < n set to 1 (kept) or 0
 * Keeps the N largest scores, equal scores going to the lower slot; when
 * n <= N every slot is kept.  -0.0 ranks as +0.0.
 */
vd_status vd_select_topn(const vd_cache_desc *desc, const float *scores,
                         const int32_t *n_valid, const int32_t *budget,
                         uint8_t *keep_mask, vd_stream stream);

/*
 * vd_compact -- slot-reuse gather of K, V and pos from a keep mask (Sec. 2.1,
 * Eq. eviction, the gather).  For units with n > N: holes = slots j < N with
 * keep_mask 0, ascending; movers = slots N <= j < n with keep_mask 1,
 * ascending; the k-th mover's K row, V row and pos entry are copied onto the
 * k-th hole.  With a mask that keeps exactly N slots this leaves the kept
 * tokens in [0, N); with any other mask only min(#holes, #movers) rows move.
 *   pos         device int32 [U][capacity] or NULL; a payload moved with the rows
 */
vd_status vd_compact(const vd_cache_desc *desc, const uint8_t *keep_mask,
                     const int32_t *n_valid, const int32_t *budget, int32_t *pos,
                     vd_stream stream);

/*
 * vd_evict_step -- the whole pass (mean, score, top-N, gather) of every unit
 * in one launch: one block-processing boundary or one decode step
 * (Sec. 2.2, Eq. block_processing).  Results equal vd_score followed by
 * vd_select_topn and vd_compact.
 *   n_valid[s]   host; n = tokens cached after the new block was appended
 *   budget[s]    host; N >= 1; units with n <= N keep everything
 *   variant      VD_SCORE_L2 .. VD_SCORE_KEY_NORM; a key-side variant needs
 *                desc->k and scores the key rows
 *   running_sum  device double [U][head_dim + 1] or NULL.  Optional state
 *                that spares re-reading the old rows for the mean: entries
 *                0..head_dim-1 hold the sum of the unit's cached rows of the
 *                scored tensor (V; K for a key-side variant) in slots
 *                [0, count) and entry head_dim holds count.  On entry, rows
 *                [count, n) are taken as new (count outside [0, n] means
 *                "recompute from all n rows"); on return the state describes
 *                the cache after the pass (count = min(n, N)).  Zero-filled
 *                memory is a valid empty state.  The caller must not change
 *                rows [0, count) between calls without resetting the state.
 *   pos          device int32 [U][capacity] or NULL; moved with the rows
 *   scores_out   device float [U][capacity] or NULL; the scores, j < n
 *   keep_out     device uint8 [U][capacity] or NULL; the keep mask, j < n
 *   workspace    may be NULL when vd_evict_step_workspace_size() returns 0
 * After the call the caller sets n_valid[s] = min(n, N).
 */
vd_status vd_evict_step(const vd_cache_desc *desc, const int32_t *n_valid,
                        const int32_t *budget, vd_variant variant, double *running_sum,
                        int32_t *pos, float *scores_out, uint8_t *keep_out,
                        void *workspace, size_t workspace_bytes, vd_stream stream);

/*
 * vd_geometry -- key and value geometry of every unit (Sec. 3.1, the spread
 * of the distances to the centroid; Sec. 4, bos-cosim).
 *   desc        K and V both required (desc->k non-NULL)
 *   n_valid[s]  host; cached tokens of sequence s, 0 <= n <= capacity
 *   k_sum,      device double [U][head_dim + 1] each, or both NULL: column
 *   v_sum       sums of the unit's K and V rows and, in entry head_dim, the
 *               number of rows they cover (the layout of vd_evict_step's
 *               running sum, which holds V's).  Where both cover exactly the
 *               n rows, the centroids come from them and K and V are read
 *               once; elsewhere they are summed from the rows first (K and V
 *               read twice).  The caller keeps them exact: the results are
 *               those of the sums given.
 *   out         device double [U][5], 8-byte aligned; per unit u
 *               out[5u+0] sigma_K, out[5u+1] sigma_V: population standard
 *                         deviation over the n rows of ||k_i - k_bar|| and
 *                         ||v_i - v_bar|| (k_bar, v_bar: means of all n rows)
 *               out[5u+2], out[5u+3]: the means of those distances
 *               out[5u+4] cosine of k_0 and the mean of k_1 .. k_{n-1}
 *                         (0 when n < 2 or either vector is zero)
 *               all five are 0 for a unit with n = 0
 * Centroids and every sum over rows are fp64; each distance is formed in
 * fp32 (relative error within a few fp32 units in the last place).  Writes
 * nothing but out.  VD_ERR_INVALID_ARG for a NULL K, counts out of range, a
 * NULL or misaligned out, misaligned sums or only one of them.
 */
vd_status vd_geometry(const vd_cache_desc *desc, const int32_t *n_valid, const double *k_sum,
                      const double *v_sum, double *out, vd_stream stream);

/*
 * vd_decode_attention_evict -- one decode step of every sequence, fused with
 * its eviction: attention of the newest token over the n cached rows (Sec.
 * 2.1, Eq. attention; B = 1 in Eq. block_processing), then, where n = N + 1,
 * the eviction of the row with the lowest score, scored in the same pass over
 * K and V.
 *   desc          K and V both required; num_q_heads = G * num_kv_heads with
 *                 G in {1, 2, 4}; query head h*G + g uses KV head h
 *   q             device float [S][L][num_q_heads][head_dim], contiguous: the
 *                 newest token's query rows
 *   scale         softmax scale (1/sqrt(head_dim) in the paper), finite
 *   n_valid[s]    host; cached tokens, the newest included; n <= budget + 1
 *   budget[s]     host; N >= 1
 *   variant       VD_SCORE_L2: s_j = ||v_j - v_bar|| (Sec. 3.2, Eq. vd);
 *                 VD_SCORE_FASTCAOTE: s_j = a_j / (1 - a_j) * ||v_j - v_bar||
 *                 (App. A, Eq. app_fastcaote), a_j the mean over the G query
 *                 heads of the KV head of their softmax weight on row j in
 *                 this very step; s_j is +infinity when 1 - a_j is 0.
 *                 Any other variant is VD_ERR_INVALID_ARG.
 *   running_sum   device double [U][head_dim + 1], required: the column sums
 *                 of the rows it covers, then their count (as vd_evict_step);
 *                 on return it covers the rows left.  Rows it does not cover
 *                 are read by every workgroup of the unit, so it should cover
 *                 all but the newest row.
 *   pos           device int32 [U][capacity] or NULL; moved with the rows
 *   out           device float [S][L][num_q_heads][head_dim]: the attention
 *                 output of every query row (0 for a sequence with n = 0)
 *   workspace     device, 16-byte aligned, at least
 *                 vd_decode_attention_workspace_size(desc, variant) bytes;
 *                 calls that share a workspace must not overlap
 * A unit's rows are split over several workgroups; a second kernel merges
 * them, so the attention reads every row before anything moves.  Eviction:
 * the row with the lowest score goes, the highest slot among equal lowest
 * scores; if it lies below N, row N takes its slot (K, V and pos).  Scores,
 * weights and softmax are fp32 (log2-domain exponentials), the mean and the
 * running sum fp64.  VD_ERR_UNSUPPORTED for n > budget + 1 or another G;
 * VD_ERR_WORKSPACE for a missing or short workspace; VD_ERR_INVALID_ARG as
 * the other calls.
 */
vd_status vd_decode_attention_evict(const vd_cache_desc *desc, const float *q, float scale,
                                    const int32_t *n_valid, const int32_t *budget,
                                    vd_variant variant, double *running_sum, int32_t *pos,
                                    float *out, void *workspace, size_t workspace_bytes,
                                    vd_stream stream);

/* Bytes of device workspace vd_decode_attention_evict needs for this
 * descriptor and variant (0 for an invalid descriptor or variant). */
size_t vd_decode_attention_workspace_size(const vd_cache_desc *desc, vd_variant variant);

/*
 * vd_decode_attention_evict_noalloc -- vd_decode_attention_evict without a
 * workspace argument, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid it).
 * The library allocates nothing here either: the split partials live in a
 * static device array of vd_decode_attention_noalloc_max_bytes() bytes
 * (32 MiB), one copy per GPU, held until the process ends.  Arguments,
 * results and errors are those of vd_decode_attention_evict, and the two
 * give bit-identical results; in addition
 *   - VD_ERR_WORKSPACE when vd_decode_attention_workspace_size(desc, variant)
 *     exceeds that maximum (nothing is queued);
 *   - VD_ERR_HIP when the stream belongs to a device other than the current
 *     one, or the array's address cannot be obtained.
 * Every call on one GPU uses the same array and leaves its contents behind:
 * calls that overlap on one GPU (other streams, other host threads) race
 * and must be ordered by the caller.  Nothing needs to start at zero: each
 * call writes every partial it reads.
 */
vd_status vd_decode_attention_evict_noalloc(const vd_cache_desc *desc, const float *q, float scale,
                                            const int32_t *n_valid, const int32_t *budget,
                                            vd_variant variant, double *running_sum, int32_t *pos,
                                            float *out, vd_stream stream);

/* Bytes of the static device array behind vd_decode_attention_evict_noalloc. */
size_t vd_decode_attention_noalloc_max_bytes(void);

/* Bytes of device workspace vd_evict_step needs for this descriptor (0 in this build). */
size_t vd_evict_step_workspace_size(const vd_cache_desc *desc);

/* A static description of a status code. */
const char *vd_status_string(vd_status status);

/* Measurement aid, not part of the method: reads `bytes` bytes of device
 * memory at `buf` once with the pass kernel's 16-byte streaming loads, over
 * the whole GPU, so that a caller can time the practical HBM read ceiling next
 * to the pass.  `buf` must be 16-byte aligned and `bytes` a multiple of 16;
 * `sink` is a device uint32 written with a value derived from the data only
 * when that value is a fixed unlikely constant (it keeps the loads from being
 * dropped).  Returns VD_ERR_INVALID_ARG for a null or misaligned argument,
 * VD_ERR_HIP if the launch fails. */
vd_status vd_stream_read(const void *buf, size_t bytes, uint32_t *sink, vd_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* VD_H */
