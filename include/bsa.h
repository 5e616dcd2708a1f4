/*
 * bsa.h - dynamic block-sparse attention (forward) with per-request planning
 *         for AMD Instinct MI355X (gfx950).
 *
 * The problem (Section 2.1, Eq. 1): for each batch b and head h,
 *     O = softmax(Q K^T / sqrt(d) + bias_M) V,
 * where the logical mask M marks blocks of B_Q query tokens by B_KV key/value
 * tokens active or inactive and bias_M is 0 on the token pairs of active
 * blocks and -inf elsewhere.  A query row with no active key gets O = 0 and
 * LSE = -inf.
 *
 * A request (Section 3, online request path; Algorithm 2) is served in two
 * calls:
 *   bsa_plan    builds the shared mask state mu(M) on the GPU (block-CSR and
 *               mask statistics), copies the statistics to the host (the one
 *               device-to-host synchronisation of a request), looks up the
 *               performance regime in the plan table, takes the first
 *               eligible plan of its ranking, and prepares only that plan's
 *               metadata on the GPU (physical tiles, membership, tasks,
 *               Split-K workspace; Section 4);
 *   bsa_forward runs the plan's kernels on any Q/K/V/O of the planned shapes
 *               (warm repeats reuse the prepared plan; Section 7.4).
 *
 * Conventions
 *   - Every entry point returns a bsa_status and never throws.  On failure a
 *     thread-local message is available from bsa_last_error().
 *   - "device" pointers are HIP device allocations of the current device;
 *     "host" pointers are ordinary host memory.
 *   - Streams are hipStream_t values passed as void*; NULL means the legacy
 *     default stream.
 *   - Tensors are bfloat16 with head_dim 128.  Strides are in elements and
 *     ordered (batch, head, token); the head-dim stride is 1 and every token
 *     row must start 16-byte aligned.
 *   - The caller owns the mask, Q, K, V, O and LSE buffers.  A plan owns its
 *     device metadata and workspace until bsa_plan_destroy.
 */
#ifndef BSA_H_
#define BSA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Only the entry points below are exported from the shared library. */
#define BSA_API __attribute__((visibility("default")))

#define BSA_VERSION_MAJOR 1
#define BSA_VERSION_MINOR 1
#define BSA_MAX_SEGMENTS 16

typedef enum {
  BSA_OK = 0,
  BSA_ERR_INVALID = 1,     /* malformed argument (null pointer, bad stride, size) */
  BSA_ERR_UNSUPPORTED = 2, /* no eligible plan for the request (Algorithm 2) */
  BSA_ERR_HIP = 3,         /* a HIP runtime call or kernel launch failed */
  BSA_ERR_OOM = 4,         /* device or host allocation failed */
  BSA_ERR_LUT = 5          /* plan table artifact missing, malformed or for another arch/version */
} bsa_status;

enum { BSA_DTYPE_BF16 = 0, BSA_DTYPE_F16 = 1, BSA_DTYPE_F32 = 2 };

/* Tensor shapes of a request (the tensor properties x of R = <A, M, B, x>,
 * Section 4.4).  Q and O are [batch, seq_q, heads, head_dim] in general
 * strided form; K and V are [batch, seq_kv, heads, head_dim]. */
typedef struct {
  int32_t batch, heads, seq_q, seq_kv, head_dim, dtype;
  int64_t q_stride[3], k_stride[3], v_stride[3], o_stride[3]; /* (batch, head, token), elements */
} bsa_shapes;

/* The logical mask M (Section 2.1).  One byte per logical block, nonzero =
 * active.  Head h of batch b is the row-major [ceil(seq_q/B_Q[h])] x
 * [ceil(seq_kv/B_KV[h])] byte matrix starting at
 *     data + b * stride_b + head_offset[h]
 * (head_offset == NULL: head h starts at h * nqb * nkb, requires one geometry
 * for all heads).  stride_b == 0 broadcasts one mask over the batch. */
typedef struct {
  const uint8_t* data;        /* device */
  const int64_t* head_offset; /* host [heads] or NULL */
  int64_t stride_b;           /* elements */
} bsa_mask;

typedef struct bsa_plan_s* bsa_plan_t; /* opaque; owns device metadata */
typedef struct bsa_lut_s* bsa_lut_t;   /* opaque; read-only after load, shareable */

/* Planning options.  Zero-initialise and set what is needed. */
typedef struct {
  int32_t force_plan;  /* >= 0: use this catalog plan for every segment (must be eligible); -1: select */
  int32_t select_mode; /* 0: plan table (Algorithm 2); 1: base plan only */
  bsa_lut_t lut;       /* NULL: the library's default table (BSA_LUT_PATH or the shipped artifact) */
  int32_t keep_row_order; /* 0: above 512 tasks, dispatch in row order except that each task moves up
                             to the first task of its head with the same KV tile list, so tasks that
                             read the same K/V run side by side and share the L2 (BSA_EXPORT_DISPATCH);
                             1: dispatch in row order.  The output is the same either way. */
} bsa_plan_opts;

/* Per-segment summary of a plan.  Heads that share one logical geometry form
 * a segment; each segment has its own regime lookup and plan. */
typedef struct {
  int32_t bq, bkv;           /* logical geometry B */
  int32_t n_heads;
  int32_t plan_id;           /* catalog id of the selected plan */
  int32_t tq, tkv, split;    /* physical tile T and Split-K partitions of that plan */
  int32_t mapping;           /* 0 Direct, 1 Coarsened, 2 Refined, 3 mixed (Section 4.2) */
  int32_t regime_hit;        /* 1 if the plan table had a ranking for the regime */
  int32_t reserved;
  int64_t nnz;               /* active logical blocks */
  int64_t blocks;            /* all logical blocks (density denominator) */
  int64_t run_blocks;        /* active blocks in runs of length >= 2 (Section 5.1) */
  int64_t max_row_nnz;       /* largest active-block count of one query-block row */
  int64_t n_rows;            /* physical query rows */
  int64_t n_tiles;           /* active physical tiles */
  int64_t n_tasks;           /* workgroup tasks */
  int64_t workspace_bytes;   /* Split-K partial-state workspace */
} bsa_segment_info;

/* One catalog entry (Section 4.4): a native kernel configuration, i.e. a
 * physical tile (Section 4.2) and a task organization (Section 4.3). */
typedef struct {
  int32_t id;
  int32_t tq, tkv;   /* physical tile */
  int32_t split;     /* Split-K partitions per query tile (1 = none) */
  int32_t stages;    /* pipeline depth (buffered K/V stages) */
  int32_t waves;     /* wavefronts per workgroup */
  int32_t xcd_group; /* traversal order: the MI355X's eight XCDs work in groups of this many (2 or 8), each
                        group through its own contiguous share of the dispatch order, the XCDs of a group
                        taking turns over runs of 8 consecutive tasks; 8 keeps every XCD on the same stretch
                        of tasks (the same heads), 2 spreads four stretches over the chip.  Without Split-K
                        the shares hold equal work (per-(b, h) active blocks), otherwise equal task counts */
} bsa_catalog_entry;

/* Regime-lookup input z_A(R) = <k_A(R), u_A(R), s_A(M)> (Eq. 3).  Tables
 * may also use two features derived from these: query_rows = batch_heads *
 * ceil(seq_q / bq), and row_imbalance = max_row_nnz * query_rows / nnz (the
 * longest query-block row against the mean row). */
typedef struct {
  int32_t bq, bkv, dtype, head_dim; /* request key (with the library's architecture) */
  int64_t batch_heads;              /* batch x heads of the segment */
  int64_t seq_q, seq_kv;
  int64_t nnz, blocks, run_blocks;  /* mask statistics */
  int64_t max_row_nnz;              /* largest active-block count of one query-block row */
} bsa_regime_query;

/* Export selectors for bsa_plan_export. */
enum {
  BSA_EXPORT_ROW_PTR = 0,     /* logical block-CSR offsets, int64 [R + 1], rows (b, h, qb) */
  BSA_EXPORT_COL_IDX = 1,     /* logical block-CSR columns, int32 [nnz] */
  BSA_EXPORT_BH_NNZ = 2,      /* active blocks per (b, h), int64 [batch * heads] */
  BSA_EXPORT_TILE_PTR = 3,    /* segment's physical tile offsets, int64 [rows + 1] */
  BSA_EXPORT_TILE_KV = 4,     /* segment's physical KV tile index per active tile, int32 */
  BSA_EXPORT_TILE_MEMBER = 5, /* segment's membership bits per tile, uint64 (Coarsened plans) */
  BSA_EXPORT_TASKS = 6,       /* segment's tasks, int64 [n_tasks][6]: bh, pq, tile_begin, tile_end, split, nsplit */
  BSA_EXPORT_DISPATCH = 7     /* segment's dispatch order, int64 [n_tasks]: the BSA_EXPORT_TASKS index of the task
                                 at each position (row order, each task moved up to the first task with the same
                                 KV tile list and member bits; the identity in row order) */
};

/* Library version. */
BSA_API bsa_status bsa_version(int32_t* major, int32_t* minor);

/* Human-readable name of a status code (static storage). */
BSA_API const char* bsa_status_string(bsa_status s);

/* Detail of the last failure on the calling thread (thread-local storage,
 * valid until the next call on this thread). */
BSA_API const char* bsa_last_error(void);

/* Load a plan-table artifact (Section 5.1: catalog + plan table + feature
 * schema, versioned together).  Host only.  Fails with BSA_ERR_LUT when the
 * file is missing or malformed, or its architecture, format version or
 * catalog does not match this library.  *out is NULL on failure. */
BSA_API bsa_status bsa_lut_load(const char* path, bsa_lut_t* out);
BSA_API bsa_status bsa_lut_destroy(bsa_lut_t lut);

/* The ranking Pi_A(r) for regime query z (Eq. 4), written to plans[0..cap).
 * *n receives the ranking length, *hit 1 if the table holds the regime and 0
 * if the lookup missed (then the ranking is the key's base plan alone,
 * Algorithm 2).  Host only; lut NULL means the default table. */
BSA_API bsa_status bsa_lut_rank(bsa_lut_t lut, const bsa_regime_query* z, int32_t* plans, int32_t cap,
                        int32_t* n, int32_t* hit);

/* Algorithm 2 on given statistics: the first eligible plan of the ranking for
 * z, for tensors of shape `shapes`.  BSA_ERR_UNSUPPORTED (and *plan_id = -1)
 * when none is eligible.  Host only. */
BSA_API bsa_status bsa_select_plan(bsa_lut_t lut, const bsa_regime_query* z, const bsa_shapes* shapes,
                           int32_t* plan_id);

/* Catalog introspection (Section 4.4).  Host only. */
BSA_API int32_t bsa_catalog_size(void);
BSA_API bsa_status bsa_catalog_get(int32_t id, bsa_catalog_entry* out);

/* Eligible(P, R) of Section 4.4 for catalog plan `plan_id`, logical geometry
 * (bq, bkv) and shapes: supported dtype, head dim, layout, tile/block nesting
 * and membership size, and one head's K and V rows addressable with 32-bit
 * byte offsets ((seq_kv + 64) * token stride * 2 + 256 < 4 GiB).  *eligible
 * receives 0 or 1.  Host only. */
BSA_API bsa_status bsa_plan_eligible(int32_t plan_id, int32_t bq, int32_t bkv, const bsa_shapes* shapes,
                             int32_t* eligible);

/* The base plan of request key (bq, bkv) (Section 5.1): a catalog plan
 * eligible for every request with that key.  Host only. */
BSA_API bsa_status bsa_base_plan(int32_t bq, int32_t bkv, int32_t* plan_id);

/*
 * Plan a request.  B_Q/B_KV hold n_geom logical geometries: n_geom == 1 for
 * one geometry shared by all heads, or n_geom == heads for one per head.  The
 * mask must stay unchanged until this call returns; the plan does not keep a
 * reference to it.  Work is ordered on `stream`; the call blocks once, for
 * the statistics copy.  On success *out owns the plan; on failure *out is
 * NULL and nothing is leaked.
 */
BSA_API bsa_status bsa_plan(const bsa_mask* mask, const int32_t* B_Q, const int32_t* B_KV, int32_t n_geom,
                    const bsa_shapes* shapes, const bsa_plan_opts* opts, void* stream,
                    bsa_plan_t* out);

/*
 * Run a plan: O (and LSE, optional) from Q, K, V of the planned shapes (all
 * device pointers).  lse is [batch, heads, seq_q] float32, natural-log
 * log-sum-exp of the scaled scores, -inf for query rows with no active key.
 * Asynchronous on `stream`; kernel faults surface as BSA_ERR_HIP at a later
 * synchronising call.  Calls on one plan must not overlap in time (the
 * Split-K workspace is shared).
 */
BSA_API bsa_status bsa_forward(bsa_plan_t plan, const void* q, const void* k, const void* v, void* o, float* lse,
                       void* stream);

/* Number of geometry segments of a plan and the summary of one. */
BSA_API bsa_status bsa_plan_num_segments(bsa_plan_t plan, int32_t* n);
BSA_API bsa_status bsa_plan_info(bsa_plan_t plan, int32_t segment, bsa_segment_info* out);

/* Heads of a segment, ascending, into heads[0..cap); *n receives the count. */
BSA_API bsa_status bsa_plan_segment_heads(bsa_plan_t plan, int32_t segment, int32_t* heads, int32_t cap, int32_t* n);

/* Copy plan metadata to host memory (synchronises the plan's stream).
 * `segment` is ignored for the logical mask-state exports.  *needed receives
 * the size in bytes; with host_buf NULL nothing is copied. */
BSA_API bsa_status bsa_plan_export(bsa_plan_t plan, int32_t segment, int32_t what, void* host_buf, size_t bytes,
                           size_t* needed);

/* Release a plan (stream-ordered on the plan's stream). */
BSA_API bsa_status bsa_plan_destroy(bsa_plan_t plan);

/*
 * Top-k block sparsifier: the step before bsa_plan that supplies the logical
 * mask M for geometry (bq, bkv) (Section 2.1: the sparsifier hands M and B to
 * the runtime), so that sparsify -> plan -> forward stays on the device.
 * For every (b, h) and query block qb, KV block kb scores
 *     s = sum_c mean(Q rows of qb)[c] * mean(K rows of kb)[c]
 * (a ragged last block averages the rows it has); the `topk` largest scores
 * of each row are active, ties going to the lower kb, and with diagonal != 0
 * every block that the token diagonal i == j passes through is added.  The
 * scores are computed in IEEE double, block sums in token order, the sum
 * over c in increasing order with one rounding per multiply and per add, so
 * the selection is reproducible bit for bit off the device.
 *
 * q: [batch, seq_q, heads, 128] and k: [batch, seq_kv, heads, 128] bf16,
 * device, strides from `shapes` (v and o strides are ignored).  mask: device
 * uint8 [batch, heads, ceil(seq_q / bq), ceil(seq_kv / bkv)], contiguous,
 * caller-owned, written entirely (1 = active); for bsa_plan pass
 * head_offset[h] = h * nqb * nkb and stride_b = heads * nqb * nkb.
 * topk <= 0 selects no block by score, topk >= nkb every block.
 * Errors: BSA_ERR_INVALID for null pointers, non-positive geometry or bad
 * shapes; BSA_ERR_UNSUPPORTED for a dtype other than bf16, a head dim other
 * than 128, or more than 6144 KV blocks per row.  Scratch memory (block
 * means and score rows of up to 256 MiB of heads at a time) is taken from
 * the device's stream-ordered pool and returned on `stream`.  Asynchronous
 * on `stream`.
 */
BSA_API bsa_status bsa_sparsify_topk(const void* q, const void* k, const bsa_shapes* shapes, int32_t bq,
                                     int32_t bkv, int32_t topk, int32_t diagonal, uint8_t* mask, void* stream);

/*
 * bsa_sparsify_topk without any device allocation, for callers that cannot
 * allocate: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Arguments, layouts, the selection and its error codes
 * are those of bsa_sparsify_topk; the result is the same mask bit for bit.
 * Its block means and score rows live in a fixed 64 MiB scratch array that
 * the library keeps on every device it runs on until the process ends
 * (looked up once per device).  One pass holds as many heads as fit, so the
 * limit is one head: (ceil(seq_q/bq) + ceil(seq_kv/bkv)) * 1024 bytes of
 * means plus ceil(seq_q/bq) * ceil(seq_kv/bkv) * 8 bytes of scores must not
 * exceed 64 MiB (BSA_ERR_INVALID otherwise, before any device work).  Every
 * call on a device shares that device's scratch and leaves its contents
 * behind: calls that overlap in time on one device (different streams or
 * threads) race and must be serialised by the caller.  Asynchronous on
 * `stream`; calls no hipMalloc, hipFree or allocating library routine.
 */
BSA_API bsa_status bsa_sparsify_topk_noalloc(const void* q, const void* k, const bsa_shapes* shapes, int32_t bq,
                                             int32_t bkv, int32_t topk, int32_t diagonal, uint8_t* mask,
                                             void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BSA_H_ */
