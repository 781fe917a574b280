/*
 * gdy.h -- C-ABI of libgdy: many independent dense GEMMs on one MI355X,
 * run either one after another or concurrently under a dynamic selector.
 *
 * Method: GOLDYLOC (Pati, Aga, Jayasena, Sinclair), "Global Optimizations &
 * Lightweight Dynamic Logic for Concurrency", arXiv 2409.02227.
 *   - GEMM definition: Sec. 2.1.2 -- C (M x N) from A (M x K) and B, with
 *     2*M*N*K flops; T1/T2 say whether A and B are used transposed.
 *   - GO-Kernels: Sec. 4.2 -- per GEMM shape, one kernel tuned for
 *     isolated execution plus one per concurrency degree (CD), found by
 *     tuning under resource constraints (fewer CUs).
 *   - Dynamic logic: Sec. 4.3 -- given the pending independent GEMMs,
 *     predict a CD from per-GEMM features with a multi-class logistic
 *     regression (Eq. 1), run min(CD, available) of them together, and
 *     bind each to the GO-Kernel tuned for that CD.
 *   - Execution configurations: Sec. 5.5 -- sequential, default (all
 *     GEMMs at once with isolation-tuned kernels), GO-Kernels, GOLDYLOC.
 *   - Heterogeneous sets: Sec. 6.7 -- GEMMs run together only if all of
 *     them prefer that CD; otherwise they are split into smaller sets.
 *
 * Storage reading (the paper fixes no base layout): every matrix is
 * row-major with a leading dimension in elements.
 *   op(A)(i,k) = A[i*lda + k]  (trans_a = 0)   or A[k*lda + i] (trans_a = 1)
 *   op(B)(k,j) = B[k*ldb + j]  (trans_b = 0)   or B[j*ldb + k] (trans_b = 1)
 *   C[i*ldc + j] = round(scale_a * scale_b * sum_k op(A)(i,k) op(B)(k,j))
 * with fp32 accumulation, alpha = 1 apart from the fp8 scales, beta = 0
 * (C is overwritten) and round-to-nearest-even into the output type.
 *
 * Supported (a_type, b_type, c_type): (F16, F16, F16), (BF16, BF16, BF16),
 * (FP8_E4M3, FP8_E4M3, BF16), (F32, F32, F32).  FP8_E4M3 is the OCP "E4M3FN"
 * encoding (bias 7, largest finite 448, no infinities).  F32 runs on the
 * fp32 MFMAs (the full-precision GEMMs of Sec. 5.2 and 6.8) and stores C
 * unrounded.
 *
 * Ownership: all matrices are device buffers owned by the caller, who keeps
 * them alive until the origin stream passes the work.  The library owns its
 * stream pool, events, split-K workspace and plan state.  No call allocates
 * device memory after gdy_create.
 *
 * Errors: every call returns a gdy_status; nothing is thrown across the ABI.
 * gdy_execute validates all descriptors before launching anything (all or
 * nothing); gdy_last_error() gives a message for the most recent failure.
 * A context is not thread-safe: use one per host thread, or lock.
 *
 * Environment: HIP maps streams onto GPU_MAX_HW_QUEUES hardware queues per
 * process (4 by default); set it to cover the stream pool plus the caller's
 * streams (24 for the default 16-stream pool) before the process first
 * touches HIP, or concurrent GEMMs share queues and serialise.
 */
#ifndef GDY_H
#define GDY_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GDY_MAX_GEMMS 256   /* most GEMMs in one submission                   */
#define GDY_N_CD 5          /* CD classes 1, 2, 4, 8, 16 (Sec. 4.3)           */
#define GDY_N_FEATURES 18   /* M, N, K, then (#WGs, occupancy, #waves) per CD */

typedef enum {
  GDY_OK = 0,
  GDY_ERR_INVALID_ARG = 1, /* null pointer, negative size, bad ld, bad mode, bad scale */
  GDY_ERR_UNSUPPORTED = 2, /* dtype triple, alignment or extent the kernels cannot take */
  GDY_ERR_ALIAS = 3,       /* a C range overlaps an A, B or C range of the submission */
  GDY_ERR_TOO_MANY = 4,    /* n > GDY_MAX_GEMMS                                      */
  GDY_ERR_TABLE = 5,       /* reserved: a bad GO table falls back instead (gdy_create)  */
  GDY_ERR_HIP = 6,         /* a HIP runtime call failed                              */
  GDY_ERR_NOMEM = 7        /* host allocation failed                                 */
} gdy_status;

typedef enum { GDY_F16 = 1, GDY_BF16 = 2, GDY_FP8_E4M3 = 3, GDY_F32 = 4 } gdy_dtype;

/* Execution configurations (Sec. 5.5). */
typedef enum {
  GDY_SEQUENTIAL = 0, /* isolation-tuned kernel per GEMM, one after another on the origin stream */
  GDY_DEFAULT = 1,    /* isolation-tuned kernels, all n GEMMs at once, one stream each           */
  GDY_GO = 2,         /* GO-Kernels for CD = n, all at once (forced_cd > 0: groups of forced_cd
                         in submission order, one after another)                          */
  GDY_SELECTOR = 3,   /* GOLDYLOC: predicted CD per GEMM, grouping, GO-Kernels per group        */
  GDY_FORCED = 4,     /* each GEMM's `variant`, round-robin over forced_cd streams (tuning)     */
  GDY_FORCED_GROUPED = 5, /* each GEMM's `variant`; consecutive runs of forced_cd GEMMs form
                             groups run one after another, dispatched as GO and SELECTOR
                             groups are (tuning)                                            */
  /* CU-Partition (Sec. 5.5, Sec. 6.9): P = forced_cd (2, 4 or 8; 0: the
     smallest of them >= the number of GEMMs, at most 8) streams on disjoint
     CU masks of CUs/P each; GEMM t of the submission runs on partition
     t mod P (plan.stream_of), one dispatch per GEMM.  Needs a context
     created with use_cu_masks & 2.  The three differ in the kernels:      */
  GDY_CU_PARTITION = 6,    /* isolation-tuned kernels (the paper's CU-Partition)             */
  GDY_CU_PARTITION_GO = 7, /* the GO-Kernels of CD class P, tuned for the unpartitioned GPU    */
  GDY_CU_PARTITION_RC = 8  /* the kernels tuned under CUs/P CUs (the GO table's partition
                              kernels; GO-Kernels of class P where the table has none)       */
} gdy_mode;

/*
 * Dispatch of a group (GO, SELECTOR, FORCED_GROUPED): the GEMMs of a group
 * that are bound to the same kernel share ONE kernel dispatch (up to 16 per
 * dispatch; each GEMM keeps its own grid cap as its share of the grid) in
 * launch order.  The first dispatch of a group runs on the origin stream,
 * further ones on pool streams forked from and joined back to it.  A
 * hardware queue switch costs tens of microseconds on MI355X, far more than
 * the small GEMMs of a group take, so the concurrency of a group lives in one
 * grid wherever its kernels allow.  Each tile is computed by the same code as
 * in an isolated launch, so results are bit-identical.  SEQUENTIAL, DEFAULT
 * and FORCED launch one dispatch per GEMM.
 */
#define GDY_MAX_FUSED 16

/* What an entry of a submission computes.  GDY_OP_ADD is the non-GEMM
 * co-runner of Sec. 7.1: C[i][j] = A[i][j] + B[i][j] over an M x N region
 * (A and B M x N with lda, ldb >= N; k must be 0; trans flags 0; a_type ==
 * b_type == c_type in {F16, BF16, F32}; the sum is formed in fp32 and
 * rounded once).  The selector lets an add join any group (it restricts
 * no concurrency); the GEMMs' predicted degrees decide whether it co-runs. */
typedef enum { GDY_OP_GEMM = 0, GDY_OP_ADD = 1 } gdy_op;

/* One GEMM (or element-wise add) of a submission. */
typedef struct {
  int64_t m, n, k;                  /* sizes; m or n == 0 is a no-op, k == 0 writes zeros   */
  int32_t a_type, b_type, c_type;   /* gdy_dtype values                                     */
  int32_t trans_a, trans_b;         /* T1, T2: 0 or 1 (see storage reading above)          */
  const void* a; int64_t lda;       /* device pointers; leading dimensions in elements      */
  const void* b; int64_t ldb;
  void* c;       int64_t ldc;       /* ldc >= n                                             */
  float scale_a, scale_b;           /* fp8 per-tensor scales; must be 1.0f for other types  */
  int32_t tenant;                   /* caller's tag, reported back in per-kernel timings    */
  int32_t variant;                  /* GDY_FORCED: variant id to use; otherwise ignored     */
  /* Strided batch (B-GEMM, Sec. 6.7): `batch` independent GEMMs of this
   * shape; item b reads A + b*stride_a, B + b*stride_b and writes
   * C + b*stride_c (strides in elements).  batch 0 or 1: a single GEMM and
   * the strides are ignored.  C items must not overlap each other; A and B
   * items may (stride 0 broadcasts one operand).  Every item obeys the
   * single-GEMM extent limits. */
  int32_t batch;
  int32_t op;                       /* gdy_op: what this entry computes (0: a GEMM)         */
  int64_t stride_a, stride_b, stride_c;
} gdy_gemm;

/* A plan: how a submission is grouped, streamed and bound to variants. */
typedef struct {
  int32_t n;                            /* GEMMs planned                                   */
  int32_t cd;                           /* largest number of GEMMs launched together       */
  int32_t n_groups;                     /* groups run one after another                    */
  int32_t fallback;                     /* 1: no usable GO table, isolated heuristics used  */
  int32_t order[GDY_MAX_GEMMS];         /* launch order: order[t] is a GEMM index          */
  int32_t group_of[GDY_MAX_GEMMS];      /* group of GEMM i                                 */
  int32_t stream_of[GDY_MAX_GEMMS];     /* pool stream slot of GEMM i's dispatch (-1: origin) */
  int32_t variant_of[GDY_MAX_GEMMS];    /* variant id bound to GEMM i (-1: not launched)   */
  int32_t pred_cd[GDY_MAX_GEMMS];       /* selector: min(predicted CD, n) of GEMM i, else 0 */
  int32_t group_size[GDY_MAX_GEMMS];    /* size of group g (first n_groups entries)        */
  int32_t n_dispatches;                 /* kernel dispatches of the submission              */
  int32_t dispatch_of[GDY_MAX_GEMMS];   /* dispatch that runs GEMM i (-1: none); dispatches
                                           are numbered in launch order                    */
  int32_t split_of[GDY_MAX_GEMMS];      /* split-K runs of GEMM i (1: none; 0: not launched) */
} gdy_plan_t;

/*
 * Split-K (all modes; a property of the library's kernels, not of the
 * paper).  A GEMM whose tiles fill at most half of the CU slots its kernel
 * has (CUs x occupancy; a grid cap does not count) and whose K is long runs
 * each tile as S work items over consecutive runs of K tiles: S is the
 * largest power of two up to 16 with S x tiles within the slots, at least
 * 16 K tiles per run and at most 16 MiB of fp32 partial planes; kernels with
 * tiles above 128 x 128 do not split.  S depends only on the GEMM and its
 * kernel -- never on what runs at the same time -- so a variant gives a GEMM
 * the same bits alone and concurrent.  Each run writes an fp32 M x N plane
 * into a workspace the context allocates at creation (256 MiB); a reduction
 * kernel on the dispatch's stream sums the planes in run order, scales,
 * rounds and stores C.  The split GEMMs of a group take consecutive regions
 * of the workspace and groups reuse it (in SEQUENTIAL each GEMM starts at
 * the beginning); a split GEMM that no longer fits in what its group has
 * left moves, with its split, to a group appended after the others (the plan
 * shows it).  Submissions of one context must be ordered (one origin stream
 * at a time): they share the workspace.
 */

/* Static description of one catalogue variant (a kernel plus its grid cap). */
typedef struct {
  char name[64];
  int32_t dtype, trans_a, trans_b;
  int32_t bm, bn, bk;       /* macro tile                                              */
  int32_t waves;            /* waves per workgroup                                     */
  int32_t mfma;             /* MFMA block edge (32 or 16)                              */
  int32_t lds_bytes;        /* LDS per workgroup                                       */
  int32_t vgprs;            /* registers per lane reported by the runtime              */
  int32_t occupancy;        /* workgroups resident per CU (runtime occupancy query)    */
  int32_t grid_cap_cus;     /* 0: one workgroup per tile; else grid = cap * occupancy  */
  int32_t direct;           /* 1: global->LDS copies; needs K % bk == 0 and 16-byte
                               aligned A/B bases and row pitches, else the staged
                               variant of the same tile and cap runs instead     */
  int32_t kind;             /* 0: a GEMM kernel; 1: the element-wise add (GDY_OP_ADD),
                               bm x bn is then its workgroup tile of elements    */
} gdy_variant_desc;

typedef struct gdy_ctx gdy_ctx;

/*
 * Create a context on HIP device `device` (the one-time set-up of Sec. 4.1:
 * the GO library tuned offline for this GPU, Sec. 4.2, and the concurrency
 * the runtime may use).  Loads the catalogue, queries each kernel's
 * occupancy, creates `max_streams` (1..64; 0 means 16) pool streams at
 * default priority and their events, and allocates the split-K workspace.
 * `table_path` names a GO table written by the offline tuner.  Without a
 * usable table -- NULL or "", missing, unreadable, built for another device
 * or naming a variant the library does not have -- the context still
 * returns GDY_OK: SELECTOR and GO modes fall back to isolated heuristics
 * (every GEMM at CD 1, i.e. isolated kernels one after another, Sec. 5.5's
 * sequential configuration) and every plan reports fallback = 1;
 * gdy_last_error() gives the reason until the next call.
 * `use_cu_masks` is a bit set: bit 0 creates one CU-masked stream for each
 * resource constraint GPU/2, GPU/4 and GPU/8 (isolated runs of the tuner);
 * bit 1 creates the CU-Partition streams (2 + 4 + 8 streams whose masks
 * split the CUs into 2, 4 or 8 disjoint parts).  Every stream needs its own
 * hardware queue (a CU mask is a queue property), so GPU_MAX_HW_QUEUES must
 * cover the pool, the masked streams and the caller's streams (24 for a
 * 16-stream pool alone; 32 for an 8-stream pool with partitions).  HIP
 * creates CU-masked streams as blocking streams, so work on the null stream
 * synchronises with all of them: give CU-Partition launches a created
 * origin stream (on the null stream a submission of 8 partitions measured
 * 2-3x slower).  On error *out is NULL.
 *
 * device < 0 creates a host-only context that plans without a GPU: its CU
 * count is GDY_HOST_CUS (default 256) or the loaded table's, kernel
 * occupancy comes from LDS size and wave count alone, the table's device
 * line is not checked, and gdy_execute returns GDY_ERR_UNSUPPORTED.
 */
gdy_status gdy_create(gdy_ctx** out, int device, const char* table_path, int32_t max_streams,
                      int32_t use_cu_masks);

/*
 * Resource constraint for subsequent launches (Sec. 4.2.1 "RC tuning"):
 * 0 = whole GPU; 128, 64 or 32 = launches that go to pool streams run on
 * the CU-masked streams restricted to that many CUs (needs use_cu_masks
 * bit 0 at create).  Pool streams carry every dispatch of GDY_DEFAULT and
 * GDY_FORCED (the tuner's isolated runs use GDY_FORCED with forced_cd 1)
 * and the further dispatches of a group; what runs on the caller's origin
 * stream (GDY_SEQUENTIAL, a group's first dispatch) is not masked.  Other
 * values: GDY_ERR_INVALID_ARG.
 */
gdy_status gdy_set_rc(gdy_ctx* ctx, int32_t budget_cus);

/* Destroy a context: synchronises its streams, then frees streams and events. */
void gdy_destroy(gdy_ctx* ctx);

/*
 * Plan a submission without touching device memory (pointers are validated
 * for null/alias only and never dereferenced).  Sec. 4.3 dynamic logic for
 * SELECTOR; see gdy_mode for the others.  forced_cd: GO and FORCED modes
 * (0 = n); ignored otherwise.
 */
gdy_status gdy_plan(gdy_ctx* ctx, const gdy_gemm* gemms, int32_t n, int32_t mode,
                    int32_t forced_cd, gdy_plan_t* out);

/*
 * Plan and launch a submission: the problem statement of Sec. 4.1 -- given a
 * set of independent GEMMs, predict a performant CD and schedule that many
 * GEMMs at a time with the kernels tuned for it (SELECTOR, Sec. 4.3), or run
 * one of the other execution configurations of Sec. 5.5 (see gdy_mode).
 * `gemms` (host array of n descriptors, read during the call only) names
 * caller-owned device buffers.  Asynchronous to the host: the work is
 * ordered after what is already on `hip_stream` (a hipStream_t; NULL is the
 * null stream) and `hip_stream` is ordered after all of it when this
 * returns.  `out` (nullable) receives the plan.  Every descriptor is
 * validated before anything launches (all or nothing).  On GDY_ERR_HIP the
 * streams are still joined back to the origin stream.
 */
gdy_status gdy_execute(gdy_ctx* ctx, const gdy_gemm* gemms, int32_t n, int32_t mode,
                       int32_t forced_cd, void* hip_stream, gdy_plan_t* out);

/*
 * gdy_execute for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation):
 * the same plan and the same kernels as gdy_execute, with the split-K
 * planes in a static device array of GDY_STATIC_SCRATCH_BYTES that the
 * library holds on every device it runs on until the process ends, instead
 * of the context's workspace.  Allocates nothing, on the device or through
 * any allocating library routine.  A plan whose split GEMMs need more than
 * the array at once (one group's planes; one GEMM's in SEQUENTIAL) returns
 * GDY_ERR_UNSUPPORTED before anything launches.  Every call on a device
 * shares that device's array, which keeps the last call's partial planes
 * (each run overwrites its plane before the reduction reads it, so nothing
 * needs clearing): calls that overlap on one device, from any context or
 * thread, race and must be ordered by the caller.  Results are bit-identical
 * to gdy_execute's.
 */
#define GDY_STATIC_SCRATCH_BYTES (64ll * 1024 * 1024)
gdy_status gdy_execute_static(gdy_ctx* ctx, const gdy_gemm* gemms, int32_t n, int32_t mode,
                              int32_t forced_cd, void* hip_stream, gdy_plan_t* out);

/*
 * Per-kernel timing (Sec. 5.3 measures each GEMM's kernel runtime, with the
 * GEMMs run back-to-back on their streams).  When enabled, every dispatch
 * of gdy_execute records a start and a stop event on the stream it runs on
 * (hipExtLaunchKernel), and a submission start event on the origin stream.
 * After the caller has synchronised, gdy_last_kernel_times fills
 * start_ms[i] / end_ms[i] (host arrays of n floats; milliseconds from the
 * submission start) for GEMM i of the last submission; GEMMs that launched
 * nothing get -1.  GEMMs that share a dispatch report that dispatch's
 * interval (a split GEMM's interval ends with its reduction).
 * GDY_ERR_INVALID_ARG when no timed submission exists or a pointer is NULL.
 */
gdy_status gdy_set_timing(gdy_ctx* ctx, int32_t enable);
gdy_status gdy_last_kernel_times(gdy_ctx* ctx, float* start_ms, float* end_ms, int32_t n);
/* Same for an earlier timed submission: back = 0 is the last one, up to 63
 * (the context keeps the events of the last 64 timed submissions). */
gdy_status gdy_kernel_times(gdy_ctx* ctx, int32_t back, float* start_ms, float* end_ms,
                            int32_t n);

/*
 * Dispatch map (host only; works on host-only contexts): plans the
 * submission as gdy_plan does, builds launch block `dispatch` of the plan
 * as gdy_execute would, and reports what each of its workgroups computes,
 * with the kernels' own mapping code.  *grid receives the dispatch's
 * workgroup count; for workgroup b < min(*grid, max_workgroups),
 * gemm_of_wg[b] is the submission index of the member it serves (-1: an
 * idle workgroup) and it runs that member's work items first_item[b],
 * first_item[b] + item_stride[b], ... below the member's item count.
 * items_of_gemm (n entries) receives each member's work items in this
 * dispatch (tiles x batch items x split runs; 0 for GEMMs of other
 * dispatches).  Lets a caller check on the CPU that every work item of a
 * dispatch is computed exactly once (XCD placement included).
 */
gdy_status gdy_dispatch_map(gdy_ctx* ctx, const gdy_gemm* gemms, int32_t n, int32_t mode, int32_t forced_cd,
                            int32_t dispatch, int32_t max_workgroups, int32_t* grid, int32_t* gemm_of_wg,
                            int32_t* first_item, int32_t* item_stride, int64_t* items_of_gemm);

/* Features of one GEMM (Sec. 4.3): M, N, K, then for each CD class
 * 1, 2, 4, 8, 16 the bound variant's #WGs, occupancy and #waves. */
gdy_status gdy_features(gdy_ctx* ctx, const gdy_gemm* gemm, double* out_features);

/* Catalogue queries.  Variant ids are 0 .. gdy_variant_count()-1. */
int32_t gdy_variant_count(gdy_ctx* ctx);
gdy_status gdy_variant_info(gdy_ctx* ctx, int32_t id, gdy_variant_desc* out);
int32_t gdy_variant_find(gdy_ctx* ctx, const char* name); /* -1 if absent */
/* Isolated (CD 1) variant the library binds to a GEMM, from the table or heuristics. */
int32_t gdy_isolated_variant(gdy_ctx* ctx, const gdy_gemm* gemm);
/* FNV-1a hash of the catalogue's variant names, as stored in GO tables. */
uint64_t gdy_catalogue_hash(gdy_ctx* ctx);
/* Number of compute units of the context's device. */
int32_t gdy_device_cus(gdy_ctx* ctx);

const char* gdy_status_string(gdy_status s);
const char* gdy_last_error(gdy_ctx* ctx); /* valid until the next call on ctx; "" if none */

#ifdef __cplusplus
}
#endif

#endif /* GDY_H */
