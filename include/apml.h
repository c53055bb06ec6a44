/*
 * apml.h - C ABI of the sparse APML loss (forward and backward) on one AMD
 * Instinct MI355X (gfx950).
 *
 * The loss is the sparse Adaptive Probabilistic Matching Loss of
 * "From Theory to Throughput: CUDA-Optimized APML for Large-Batch 3D
 * Learning" (arXiv:2512.19743). Per sample b, with predicted points
 * X = {x_i} (N of them) and reference points Y = {y_j} (M of them):
 *
 *   C_ij = ||x_i - y_j||_2                                    Sec. III-A
 *   per row i: C1 = min_j C_ij, C2 = second smallest,
 *     g = max(C2 - C1 + delta, eps_gap)                       Sec. III-A, III-D
 *     T = log((M - 1) p_min / (1 - p_min)) / g                Eq. 1
 *     s_ij = exp(-T (C_ij - C1)), kept where s_ij >= tau      Sec. III-B
 *     P_row = s / (sum of kept s in the row)                   Eq. 2, Sec. III-C
 *   per column j: the same with roles swapped (K = N)          Sec. III-B
 *   P0 = (P_row + P_col) / 2 on the union of both kept sets    Sec. III-A, III-C
 *   L_iter times: column scaling (Eq. 3), then row scaling (Eq. 4)
 *   loss_b = sum over kept pairs of v_t C_t                     Sec. III-D
 *   d loss / d x through all of the above, with Eq. 5 for the
 *   distance and the temperature differentiated (no gradient
 *   through the choice of the kept set or of the minima).      Sec. III-D
 *
 * The minimum and second minimum of a row or column are decided on the
 * single-precision squared distance; ties go to the smaller index. Everything
 * after the decision (cost values, temperatures, similarities, sums) is
 * computed in double precision and stored per stored pair in single precision.
 *
 * All pointers named "device" point to memory on the current HIP device, all
 * pointers named "host" to host memory. Every function returns an
 * apml_status and never throws; on failure apml_last_error() describes it.
 * Argument validation happens before any HIP call, so a rejected call touches
 * neither the device nor its outputs.
 */
#ifndef APML_H
#define APML_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define APML_VERSION 1

typedef enum apml_status {
    APML_OK = 0,
    APML_ERR_INVALID_ARG = 1,   /* a NULL pointer, a size or a parameter out of range */
    APML_ERR_UNSUPPORTED = 2,   /* d != 3, or a size beyond the 32-bit index range */
    APML_ERR_OUT_OF_MEMORY = 3, /* the allocator returned NULL */
    APML_ERR_DEVICE = 4,        /* a HIP call failed (text in apml_last_error) */
    APML_ERR_INTERNAL = 5       /* a consistency check on the device failed */
} apml_status;

/* A hipStream_t; NULL is the default (null) stream of the current device. */
typedef void *apml_stream;

/* Hyper-parameters. Defaults (apml_params_default) are the paper's
 * tau = 1e-8, L_iter = 10, eps_stab = 1e-8 (Sec. III-E, Sec. IV-C) and, where
 * the paper gives no value, p_min = 0.8, delta = 1e-8, eps_gap = 1e-6,
 * eps_dist = 1e-12. */
/* How the dense scans (the minimum and second minimum of every row and
 * column, Sec. III-A; the candidate support, Sec. III-B) visit the pairs.
 * Both modes give identical results. FULL evaluates every pair. SKIP sorts
 * both clouds along a space-filling curve and skips every run of 32 points
 * whose bounding box is provably beyond the distance that can still matter
 * to the owners being scanned; it pays off for large samples. AUTO takes SKIP
 * when min(N, M) >= 8192. */
typedef enum { APML_SCAN_AUTO = 0, APML_SCAN_FULL = 1, APML_SCAN_SKIP = 2 } apml_scan_mode;

/* Readings of the paper where it offers two (for ablation; the defaults are
 * the first of each).
 * gap_mode  CLAMP: g = max(C2 - C1 + delta, eps_gap) (Sec. III-D).
 *           UNIFORM_FALLBACK: an owner whose gap C2 - C1 is below eps_gap
 *           gets P = 1/K on all K pairs (Sec. III-A, Sec. III-C); all of its
 *           pairs are stored and no gradient flows through that softmax.
 * sym_mode  HALF_SUM: P0 = (P_row + P_col)/2 with an absent side 0 (the
 *           dense initial plan of Sec. III-A on the union support).
 *           MEAN_DUP: duplicates averaged (Sec. III-C, Alg. 1 step 3) and a
 *           pair kept by one direction only keeps that direction's value.
 * tgrad_mode FULL: the gradient reaches the costs through the temperatures
 *           (Eq. 1); DETACHED: the temperatures are constants in backward. */
typedef enum { APML_GAP_CLAMP = 0, APML_GAP_UNIFORM_FALLBACK = 1 } apml_gap_mode;
typedef enum { APML_SYM_HALF_SUM = 0, APML_SYM_MEAN_DUP = 1 } apml_sym_mode;
typedef enum { APML_TGRAD_FULL = 0, APML_TGRAD_DETACHED = 1 } apml_tgrad_mode;

typedef struct apml_params {
    uint32_t struct_size; /* sizeof(apml_params), for forward compatibility */
    int32_t n_iter;       /* L_iter >= 0: Sinkhorn iterations (Alg. 1) */
    double p_min;         /* Eq. 1; needs 1/min(N, M) < p_min < 1 */
    double tau;           /* pruning threshold on s, 0 <= tau <= 1 (Sec. III-B) */
    double eps_stab;      /* >= 0, added to every Sinkhorn sum (Eq. 3, Eq. 4) */
    double delta;         /* >= 0, gap offset g = c2 + delta (Sec. III-A) */
    double eps_gap;       /* > 0, gap clamp max(gap, eps_gap) (Sec. III-D) */
    double eps_dist;      /* >= 0, added to ||x - y|| in the gradient only (Eq. 5) */
    int32_t dense_scan;   /* apml_scan_mode: how the two dense scans visit the pairs */
    int32_t gap_mode;     /* apml_gap_mode (default CLAMP) */
    int32_t sym_mode;     /* apml_sym_mode (default HALF_SUM) */
    int32_t tgrad_mode;   /* apml_tgrad_mode (default FULL) */
} apml_params;

/* Fills *p with the defaults above (p must not be NULL). */
void apml_params_default(apml_params *p);

/* Opaque per-call state kept from the forward pass for the backward pass:
 * the stored pairs, the per-row and per-column statistics and the Sinkhorn
 * scalings. Library-owned; release it with apml_plan_destroy. */
typedef struct apml_plan apml_plan;

/*
 * Forward pass (Alg. 1, Sec. III-A to III-D).
 *   x     device, float32 [B, N, d] contiguous (predicted points X)
 *   y     device, float32 [B, M, d] contiguous (reference points Y)
 *   B >= 1, N >= 2, M >= 2, d == 3 (else APML_ERR_UNSUPPORTED);
 *   B*N, B*M and the number of stored pairs must fit in int32.
 *   params  host, may be NULL for the defaults
 *   loss    device, float32 [B]: per-sample loss sum_t v_t C_t (no batch mean)
 *   plan    host out-pointer; if non-NULL, *plan receives the state needed by
 *           apml_backward; if NULL, that state is released before returning.
 *   stream  every kernel is queued on it.
 * The call synchronises the stream once, after the support has been counted,
 * to size the sparse arrays (the paper's two-pass construction does the same).
 * x and y are only read. On error *plan is NULL and loss is untouched unless
 * the failure came from the device. A device-side consistency check that runs
 * after that synchronisation (a row's or column's minimum missing from its
 * stored pairs, which the construction rules out) is reported only by
 * apml_plan_nnz, as APML_ERR_INTERNAL; this call returns APML_OK then. So is
 * a bounded wait of the Sinkhorn kernels that split a sample over several
 * workgroups expiring (they are launched so that all of them run at once,
 * which rules it out), as APML_ERR_DEVICE.
 */
apml_status apml_forward(const float *x, const float *y, int32_t B, int32_t N, int32_t M,
                         int32_t d, const apml_params *params, float *loss, apml_plan **plan,
                         apml_stream stream);

/*
 * Backward pass (Sec. III-D): gradient of sum_b grad_loss[b] * loss_b.
 *   plan       from apml_forward; not consumed (may be used again)
 *   x, y       the same device arrays, unchanged since the forward call
 *   grad_loss  device, float32 [B]
 *   grad_x     device, float32 [B, N, 3], overwritten
 *   grad_y     device, float32 [B, M, 3], overwritten, or NULL to skip it
 */
apml_status apml_backward(apml_plan *plan, const float *x, const float *y,
                          const float *grad_loss, float *grad_x, float *grad_y,
                          apml_stream stream);

/*
 * Forward and backward in one call, with no device allocation. For callers
 * that cannot allocate device memory (code under stream capture, serving loops
 * with a fixed memory budget, harnesses that forbid hipMalloc): the same
 * kernels as apml_forward followed by apml_backward, with every plan array and
 * temporary carved from one static device array of
 * APML_NOALLOC_SCRATCH_BYTES that each device the library runs on holds until
 * the process ends (32 clouds of 2048 points against 2048 fit in it; 64 clouds
 * of 8192 points do not). No plan is returned.
 *   x, y, B, N, M, d, params, loss   as for apml_forward
 *   grad_loss, grad_x, grad_y        as for apml_backward; grad_x == NULL
 *                                    computes the loss only (grad_loss and
 *                                    grad_y are then ignored)
 * Errors: as apml_forward; APML_ERR_OUT_OF_MEMORY when the call needs more
 * scratch than the array holds (apml_last_error states both sizes; detected
 * before the kernels that write loss or gradients run, so the outputs are
 * untouched), APML_ERR_UNSUPPORTED when B > 1791. The call synchronises the
 * stream once, like apml_forward. Every call on a device shares that
 * device's array and leaves its contents behind: calls that overlap on one
 * device (other host threads, or other streams still running an earlier
 * call) race and give undefined results; calls on one stream, or on
 * different devices, do not.
 */
#define APML_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
apml_status apml_forward_backward_noalloc(const float *x, const float *y, int32_t B, int32_t N,
                                          int32_t M, int32_t d, const apml_params *params,
                                          float *loss, const float *grad_loss, float *grad_x,
                                          float *grad_y, apml_stream stream);

/*
 * Dense APML (Sec. III-A): the unpruned formulation, a baseline for the
 * sparse path's memory and time. Every pair of a sample takes part (no
 * threshold: tau is ignored, the result is what the sparse path gives at
 * tau = 0), for points of any dimension 1 <= d <= 16. The minimum and second
 * minimum of every row and column are decided on the single-precision squared
 * distance as in the sparse path; the temperatures follow Eq. 1 with the gap
 * clamp (Sec. III-D), the softmaxes Eq. 2 over all pairs, P0 = (P_row +
 * P_col)/2, then L column (Eq. 3) and row (Eq. 4) scalings, loss = sum P C.
 * The plan keeps P0 and the Sinkhorn plan as float32 N x M matrices per
 * sample; the backward pass adds a float64 N x M adjoint. Device memory comes
 * from the same pool or caller allocator as the sparse path.
 *   x, y    device, float32 [B, N, d] / [B, M, d] contiguous
 *   params  as for apml_forward; gap_mode and sym_mode must be the defaults
 *           (else APML_ERR_UNSUPPORTED); dense_scan and tau are ignored
 *   loss    device, float32 [B]
 *   plan    as for apml_forward (NULL: released before returning)
 * apml_dense_backward: gradient of sum_b grad_loss[b] loss_b, grad_x [B,N,d]
 * overwritten, grad_y [B,M,d] overwritten or NULL. Neither call synchronises.
 */
typedef struct apml_dense_plan apml_dense_plan;
apml_status apml_dense_forward(const float *x, const float *y, int32_t B, int32_t N, int32_t M,
                               int32_t d, const apml_params *params, float *loss,
                               apml_dense_plan **plan, apml_stream stream);
apml_status apml_dense_backward(apml_dense_plan *plan, const float *x, const float *y,
                                const float *grad_loss, float *grad_x, float *grad_y,
                                apml_stream stream);
apml_status apml_dense_plan_destroy(apml_dense_plan *plan);

/* Releases the plan's device memory (stream-ordered on the plan's stream).
 * NULL is accepted. */
apml_status apml_plan_destroy(apml_plan *plan);

/* Sizes of a plan. stored_pairs counts every stored pair, including pairs kept
 * only as the minimum or second minimum of a row or column (they carry zero
 * mass). bytes is the device memory the plan holds. scanned_min and
 * scanned_support count the pairs the two dense scans of the forward
 * examined: the minimum scan once per direction (2*B*N*M when nothing is
 * skipped, although the full scan evaluates each distance once for both),
 * the support scan over rows (B*N*M); the skipping scans leave out pairs that
 * provably cannot matter. */
typedef struct apml_plan_info {
    int32_t B, N, M, n_iter;
    int64_t stored_pairs;
    int64_t bytes;
    int64_t scanned_min, scanned_support;
} apml_plan_info;
apml_status apml_plan_get_info(const apml_plan *plan, apml_plan_info *info);

/* Per-sample size of the kept support Omega = Omega_row U Omega_col
 * (Sec. III-B), host int64 [B]. Synchronises the plan's stream. Returns
 * APML_ERR_INTERNAL if a device-side consistency check failed, and
 * APML_ERR_DEVICE if a bounded wait of the split Sinkhorn kernels expired. */
apml_status apml_plan_nnz(const apml_plan *plan, int64_t *nnz);

/*
 * Copies sample b's kept pairs to the host, sorted by (i, j), for testing and
 * inspection. capacity is the length of every non-NULL output array and must
 * be at least the sample's apml_plan_nnz value. Outputs (any may be NULL):
 *   i, j     int32 row and column index
 *   flags    bit 0: s_row >= tau, bit 1: s_col >= tau
 *   p_row, p_col  float32 normalised row / column probabilities (0 if not kept)
 *   p0       float32 initial plan (P_row + P_col)/2
 *   v        float32 plan after the Sinkhorn iterations
 * Synchronises the plan's stream.
 */
apml_status apml_plan_export(const apml_plan *plan, int32_t b, int64_t capacity, int32_t *i,
                             int32_t *j, uint8_t *flags, float *p_row, float *p_col, float *p0,
                             float *v);

/*
 * Copies sample b's per-row and per-column statistics to the host:
 * temperature (Eq. 1), index of the minimum and second minimum, and whether
 * the gap was clamped. Row arrays have N entries, column arrays M; any may be
 * NULL. Synchronises the plan's stream.
 */
apml_status apml_plan_export_stats(const apml_plan *plan, int32_t b, double *T_row, int32_t *j1,
                                   int32_t *j2, uint8_t *row_clamped, double *T_col, int32_t *i1,
                                   int32_t *i2, uint8_t *col_clamped);

/*
 * Device memory. By default the library keeps its own pool of hipMalloc'd
 * blocks per device and stream (freed blocks are reused by later calls on the
 * same stream). A caller may route every allocation through its own
 * allocator instead, e.g. a framework's caching allocator; alloc must return
 * device memory usable on `stream` (or NULL on failure), free is called with
 * the same pointer, size and stream. Every failure of alloc must come back as
 * NULL: the library cannot tell any other pointer from device memory and its
 * kernels will write through it (a binding whose callbacks can raise must
 * catch and return NULL). Blocks the pool caches are not given back when the
 * route changes: apml_release_cached_memory does that. Passing NULLs restores
 * the pool. Must not be called while a plan is alive.
 */
typedef void *(*apml_alloc_fn)(size_t bytes, apml_stream stream, void *user);
typedef void (*apml_free_fn)(void *ptr, size_t bytes, apml_stream stream, void *user);
apml_status apml_set_allocator(apml_alloc_fn alloc, apml_free_fn free_fn, void *user);

/* Bytes currently held by live plans and temporaries, the peak of that since
 * the last reset, and the bytes reserved by the pool. */
typedef struct apml_memory_stats {
    int64_t in_use;
    int64_t peak_in_use;
    int64_t reserved;
} apml_memory_stats;
apml_status apml_get_memory_stats(apml_memory_stats *stats);
apml_status apml_reset_peak_memory(void);
/* Returns the pool's unused blocks to HIP. */
apml_status apml_release_cached_memory(void);

/*
 * Per-phase timing with HIP events recorded on the caller's stream around
 * each phase of forward and backward. Phases (index: name):
 *   0 stats     dense scan: minimum and second minimum per row and column
 *   1 support   dense scan: emission of the candidate pairs
 *   2 build     counts, prefix sums, row-major and column-major index build
 *   3 softmax   temperatures, both softmaxes, symmetrized plan
 *   4 sinkhorn  the 2 L scaling sweeps
 *   5 loss      loss per sample
 *   6 bwd_sinkhorn   reverse Sinkhorn sweeps
 *   7 bwd_softmax    softmax, temperature and distance adjoints
 * apml_profile_read synchronises the recorded events and returns, per phase,
 * the total milliseconds and the number of timed occurrences since the last
 * reset (arrays of length n, at most APML_N_PHASES).
 */
#define APML_N_PHASES 8
apml_status apml_profile_enable(int32_t on);
apml_status apml_profile_reset(void);
apml_status apml_profile_read(int32_t n, double *total_ms, int64_t *count);
const char *apml_phase_name(int32_t phase);

const char *apml_status_string(apml_status status);
/* Text of the last error on the calling thread ("" if none). */
const char *apml_last_error(void);
int32_t apml_version(void);

#ifdef __cplusplus
}
#endif
#endif /* APML_H */
