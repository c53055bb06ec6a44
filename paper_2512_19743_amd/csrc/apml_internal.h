// Internal declarations shared by the kernels and the host orchestration of
// libapml. Not part of the public ABI (include/apml.h is).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace apml {

constexpr int kBlock = 256;       // threads per workgroup of the grid-wide kernels
constexpr int kGroup = 4;         // lanes per row / column in the sparse kernels

constexpr int kScanSlots = 64;

// Device-side counters of one forward call (cleared by the first kernel that
// runs after them: the full scan's finalize kernel or the spatial sort).
struct Counters {
    unsigned int error;            // bit 0: a row's minima not found among its pairs; bit 1: a column's;
                                   // bit 2: a meeting of the split streamed Sinkhorn kernels timed out
    unsigned int overflow;         // a tile of the full support scan (a row of the skipping one) is written by
                                   // a second pass: its further hits did not fit
    // pairs evaluated by the skipping scans (minimum scan, support scan), in
    // kScanSlots partial sums: workgroup w adds to slot w % kScanSlots, so
    // that no single address takes every workgroup's atomic
    unsigned long long scanned[2][kScanSlots];
    // entries requested from the full support scan's pool of further hits
    // (64-bit: tiles that find the pool full still add theirs)
    unsigned long long spill_fill;
};

struct Params {
    double p_min, tau, eps_stab, delta, eps_gap, eps_dist;
    double log_inv_tau;    // log(1/tau); +inf when tau == 0
    double lk_row, lk_col; // -log((1-p) / ((K-1) p)) for rows (K = M) and columns (K = N)
    int n_iter;
    int gap_mode, sym_mode, tgrad_mode; // apml_gap_mode, apml_sym_mode, apml_tgrad_mode
};

constexpr int kGapFallback = 1;  // APML_GAP_UNIFORM_FALLBACK
constexpr int kSymMeanDup = 1;   // APML_SYM_MEAN_DUP
constexpr int kTgradDetached = 1; // APML_TGRAD_DETACHED

// Squared radius of an owner's emission ball from its single-precision
// minimum and second minimum m1 <= m2 (log_ratio: Eq. 1's numerator for the
// owner's direction). The kept set s >= tau is the ball C <= C1 + log(1/tau)/T
// (Sec. III-B, Eq. 1); the margin covers the rounding of this estimate
// (relative ~1e-7 (1 + 2 kappa)) and of the single-precision distance; the
// second minimum is always inside. An owner that may take the uniform
// fallback (its gap within rounding of eps_gap: the fp32 costs differ from
// the double ones by ~1.2e-7 relative) gets an infinite radius: every pair is
// a candidate, and the softmax decides in double precision.
__device__ inline double emission_radius2(float m1, float m2, double log_ratio, const Params &p)
{
    const double c1 = sqrt((double)m1), c2 = sqrt((double)m2);
    if (p.gap_mode == kGapFallback && (c2 - c1) < p.eps_gap + 1e-5 * (c1 + c2))
        return HUGE_VAL;
    const double gap = (c2 - c1) + p.delta;
    const double g = gap < p.eps_gap ? p.eps_gap : gap;
    const double kappa = p.log_inv_tau / log_ratio; // log(1/tau) / (T g)
    const double radius = c1 + g * kappa;
    const double margin = 1e-5 * (1.0 + kappa);
    const double e = radius * radius * (1.0 + margin);
    return fmax(e, (double)m2);
}

// ---------------------------------------------------------------------------
// dense phase
// ---------------------------------------------------------------------------

// One direction of the dense minimum / second-minimum scan. Owners are the
// points whose statistics are computed (X for rows, Y for columns); the
// broadcast set is scanned against every owner.
// Columns of a support-scan chunk are a multiple of this.
constexpr int kUnroll = 8;

struct FinalizeDir {
    const float2 *partial; // [S][B * n_own]
    const float *own;      // owner coordinates [B, n_own, 3]
    float2 *m12;           // out: (m1, m2) per owner
    float *E;              // out (rows): emission threshold on the squared distance
    float4 *packed;        // out (columns): (x, y, z, emission threshold)
    int32_t *zero_a, *zero_b; // (columns) per-owner counters cleared here
    int n_own, S;
    double log_ratio;      // -log((1-p)/((K-1)p)), K = length of the other set
};


// The minimum scan with one evaluation per pair (k_top2_pairs): each
// workgroup takes a block of 64 kPairR rows (x) and one chunk of columns (y);
// its per-row partials are the row direction's chunk partials (S = S_r), its
// per-column partials those of the column direction (S = S_c, one per row
// block).
constexpr int kPairR = 8;            // rows per lane
constexpr int kPairWaves = 4;        // waves per workgroup (a quarter of the chunk each)
constexpr int kPairThreads = 64 * kPairWaves;
constexpr int kPairMaxChunk = 4096;  // columns per chunk at most
constexpr int kPairTargetWaves = 8192;
struct PairScan {
    const float *x, *y;  // [B, N, 3], [B, M, 3]
    float2 *row_partial; // [S_r][B * N]
    float2 *col_partial; // [S_c][B * M]
    int B, N, M;
    int chunk, S_r;      // columns per chunk (a multiple of 32) and chunks
    int S_c;             // row blocks of 64 kPairR rows
};
void choose_pair_scan(PairScan &p, int B, int N, int M);
void launch_top2_pairs(const PairScan &p, hipStream_t s);
void launch_finalize(const FinalizeDir &rows, const FinalizeDir &cols, int B, const Params &p,
                     Counters *ctr, hipStream_t s);

// The counting pass of the support scan keeps the first kst hits of every
// (row, chunk) (kst = stage_slots(S), at most kStage: fewer when the columns
// are cut into many chunks, each of which then holds few of a row's hits).
// The further hits of a tile (kBlock rows, one chunk), up to kTileList, are
// collected in LDS and, once the tile is scanned, written row by row into a
// region of a shared pool (kSpillPerTile 16-bit entries per tile on
// average): kBlock row starts, then the hits. Only a tile whose hits exceed
// its list or find the pool full is scanned again by the writing pass.
constexpr int kStage = 16;
constexpr int kTileList = 2048;
constexpr int kSpillPerTile = 1024;
inline int stage_slots(int S) { return S >= 32 ? 2 : S >= 16 ? 4 : S >= 8 ? 8 : kStage; }

struct EmitArgs {
    const float *x;      // [B, N, 3]
    const float4 *ypack; // [B, M]: y and its column threshold
    const float *E_row;  // [B*N]
    int B, N, M, S, chunk, owner_blocks;
    int32_t *cnt;        // [B*N][S] stored pairs per (row, column chunk)
    int32_t *col_cnt;    // [B*M] stored pairs per column
    uint16_t *stage;     // [B*N][S][kst] column offsets within the chunk of the first hits, or NULL;
                         // one byte each when stage_narrow (chunks of at most 256 columns)
    int kst;             // staged hits per (row, chunk)
    int stage_narrow;
    uint16_t *spill;     // pool of further hits: per tile kBlock row starts, then the offsets in the chunk
    int64_t spill_cap;   // entries of the pool
    int32_t *spill_base; // [tiles]: the tile's region in the pool; -1: the tile is scanned again
    Counters *ctr;
    // second pass (or compaction of the staged hits)
    const int32_t *row_ptr; // [B*N+1]
    int32_t *csr_col, *csr_row;
    // column-major placement done by the compaction (when no tile is rescanned)
    const int32_t *col_ptr; // [B*M+1]
    int32_t *col_fill;      // [B*M], zero
    int32_t *tmp_row, *tmp_src, *csc_col;
};
// Pass 1 counts the candidate support per (row, chunk) and per column; pass 2
// (after the offsets are known) writes it into the CSR arrays.
void launch_emit_count(const EmitArgs &a, hipStream_t s);
void launch_emit_write(const EmitArgs &a, hipStream_t s);
// Writes the CSR from the staged hits of every tile whose list did not
// overflow; with overflow set, the writing pass then rescans only the tiles
// whose list overflowed.
struct DevPlan;
// place: the compaction also takes each pair's column slot. pieces_place
// (non-NULL, with place false): the same launch also places the pieces of the
// per-sample Sinkhorn kernels (place_order) for plan d.
void launch_emit_compact(const EmitArgs &a, bool overflow, bool place, const DevPlan *d, int32_t *pieces_place,
                         hipStream_t s);

// The skipping scans (cull.hip), for large samples. Both clouds are sorted
// along a Hilbert curve per sample (spatial.hip). A sorted cloud is [B][pad]
// float4 (x, y, z, original index as bits), pad = the point count rounded up
// to a multiple of 64, with the bounding box of every run of kRun consecutive
// points ([B][pad / kRun]). The scans skip every run whose box is provably
// too far from the box of their rows.
constexpr int kRun = 32;      // points per box
constexpr int kScanRows = 64; // owners per wave of the dense scans (one per lane)
inline int pad64(int n) { return (n + 63) / 64 * 64; }

struct Box {
    float4 lo, hi; // hi.w: (columns, after the finalize kernel) the largest emission threshold of the run
};

struct SpatialArgs {
    const float *x, *y; // [B, N, 3], [B, M, 3]
    int B, N, M, pad_x, pad_y;
    uint32_t *key[2], *val[2]; // scratch: [B * pad_x + B * pad_y] each
    float *frame_part;         // scratch [B][frame_slices][6] when a cloud exceeds one sort chunk, else NULL
    int frame_slices;
    float4 *sx, *sy;           // out: sorted clouds
    Box *box_x, *box_y;        // out: boxes of the runs
    Counters *ctr;             // cleared here
};
// Batches of 64 runs (2048 sorted points): the scans test a batch's box
// before its runs'.
__host__ __device__ inline int batches(int pad) { return (pad / kRun + 63) / 64; }
// The box of every batch of runs of both sorted clouds (columns_only: of the
// columns, hi.w the largest of the runs' hi.w).
void launch_batch_boxes(const Box *box_x, const Box *box_y, Box *batch_x, Box *batch_y, int B, int pad_x, int pad_y,
                        bool columns_only, hipStream_t s);
size_t spatial_sort_lds();
// Points one workgroup of the spatial sort takes; larger clouds are sorted in
// chunks, then merged.
constexpr int kSortChunkPoints = 8192;
hipError_t launch_spatial_sort(const SpatialArgs &a, hipStream_t s);

// One direction of the minimum / second-minimum scan: owners (X for rows, Y
// for columns) against every point of the other cloud.
struct CullDir {
    const float4 *own, *bc; // sorted owners [B][pad_own] and other cloud [B][pad_bc]
    const Box *own_box;     // [B][pad_own / kRun]
    const Box *bc_box;      // [B][pad_bc / kRun]
    const Box *bc_batch;    // [B][batches(pad_bc)]: union of the boxes of 64 consecutive runs
    float2 *m12s;           // out [B][pad_own]: (min, second min) of the squared distance, sorted position
    int n_own, n_bc, pad_own, pad_bc;
    int waves;              // per sample: ceil(n_own / kScanRows)
};

struct CullFinalizeDir {
    const float2 *m12s;       // [B][pad]
    const float4 *own;        // sorted owners [B][pad]
    float2 *m12;              // out: (m1, m2) per owner, original order [B * n_own]
    float *E;                 // out (rows): emission threshold on the squared distance, sorted [B][pad]
    float4 *packed;           // out (columns): (x, y, z, emission threshold), sorted [B][pad]
    Box *box;                 // (columns) hi.w of every run: its largest threshold
    int32_t *zero_a, *zero_b; // (columns) per-owner counters cleared here, original order
    int n_own, pad;
    double log_ratio;         // -log((1-p)/((K-1)p)), K = length of the other set
};

void launch_cull_top2(const CullDir &rows, const CullDir &cols, int B, Counters *ctr, hipStream_t s);
void launch_cull_finalize(const CullFinalizeDir &rows, const CullFinalizeDir &cols, int B, const Params &p,
                          hipStream_t s);

struct CullEmitArgs {
    const float4 *sx;    // sorted rows [B][pad_x]
    const float *E;      // their thresholds [B][pad_x]
    const float4 *yp;    // sorted columns with their thresholds [B][pad_y]
    const float4 *sy;    // sorted columns with their original index [B][pad_y]
    const Box *box_x;    // [B][pad_x / kRun]
    const Box *box_y;    // [B][pad_y / kRun]
    const Box *batch_y;  // [B][batches(pad_y)]: union of 64 runs' boxes, hi.w their largest column threshold
    int B, N, M, pad_x, pad_y, waves;
    int32_t *cnt;        // [B*N] stored pairs per row
    int32_t *col_cnt;    // [B*M] stored pairs per column
    int32_t *stage;      // [B*N][kCullStage] the first columns of each row, in scan order
    uint8_t *wg_over;    // [B * waves] a row of this workgroup has more than kCullStage pairs
    Counters *ctr;       // overflow: some row has more than kCullStage pairs
    // writing pass (rows beyond the staging only) and ordering
    const int32_t *row_ptr; // [B*N+1]
    int32_t *tmp_col;       // [nnz] the columns of those rows in scan order
    int32_t *csr_col, *csr_row;
    int64_t nnz;
};
constexpr int kCullStage = 16;
// Pass 1 counts the candidate support per row and per column and keeps each
// row's first kCullStage columns; the ordering writes every row that fits
// there in increasing column order and (pieces_place non-NULL) places the
// pieces of the per-sample Sinkhorn kernels (place_order) in the same
// launch. Only when a row overflowed does pass 2 (after the offsets are known)
// write the columns of the overflowing rows, which a ranking then orders.
void launch_cull_emit_count(const CullEmitArgs &a, hipStream_t s);
void launch_cull_emit_write(const CullEmitArgs &a, hipStream_t s);
void launch_cull_emit_order(const CullEmitArgs &a, const DevPlan *d, int32_t *pieces_place, hipStream_t s);
void launch_cull_emit_rank(const CullEmitArgs &a, hipStream_t s);

// ---------------------------------------------------------------------------
// sparse structure
// ---------------------------------------------------------------------------


// Pieces of the per-sample Sinkhorn kernels. Each row's (column's) pairs are
// cut into pieces of kSinkPiece consecutive pairs; an owner with n pieces
// takes a group of 2^ceil(log2 n) consecutive positions (padding pieces are
// empty), groups are ordered by size, largest first, so every group is
// aligned to its size. Position p belongs to lane p % kSinkLanes, slot
// p / kSinkLanes. Arrays are plane-major so that the lanes of a wave read
// consecutive words: word w of lane l, slot s, sample b sits at
// ((b * slots + s) * words + w) * kSinkLanes + l, where slots (1..kSinkMaxSlots)
// is the smallest count that holds the batch's largest sample.
constexpr int kSinkLanes = 1024; // threads of a per-sample Sinkhorn workgroup
constexpr int kSinkMaxSlots = 6; // most positions per lane and order (the layout of a plan uses 1..6)
constexpr int kSinkPiece = 4;    // pairs per piece
constexpr int kSinkOwners = 2048; // rows or columns a workgroup covers
constexpr int kSinkMaxGroup = 64; // largest group (pieces of one owner)

struct PackedOrder {
    float *p0;      // [B][slots][kSinkPiece][lanes]: P0 (0 for padding)
    uint32_t *gi;   // [B][slots][kSinkPiece/2][lanes]: byte offsets of the gathered 8-byte values, two per word
    uint32_t *info; // [B][slots][lanes]: owner | log2(group) << 11 | head << 14 | valid << 15 | first position << 16 (rows)
    uint32_t *pos;  // [B][slots][kSinkPiece/2][lanes]: row-major positions within the sample (columns only)
    int32_t *n_pos; // [B]: positions used
    int slots;      // positions per lane of this layout
};

// Pieces of the per-sample Sinkhorn kernels for larger samples (up to
// kSinkOwnersW points per side): the same plane-major layout, with more slots
// (1..kSinkMaxSlotsW), streamed from memory in every sweep instead of held in
// registers. info: owner | log2(group) << 13 | head << 16 | valid << 17.
constexpr int kSinkOwnersW = 8192;
constexpr int kSinkMaxSlotsW = 32;
struct WideOrder {
    float *p0;      // [B][slots][kSinkPiece][lanes]
    uint32_t *gi;   // [B][slots][kSinkPiece/2][lanes]: byte offsets of the gathered 8-byte values, two per word
    uint32_t *info; // [B][slots][lanes]
    int32_t *n_pos; // [B]: positions used
    int slots;
};

// Device view of a plan, passed by value to the sparse kernels.
struct DevPlan {
    int B, N, M, L;
    int64_t nnz;
    const float *x, *y;
    int32_t *row_ptr, *col_ptr;   // [B*N+1], [B*M+1] global offsets
    int32_t *csr_col, *csr_row;   // [nnz] row-major: column j in sample, global row b*N+i
    int32_t *csc_row, *csc_col;   // [nnz] column-major: row i in sample, global column b*M+j
    int32_t *csc_perm;            // [nnz] row-major position of each column-major entry
    uint8_t *flags;               // bit 0: s_row >= tau, bit 1: s_col >= tau
    float *p_row, *p0r;           // row-major
    float *p_col, *p0c;           // column-major
    double *cost;                 // row-major C_t
    float2 *m12_row, *m12_col;
    double *T_row, *C1_row, *g_row, *T_col, *C1_col, *g_col;
    int32_t *pos_row;             // [2*B*N] row-major positions of the two minima
    int32_t *pos_col;             // [2*B*M] column-major positions
    uint8_t *clamp_row, *clamp_col;
    double *alpha, *beta;         // [(L+1)][B*N], [(L+1)][B*M] Sinkhorn scalings
    Counters *ctr;
    float *loss;                  // [B]
    // backward
    const float *grad_loss;
    float *grad_x, *grad_y;
    double *adj, *cbar;           // [nnz] row-major
    double *dvec;                 // [B*N] row losses of the per-iteration forward kernels
    double4 *xyr, *xyc;           // [B*N], [B*M] per-owner values of the per-iteration reverse sweeps: X, Y and
                                  // the reciprocal of the owner's scaling
    double *rz, *kz;              // [nnz] reverse-sweep adjoints in row and in column order (per-iteration
                                  // kernels; rz shares adj's memory and cbar kz's)
    PackedOrder pk_row, pk_col;   // per-sample Sinkhorn pieces (when that path is taken)
    WideOrder wk_row, wk_col;     // streamed per-sample pieces (larger samples)
    float *wr, *wc;               // backward of the streamed path: the plan adjoint in row and in column pieces
    uint32_t *split_sync;         // [B][2][kSplitSyncStride]: meeting counter (word 0) and the workgroups' XCDs
                                  // (words 1..K) of the split streamed kernels
                                  // (forward, backward), cleared before each launch
    float *yr, *yc;               // [L][B*N + kSinkOwnersW], [L][B*M + kSinkOwnersW]: owners' words published by
                                  // the split reverse kernels, one padded region per phase
    const int32_t *sink_place;    // during the forward softmax of that path: the pieces' placement, so that the
                                  // column softmax writes every pair into its pieces; else NULL
};

struct BuildArgs {
    int32_t *col_fill;          // [B*M], cleared by the finalize kernel
    int32_t *tmp_row, *tmp_src; // column-major staging [nnz]
};

void launch_csc_build(const DevPlan &d, const BuildArgs &a, hipStream_t s);
// With the column slots taken by the compaction, only the canonical order of
// each column remains.
void launch_csc_sort(const DevPlan &d, const BuildArgs &a, hipStream_t s);
// The column-major view of each sample in one workgroup (LDS counters), when
// the sample's column offsets and pairs fit in LDS: launched together with
// the row softmax, then the column softmax.
bool csc_sample_fits(int N, int M, int64_t max_pairs);
hipError_t launch_csc_and_softmax(const DevPlan &d, const Params &p, int64_t max_pairs, hipStream_t s);

// hipFuncSetAttribute(k, MaxDynamicSharedMemorySize, bytes) on the current
// device, made once per device and kernel for every larger size (the forward
// and backward would otherwise make the runtime call on every call).
hipError_t set_dynamic_lds(const void *k, size_t bytes);

void launch_softmax(const DevPlan &d, const Params &p, hipStream_t s);
// Backward of both softmaxes and the distance gradient. double_p: P formed
// again in double precision from the stored costs (for plans whose reverse
// sweeps keep the adjoint in double, or that have none), else read as stored.
void launch_bwd_softmax(const DevPlan &d, const Params &p, bool double_p, hipStream_t s);

// Sinkhorn. The per-sample kernels run all iterations in one workgroup per
// sample with the sample's pairs in registers; the per-iteration kernels are
// the general fallback.
//
// Pieces of a row or column with len pairs, and log2 of its group size.
__device__ __forceinline__ int sink_pieces(int len) { return len < kSinkPiece ? 1 : (len + kSinkPiece - 1) / kSinkPiece; }
__device__ __forceinline__ int sink_log2_group(int np) { return np <= 1 ? 0 : 32 - __clz(np - 1); }

// What the host reads back after the support scan, in one copy: the
// counters, then per sample the stored pairs counted over rows and over
// columns (int64 [2][B]), the pair offsets of the samples (int32 [B + 1],
// row_ptr[b*N]) and the piece counts (int32 [B][4]: positions needed by the
// rows, by the columns, most pieces of a row, of a column).
struct Readback {
    Counters ctr;
};
inline size_t readback_bytes(int B) { return sizeof(Readback) + 16 * (size_t)B + 4 * (5 * (size_t)B + 1); }
__host__ __device__ inline int64_t *readback_totals(Readback *r) { return reinterpret_cast<int64_t *>(r + 1); }
__host__ __device__ inline int32_t *readback_offsets(Readback *r, int B) { return reinterpret_cast<int32_t *>(readback_totals(r) + 2 * B); }
__host__ __device__ inline int32_t *readback_pieces(Readback *r, int B) { return readback_offsets(r, B) + B + 1; }

// Row and column offsets of all samples (row_ptr [B*N+1] from the per-(row,
// chunk) counts cnt [B*N][S], col_ptr [B*M+1] from col_cnt) and the read-back
// block, in two launches. tiles is device scratch of offsets_scratch_ints
// ints (per-tile totals); rb_host, mapped pinned host memory, receives the
// whole block, written by the kernels.
size_t offsets_scratch_ints(int B, int N, int M);
void launch_offsets(const int32_t *cnt, int S, const int32_t *col_cnt, const Counters *ctr, int B, int N, int M,
                    int32_t *row_ptr, int32_t *col_ptr, int32_t *tiles, Readback *rb_host, hipStream_t s);
// Whether the per-sample kernels take a batch: counts are the host copy of the
// piece counts of the read-back block, max_pairs the largest sample's stored
// pairs.
// Positions per lane the per-sample kernels need for a batch (1..kSinkMaxSlots),
// 0 when it does not fit them.
int sinkhorn_slots(int N, int M, const int32_t *counts, int B);
// Slots of the streamed per-sample path for a batch (1..kSinkMaxSlotsW), 0
// when it does not take it.
int sinkhorn_slots_wide(int N, int M, const int32_t *counts, int B);
// Places the streamed pieces (place: [B][2][kSinkOwnersW] int32 scratch)
// and writes every pair into them (after the softmax).
void launch_wide_pack(const DevPlan &d, int32_t *place, hipStream_t s);
// Workgroups per sample of the split streamed kernels for a batch of B on the
// current device (2..kSplitMax; every workgroup of the grid must be resident
// at once), or 1 when the one-workgroup kernels are taken (also when the
// environment sets APML_SINKHORN_SPLIT=0; =streamed keeps the split kernels'
// streamed variants at every share).
constexpr int kSplitMax = 8;
constexpr int kSplitSyncStride = 32; // counters 128 bytes apart
int sinkhorn_split_factor(int B);
// Workgroups of a split launch: B rounded up to a multiple of the 8 XCDs, times K.
inline int split_grid(int B, int K) { return (B + 7) / 8 * 8 * K; }
// Streamed kernels, split over sinkhorn_split_factor(B) workgroups per sample
// when that is above 1 (the reverse kernel then needs d.yr, d.yc), else one.
hipError_t launch_sinkhorn_fwd_wide(const DevPlan &d, double eps, hipStream_t s);
hipError_t launch_sinkhorn_bwd_wide(const DevPlan &d, hipStream_t s);
bool sinkhorn_bwd_fits(int slots, int64_t max_pairs);
size_t packed_order_words(int B, int slots); // 32-bit words of one PackedOrder's p0 array
// Lays out the pieces of both orders; place: [B][2][2048] int32 scratch.
// placed: place[] and the info words are already written (with the compaction).
void launch_pack(const DevPlan &d, int32_t *place, bool placed, hipStream_t s);
// Only the placement (place[] and the info words), when the column softmax
// packs the pairs.
void launch_place(const DevPlan &d, int32_t *place, hipStream_t s);
hipError_t launch_sinkhorn_fwd(const DevPlan &d, double eps, hipStream_t s);
hipError_t launch_sinkhorn_bwd(const DevPlan &d, int64_t max_pairs, hipStream_t s);
void launch_sinkhorn_fwd_steps(const DevPlan &d, double eps, hipStream_t s);
void launch_sinkhorn_bwd_steps(const DevPlan &d, hipStream_t s);

// Kept pairs per sample, in count_support_chunks(largest sample) partial
// counts per sample: out [B][chunks].
int count_support_chunks(int64_t max_pairs);
void launch_count_support(const int32_t *row_ptr, const uint8_t *flags, int B, int N, int chunks,
                          unsigned long long *out, hipStream_t s);

// ---------------------------------------------------------------------------
// dense APML (the unpruned formulation of Sec. III-A, any dimension d)
// ---------------------------------------------------------------------------

constexpr int kDenseMaxD = 16; // largest point dimension of the dense path

// Per-owner vectors of one direction (rows: [B*N], columns: [B*M]).
struct DenseSide {
    int32_t *k1, *k2;          // indices of the minimum and the second minimum
    double *c1, *g, *T, *Z;    // minimum cost, clamped gap, temperature (Eq. 1), softmax normaliser (Eq. 2)
    uint8_t *clamped;          // gap clamped: no temperature gradient
    double *sigma, *gbar, *e;  // backward: softmax adjoint sum, gap adjoint, scratch
};

struct DenseDev {
    int B, N, M, d, L;
    double delta, eps_gap, eps_stab, eps_dist;
    int tgrad_full;              // temperature differentiated (apml_tgrad_mode FULL)
    const float *x, *y;          // [B, N, d], [B, M, d]
    DenseSide row, col;
    float *P0, *P;               // [B][N][M]: initial plan, plan after the Sinkhorn iterations
    double *S, *R;               // [L][B*M], [L][B*N]: column and row sums of every iteration
    double *a_cum, *c_cum;       // [L+1][B*N], [L+1][B*M]: cumulative row and column scalings
    double *part;                // [chunks][B*M] (x d for the gradient): partial sums of the column passes
    int chunks, chunk;           // row chunks of the column passes and their length
    float *loss;                 // [B]
    double *A;                   // [B][N][M]: plan adjoint (backward)
    const float *grad_loss;
    float *grad_x, *grad_y;
};

void dense_chunks(int B, int N, int M, int *chunks, int *chunk);
void launch_dense_forward(const DenseDev &D, double lk_row, double lk_col, hipStream_t s);
void launch_dense_backward(const DenseDev &D, hipStream_t s);

} // namespace apml
