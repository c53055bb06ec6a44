// Internal declarations shared by the kernels and the host orchestration of
// libapml. Not part of the public ABI (include/apml.h is).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace apml {

constexpr int kBlock = 256;   // threads per workgroup (4 wave64)
constexpr int kUnroll = 8;    // broadcast points per inner step of the dense scans

// Device-side counters of one forward call.
struct Counters {
    unsigned long long stored; // pairs emitted by the support scan
    unsigned int overflow;     // emitted pairs that did not fit their slot group
    unsigned int error;        // bit 0: a row's minima not found among its pairs; bit 1: a column's
};

// A pair that did not fit its (row, chunk) slot group.
struct OverflowEntry {
    int32_t row;   // global row b*N + i
    int32_t chunk; // column chunk that emitted it
    int32_t rank;  // position among the pairs of this (row, chunk)
    int32_t col;   // column j within the sample
};

// One direction of the dense minimum / second-minimum scan. Owners are the
// points whose statistics are computed (X for rows, Y for columns); the
// broadcast set is scanned against every owner.
struct ScanDir {
    const float *own;    // [B, n_own, 3]
    const float *bcast;  // [B, n_bc, 3]
    float2 *partial;     // [S][B * n_own]: (min, second min) of squared distance per chunk
    int n_own, n_bc;
    int S, chunk;        // chunks of the broadcast range and their length
    int owner_blocks;    // workgroups per sample over the owners
    int tiles;           // B * S * owner_blocks
};

struct FinalizeDir {
    const float2 *partial; // [S][B * n_own]
    const float *own;      // owner coordinates [B, n_own, 3]
    float2 *m12;           // out: (m1, m2) per owner
    float *E;              // out (rows): emission threshold on the squared distance
    float4 *packed;        // out (columns): (x, y, z, emission threshold)
    int n_own, S;
    double log_ratio;      // log((K-1) p_min / (1 - p_min)), K = length of the other set
};

struct Params {
    double p_min, tau, eps_stab, delta, eps_gap, eps_dist;
    double log_inv_tau; // log(1/tau); +inf when tau == 0
    double lk_row, lk_col; // log((K-1) p / (1-p)) for rows (K = M) and columns (K = N)
    int n_iter;
};

// Host launch wrappers (kernels.hip).
void launch_top2(const ScanDir &rows, const ScanDir &cols, int B, hipStream_t s);
void launch_finalize(const FinalizeDir &rows, const FinalizeDir &cols, int B, const Params &p,
                     hipStream_t s);
struct EmitArgs {
    const float *x;      // [B, N, 3]
    const float4 *ypack; // [B, M]: y and its column threshold
    const float *E_row;  // [B*N]
    int B, N, M, S, chunk, K, owner_blocks;
    int32_t *slots;      // [B*N][S][K]
    int32_t *cnt;        // [B*N][S]
    int32_t *col_cnt;    // [B*M]
    OverflowEntry *ovf;
    unsigned ovf_cap;
    Counters *ctr;
};
void launch_emit(const EmitArgs &a, hipStream_t s);

// Exclusive prefix sums of two count arrays at once. Element k of array a
// is the sum of in[k*S .. k*S+S-1]; out has n+1 entries (out[n] = total).
struct ScanArray {
    const int32_t *in;
    int n, S;
    int32_t *out;
    int32_t *tile_sums;
    int tiles;
};
int scan_tile_items();
void launch_scan(const ScanArray &a0, const ScanArray &a1, hipStream_t s);

struct BuildArgs {
    int B, N, M, S, K;
    const int32_t *slots, *cnt, *row_ptr, *col_ptr;
    const OverflowEntry *ovf;
    int n_ovf;
    int32_t *csr_col;
    int32_t *col_fill;                  // [B*M], zeroed
    int32_t *tmp_row, *tmp_src, *tmp_gc; // column-major staging [nnz]
    int32_t *csc_row, *csc_perm;
    int64_t nnz;
};
void launch_build(const BuildArgs &a, hipStream_t s);

struct SoftmaxArgs {
    const float *x, *y;
    int B, N, M;
    const int32_t *row_ptr, *col_ptr, *csr_col, *csc_row, *csc_perm;
    const float2 *m12_row, *m12_col;
    uint8_t *flags;
    float *p_row, *p_col, *p0r, *p0c;
    double *T_row, *C1_row, *g_row, *T_col, *C1_col, *g_col;
    int32_t *pos_row, *pos_col; // [2 * B*N], [2 * B*M]: positions of the two minima
    uint8_t *clamp_row, *clamp_col;
    Counters *ctr;
};
void launch_softmax(const SoftmaxArgs &a, const Params &p, hipStream_t s);

struct SinkhornArgs {
    int B, N, M, L;
    const int32_t *row_ptr, *col_ptr, *csr_col, *csc_row;
    const float *p0r, *p0c;
    double *alpha; // [(L+1) * B*N]
    double *beta;  // [(L+1) * B*M]
    double *rden;  // [L * B*N]: R + eps per iteration
    double *sden;  // [L * B*M]: S + eps per iteration
};
void launch_sinkhorn_init(const SinkhornArgs &a, hipStream_t s);
void launch_sinkhorn_step(const SinkhornArgs &a, int l, double eps, hipStream_t s);

struct LossArgs {
    const float *x, *y;
    int B, N, M;
    const int32_t *row_ptr, *csr_col;
    const float *p0r;
    const double *alpha_L, *beta_L;
    double *loss_rows; // [B*N] scratch
    float *loss;       // [B]
};
void launch_loss(const LossArgs &a, hipStream_t s);

struct BackwardArgs {
    const float *x, *y, *grad_loss;
    float *grad_x, *grad_y;
    int B, N, M, L;
    const int32_t *row_ptr, *col_ptr, *csr_col, *csc_row, *csc_perm;
    const uint8_t *flags;
    const float *p_row, *p_col, *p0r, *p0c;
    const double *alpha, *beta, *rden, *sden;
    const double *T_row, *C1_row, *g_row, *T_col, *C1_col, *g_col;
    const int32_t *pos_row, *pos_col;
    const uint8_t *clamp_row, *clamp_col;
    double *adj;  // [nnz] adjoint of the plan, row-major order
    double *cbar; // [nnz] adjoint of the cost, row-major order
};
void launch_bwd_sinkhorn_step(const BackwardArgs &a, int l, hipStream_t s);
void launch_bwd_softmax(const BackwardArgs &a, const Params &p, hipStream_t s);

void launch_count_support(const int32_t *row_ptr, const uint8_t *flags, int B, int N,
                          unsigned long long *out, hipStream_t s);

} // namespace apml
