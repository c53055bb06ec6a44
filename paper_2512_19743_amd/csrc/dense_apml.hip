// Dense APML (Sec. III-A): the formulation that sparse APML prunes, kept as a
// baseline. Every pair (i, j) of a sample takes part: no threshold, so the
// plan is the full N x M matrix, for points of any dimension d.
//
//   C_ij = ||x_i - y_j||_2; per row the two smallest costs (decided on the
//   single-precision squared distance, ties to the smaller index), the
//   clamped gap g and the temperature T (Eq. 1); P_row = softmax over the
//   whole row (Eq. 2); the same per column; P0 = (P_row + P_col) / 2;
//   L times column scaling (Eq. 3) then row scaling (Eq. 4); loss = sum P C;
//   the gradient through all of it, temperatures included (Eq. 5 for the
//   distance).
//
// Materialised per sample: P0 and the plan P (float32, N x M), and in the
// backward pass the plan adjoint (float64, N x M). Everything else is a
// per-row or per-column vector; C and the softmaxes are recomputed from the
// coordinates where they are needed. Row passes take one wave per row
// (coalesced along the row); column passes take one thread per column and
// chunk of rows (coalesced across the columns of a wave), and a second launch
// adds the chunks' partial sums in a fixed order, so every result is bitwise
// reproducible.
#include "apml_internal.h"
#include "device_common.h"

namespace apml {
namespace {

constexpr int kWavesPerBlock = 4;

// Squared distance of two d-dimensional float points in single precision:
// s = d0*d0, then s = fma(dk, dk, s) for k = 1.. (for d = 3 the sequence of
// the sparse path's scans).
__device__ __forceinline__ float dsq_f32(const float *a, const float *b, int d)
{
    float t = a[0] - b[0];
    float s = t * t;
    for (int k = 1; k < d; ++k) {
        t = a[k] - b[k];
        s = __builtin_fmaf(t, t, s);
    }
    return s;
}

// C = ||a - b||_2 in double precision (Sec. III-A).
__device__ __forceinline__ double dcost(const float *a, const float *b, int d)
{
    double t = (double)a[0] - (double)b[0];
    double s = t * t;
    for (int k = 1; k < d; ++k) {
        t = (double)a[k] - (double)b[k];
        s += t * t;
    }
    return sqrt(s);
}

// (value, index) is smaller than (v2, i2) in lexicographic order.
__device__ __forceinline__ bool before(float v, int i, float v2, int i2) { return v < v2 || (v == v2 && i < i2); }

// Merges another lane's two smallest (value, index) pairs into this lane's:
// the two smallest of the union multiset, ties to the smaller index.
__device__ __forceinline__ void merge_top2(float &m1, int &k1, float &m2, int &k2, float n1, int q1, float n2,
                                           int q2)
{
    if (before(n1, q1, m1, k1)) {
        // the other list's first is the new first; the second is the smaller
        // of this list's first and the other's second
        if (before(m1, k1, n2, q2)) {
            m2 = m1;
            k2 = k1;
        } else {
            m2 = n2;
            k2 = q2;
        }
        m1 = n1;
        k1 = q1;
    } else if (before(n1, q1, m2, k2)) {
        m2 = n1;
        k2 = q1;
    }
}

// Per owner (a row, ROWS, or a column): the two nearest points of the other
// cloud, the clamped gap and the temperature (Eq. 1), and the softmax
// normaliser Z = sum over all K of exp(-T (C - C1)) (Eq. 2). One wave per
// owner.
template <bool ROWS> __global__ __launch_bounds__(64 * kWavesPerBlock) void k_dstats(DenseDev D, double log_ratio)
{
    const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int n_own = ROWS ? D.N : D.M, n_oth = ROWS ? D.M : D.N;
    if (w >= (int64_t)D.B * n_own)
        return;
    const int b = (int)(w / n_own), lane = lane_id(), d = D.d;
    const float *own = (ROWS ? D.x : D.y) + w * d;
    const float *oth = (ROWS ? D.y : D.x) + (int64_t)b * n_oth * d;
    float m1 = kInf, m2 = kInf;
    int k1 = INT_MAX, k2 = INT_MAX;
    for (int k = lane; k < n_oth; k += 64) {
        const float s = dsq_f32(own, oth + (int64_t)k * d, d);
        if (s < m1) {
            m2 = m1;
            k2 = k1;
            m1 = s;
            k1 = k;
        } else if (s < m2) {
            m2 = s;
            k2 = k;
        }
    }
    for (int o = 1; o < 64; o <<= 1) {
        const float n1 = __shfl_xor(m1, o), n2 = __shfl_xor(m2, o);
        const int q1 = __shfl_xor(k1, o), q2 = __shfl_xor(k2, o);
        merge_top2(m1, k1, m2, k2, n1, q1, n2, q2);
    }
    // only distances that overflow single precision leave an index unset
    if (k1 == INT_MAX)
        k1 = 0;
    if (k2 == INT_MAX || k2 == k1)
        k2 = k1 == 0 ? 1 : 0;
    const double c1 = dcost(own, oth + (int64_t)k1 * d, d);
    const double c2 = dcost(own, oth + (int64_t)k2 * d, d);
    const double gap = (c2 - c1) + D.delta;
    const bool clamped = gap < D.eps_gap;
    const double g = clamped ? D.eps_gap : gap;
    const double T = log_ratio / g;
    double z = 0.0;
    for (int k = lane; k < n_oth; k += 64)
        z += exp(-T * (dcost(own, oth + (int64_t)k * d, d) - c1));
    z = wave_sum(z);
    if (lane == 0) {
        DenseSide &s = ROWS ? D.row : D.col;
        s.k1[w] = k1;
        s.k2[w] = k2;
        s.c1[w] = c1;
        s.g[w] = g;
        s.T[w] = T;
        s.Z[w] = z;
        s.clamped[w] = clamped;
    }
}

// The softmaxes of pair (i, j) of sample b (Eq. 2), from the statistics.
__device__ __forceinline__ double p_row(const DenseDev &D, int64_t r, double C)
{
    return exp(-D.row.T[r] * (C - D.row.c1[r])) / D.row.Z[r];
}
__device__ __forceinline__ double p_col(const DenseDev &D, int64_t c, double C)
{
    return exp(-D.col.T[c] * (C - D.col.c1[c])) / D.col.Z[c];
}

// P0 = (P_row + P_col) / 2 on every pair (the initial plan of Sec. III-A),
// into P0 and P. One thread per pair.
__global__ __launch_bounds__(kBlock) void k_dp0(DenseDev D)
{
    const int64_t NM = (int64_t)D.N * D.M, total = (int64_t)D.B * NM;
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < total; e += (int64_t)gridDim.x * kBlock) {
        const int64_t b = e / NM, ij = e - b * NM;
        const int64_t i = ij / D.M, j = ij - i * D.M;
        const int64_t r = b * D.N + i, c = b * D.M + j;
        const double C = dcost(D.x + r * D.d, D.y + c * D.d, D.d);
        const float p0 = (float)(0.5 * (p_row(D, r, C) + p_col(D, c, C)));
        D.P0[e] = p0;
        D.P[e] = p0;
    }
}

// Row step l of the forward Sinkhorn, with column step l applied on the fly:
// u = P / (S^l_j + eps) is the plan after Eq. 3, R_i = sum_j u (saved), and
// P = u / (R_i + eps) after Eq. 4. One wave per row.
__global__ __launch_bounds__(64 * kWavesPerBlock) void k_drow_step(DenseDev D, int l)
{
    const int64_t r = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (r >= (int64_t)D.B * D.N)
        return;
    const int64_t b = r / D.N;
    const double *S = D.S + (int64_t)(l - 1) * D.B * D.M + b * D.M;
    float *P = D.P + r * D.M;
    const double eps = D.eps_stab;
    double acc = 0.0;
    for (int j = lane_id(); j < D.M; j += 64)
        acc += (double)P[j] / (S[j] + eps);
    const double R = wave_sum(acc);
    if (lane_id() == 0)
        D.R[(int64_t)(l - 1) * D.B * D.N + r] = R;
    for (int j = lane_id(); j < D.M; j += 64)
        P[j] = (float)((double)P[j] / (S[j] + eps) / (R + eps));
}

// What a column pass adds up over the rows of one column.
enum ColOp {
    COL_SUM_P,    // S_j = sum_i P_ij (Eq. 3)
    COL_ADJ_DOT,  // e_j = sum_i Abar_ij u_ij, u the plan after column step l
    COL_SIGMA,    // sigma'_j = sum_i P_col_ij Pbar_col_ij, Pbar_col = Abar / 2
    COL_TBAR,     // Tbar'_j = -sum_i abar'_ij (C_ij - C1'_j), abar' = P_col (Pbar_col - sigma'_j)
    COL_GRAD_Y    // sum_i Cbar_ij (x_i - y_j) / (C_ij + eps_dist), per coordinate
};

// Cost adjoint of pair (i, j): the direct term grad_loss * v (v the final
// plan), both softmax adjoints through the costs (-T abar), and the gap terms
// of the temperature adjoint at the row's and the column's two minima.
__device__ __forceinline__ double cost_adjoint(const DenseDev &D, int64_t b, int64_t i, int64_t j, int64_t e,
                                               double C)
{
    const int64_t r = b * D.N + i, c = b * D.M + j;
    const int64_t BN = (int64_t)D.B * D.N, BM = (int64_t)D.B * D.M;
    const double v = (double)D.P0[e] * D.a_cum[(int64_t)D.L * BN + r] * D.c_cum[(int64_t)D.L * BM + c];
    const double half = 0.5 * D.A[e];
    const double ar = p_row(D, r, C) * (half - D.row.sigma[r]);
    const double ac = p_col(D, c, C) * (half - D.col.sigma[c]);
    double cb = D.grad_loss[b] * v - D.row.T[r] * ar - D.col.T[c] * ac;
    if (j == D.row.k2[r]) cb += D.row.gbar[r];
    if (j == D.row.k1[r]) cb -= D.row.gbar[r];
    if (i == D.col.k2[c]) cb += D.col.gbar[c];
    if (i == D.col.k1[c]) cb -= D.col.gbar[c];
    return cb;
}

// Partial sums of a column pass: thread (chunk, column) adds its chunk's rows
// into part[chunk][column] (part[chunk][column][k] for the gradient).
template <int OP> __global__ __launch_bounds__(kBlock) void k_dcol_part(DenseDev D, int l)
{
    const int64_t BM = (int64_t)D.B * D.M;
    const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (t >= BM * D.chunks)
        return;
    const int64_t ch = t / BM, c = t - ch * BM, b = c / D.M, j = c - b * D.M;
    const int i0 = (int)(ch * D.chunk), i1 = min(D.N, i0 + D.chunk);
    const int d = D.d;
    const float *yj = D.y + c * d;
    const int64_t BN = (int64_t)D.B * D.N;
    double acc[OP == COL_GRAD_Y ? kDenseMaxD : 1] = {};
    for (int i = i0; i < i1; ++i) {
        const int64_t e = (b * D.N + i) * D.M + j, r = b * D.N + i;
        if constexpr (OP == COL_SUM_P) {
            acc[0] += (double)D.P[e];
        } else if constexpr (OP == COL_ADJ_DOT) {
            const double u = (double)D.P0[e] * D.a_cum[(int64_t)(l - 1) * BN + r] * D.c_cum[(int64_t)l * BM + c];
            acc[0] += D.A[e] * u;
        } else {
            const float *xi = D.x + r * d;
            const double C = dcost(xi, yj, d);
            if constexpr (OP == COL_SIGMA) {
                acc[0] += p_col(D, c, C) * (0.5 * D.A[e]);
            } else if constexpr (OP == COL_TBAR) {
                acc[0] -= p_col(D, c, C) * (0.5 * D.A[e] - D.col.sigma[c]) * (C - D.col.c1[c]);
            } else {
                const double w = cost_adjoint(D, b, i, j, e, C) / (C + D.eps_dist);
                for (int k = 0; k < d; ++k)
                    acc[k] += w * ((double)xi[k] - (double)yj[k]);
            }
        }
    }
    if constexpr (OP == COL_GRAD_Y) {
        for (int k = 0; k < d; ++k)
            D.part[(ch * BM + c) * d + k] = acc[k];
    } else {
        D.part[ch * BM + c] = acc[0];
    }
}

// Adds the chunks' partial sums of each column in chunk order.
template <int OP> __global__ __launch_bounds__(kBlock) void k_dcol_final(DenseDev D, int l)
{
    const int64_t BM = (int64_t)D.B * D.M;
    const int64_t c = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (c >= BM)
        return;
    if constexpr (OP == COL_GRAD_Y) {
        for (int k = 0; k < D.d; ++k) {
            double s = 0.0;
            for (int ch = 0; ch < D.chunks; ++ch)
                s += D.part[(ch * BM + c) * D.d + k];
            D.grad_y[c * D.d + k] = (float)(-s);
        }
        return;
    }
    double s = 0.0;
    for (int ch = 0; ch < D.chunks; ++ch)
        s += D.part[ch * BM + c];
    if constexpr (OP == COL_SUM_P) {
        D.S[(int64_t)(l - 1) * BM + c] = s;
    } else if constexpr (OP == COL_ADJ_DOT) {
        D.col.e[c] = s;
    } else if constexpr (OP == COL_SIGMA) {
        D.col.sigma[c] = s;
    } else if constexpr (OP == COL_TBAR) {
        // temperature adjoint (unclamped columns): gap adjoint -Tbar T / g
        D.col.gbar[c] = (D.tgrad_full && !D.col.clamped[c]) ? -s * D.col.T[c] / D.col.g[c] : 0.0;
    }
}

// Cumulative scalings: a^l_i = prod_{k<=l} 1/(R^k_i + eps) and
// c^l_j = prod_{k<=l} 1/(S^k_j + eps), so that the plan after row step l is
// P0 a^l c^l and after column step l is P0 a^(l-1) c^l.
__global__ __launch_bounds__(kBlock) void k_dcum(DenseDev D)
{
    const int64_t BN = (int64_t)D.B * D.N, BM = (int64_t)D.B * D.M;
    const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (t < BN) {
        double a = 1.0;
        D.a_cum[t] = a;
        for (int l = 1; l <= D.L; ++l) {
            a /= (D.R[(int64_t)(l - 1) * BN + t] + D.eps_stab);
            D.a_cum[(int64_t)l * BN + t] = a;
        }
    } else if (t < BN + BM) {
        const int64_t c = t - BN;
        double s = 1.0;
        D.c_cum[c] = s;
        for (int l = 1; l <= D.L; ++l) {
            s /= (D.S[(int64_t)(l - 1) * BM + c] + D.eps_stab);
            D.c_cum[(int64_t)l * BM + c] = s;
        }
    }
}

// loss_b = sum_ij P_ij C_ij (Sec. III-D): row sums, then per sample in order.
__global__ __launch_bounds__(64 * kWavesPerBlock) void k_dloss_rows(DenseDev D)
{
    const int64_t r = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (r >= (int64_t)D.B * D.N)
        return;
    const int64_t b = r / D.N;
    const float *xi = D.x + r * D.d, *yb = D.y + b * D.M * D.d;
    const float *P = D.P + r * D.M;
    double acc = 0.0;
    for (int j = lane_id(); j < D.M; j += 64)
        acc += (double)P[j] * dcost(xi, yb + (int64_t)j * D.d, D.d);
    acc = wave_sum(acc);
    if (lane_id() == 0)
        D.row.e[r] = acc;
}

__global__ __launch_bounds__(kBlock) void k_dloss_sum(DenseDev D)
{
    __shared__ double part[kBlock / 64];
    const int b = blockIdx.x;
    double acc = 0.0;
    for (int i = threadIdx.x; i < D.N; i += kBlock)
        acc += D.row.e[(int64_t)b * D.N + i];
    acc = wave_sum(acc);
    if (lane_id() == 0)
        part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        double s = 0.0;
        for (int w = 0; w < kBlock / 64; ++w)
            s += part[w];
        D.loss[b] = (float)s;
    }
}

// Reverse row step l (Eq. 4 backwards): u = P0 a^l c^l, d_i = sum_j Abar u,
// Abar = (Abar - d_i) / (R^l_i + eps). The first reverse step starts from the
// loss adjoint grad_loss * C; with pending, the column step l+1's update
// (Abar - e_j) / (S^(l+1)_j + eps) is applied first. One wave per row.
__global__ __launch_bounds__(64 * kWavesPerBlock) void k_drow_adj(DenseDev D, int l, int first, int pending)
{
    const int64_t r = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (r >= (int64_t)D.B * D.N)
        return;
    const int64_t b = r / D.N, BN = (int64_t)D.B * D.N, BM = (int64_t)D.B * D.M;
    const float *xi = D.x + r * D.d, *yb = D.y + b * D.M * D.d;
    double *A = D.A + r * D.M;
    const float *P0 = D.P0 + r * D.M;
    const double al = D.a_cum[(int64_t)l * BN + r];
    const double *cl = D.c_cum + (int64_t)l * BM + b * D.M;
    const double *Sp = D.S + (int64_t)l * BM + b * D.M; // S^(l+1) when pending
    const double *ep = D.col.e + b * D.M;
    const double g = D.grad_loss[b], eps = D.eps_stab;
    auto adj = [&](int j) {
        double a;
        if (first)
            a = g * dcost(xi, yb + (int64_t)j * D.d, D.d);
        else
            a = A[j];
        if (pending)
            a = (a - ep[j]) / (Sp[j] + eps);
        return a;
    };
    double acc = 0.0;
    for (int j = lane_id(); j < D.M; j += 64)
        acc += adj(j) * ((double)P0[j] * al * cl[j]);
    const double dsum = wave_sum(acc);
    const double R = D.R[(int64_t)(l - 1) * BN + r];
    for (int j = lane_id(); j < D.M; j += 64)
        A[j] = (adj(j) - dsum) / (R + eps);
}

// Abar = (Abar - e_j) / (S^l_j + eps) on every pair (the last reverse column
// step), or Abar = grad_loss * C when there are no Sinkhorn iterations.
__global__ __launch_bounds__(kBlock) void k_dadj_final(DenseDev D, int l)
{
    const int64_t NM = (int64_t)D.N * D.M, total = (int64_t)D.B * NM, BM = (int64_t)D.B * D.M;
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < total; e += (int64_t)gridDim.x * kBlock) {
        const int64_t b = e / NM, ij = e - b * NM, i = ij / D.M, j = ij - i * D.M;
        const int64_t c = b * D.M + j;
        if (l == 0)
            D.A[e] = D.grad_loss[b] * dcost(D.x + (b * D.N + i) * D.d, D.y + c * D.d, D.d);
        else
            D.A[e] = (D.A[e] - D.col.e[c]) / (D.S[(int64_t)(l - 1) * BM + c] + D.eps_stab);
    }
}

// Row softmax adjoint (Sec. III-D): Pbar_row = Abar / 2, sigma_i = sum P_row
// Pbar_row, abar = P_row (Pbar_row - sigma_i), Tbar_i = -sum abar (C - C1_i),
// and the gap adjoint -Tbar T / g of an unclamped row. One wave per row.
__global__ __launch_bounds__(64 * kWavesPerBlock) void k_drow_softmax_adj(DenseDev D)
{
    const int64_t r = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (r >= (int64_t)D.B * D.N)
        return;
    const int64_t b = r / D.N;
    const float *xi = D.x + r * D.d, *yb = D.y + b * D.M * D.d;
    const double *A = D.A + r * D.M;
    double acc = 0.0;
    for (int j = lane_id(); j < D.M; j += 64)
        acc += p_row(D, r, dcost(xi, yb + (int64_t)j * D.d, D.d)) * (0.5 * A[j]);
    const double sigma = wave_sum(acc);
    acc = 0.0;
    for (int j = lane_id(); j < D.M; j += 64) {
        const double C = dcost(xi, yb + (int64_t)j * D.d, D.d);
        acc -= p_row(D, r, C) * (0.5 * A[j] - sigma) * (C - D.row.c1[r]);
    }
    const double tbar = wave_sum(acc);
    if (lane_id() == 0) {
        D.row.sigma[r] = sigma;
        D.row.gbar[r] = (D.tgrad_full && !D.row.clamped[r]) ? -tbar * D.row.T[r] / D.row.g[r] : 0.0;
    }
}

// grad_x_i = sum_j Cbar_ij (x_i - y_j) / (C_ij + eps_dist) (Eq. 5). One wave per row.
__global__ __launch_bounds__(64 * kWavesPerBlock) void k_dgrad_x(DenseDev D)
{
    const int64_t r = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (r >= (int64_t)D.B * D.N)
        return;
    const int64_t b = r / D.N, i = r - b * D.N;
    const int d = D.d;
    const float *xi = D.x + r * d, *yb = D.y + b * D.M * d;
    double acc[kDenseMaxD] = {};
    for (int j = lane_id(); j < D.M; j += 64) {
        const float *yj = yb + (int64_t)j * d;
        const double C = dcost(xi, yj, d);
        const double w = cost_adjoint(D, b, i, j, r * D.M + j, C) / (C + D.eps_dist);
        for (int k = 0; k < d; ++k)
            acc[k] += w * ((double)xi[k] - (double)yj[k]);
    }
    for (int k = 0; k < d; ++k) {
        const double s = wave_sum(acc[k]);
        if (lane_id() == 0)
            D.grad_x[r * d + k] = (float)s;
    }
}

unsigned wave_blocks(int64_t owners) { return (unsigned)((owners + kWavesPerBlock - 1) / kWavesPerBlock); }

unsigned stride_blocks(int64_t n) { return (unsigned)std::min<int64_t>((n + kBlock - 1) / kBlock, 65536); }

template <int OP> void col_pass(const DenseDev &D, int l, hipStream_t s)
{
    const int64_t BM = (int64_t)D.B * D.M;
    k_dcol_part<OP><<<blocks_for(BM * D.chunks, kBlock), kBlock, 0, s>>>(D, l);
    k_dcol_final<OP><<<blocks_for(BM, kBlock), kBlock, 0, s>>>(D, l);
}

} // namespace

void dense_chunks(int B, int N, int M, int *chunks, int *chunk)
{
    // about 2^18 threads per column pass, chunks of at least 64 rows
    const int64_t cols = (int64_t)B * M;
    int64_t c = std::max<int64_t>(1, ((int64_t)1 << 18) / std::max<int64_t>(cols, 1));
    c = std::min<int64_t>(c, std::max(1, N / 64));
    *chunk = (int)((N + c - 1) / c);
    *chunks = (N + *chunk - 1) / *chunk;
}

void launch_dense_forward(const DenseDev &D, double lk_row, double lk_col, hipStream_t s)
{
    const int64_t BN = (int64_t)D.B * D.N, BM = (int64_t)D.B * D.M;
    k_dstats<true><<<wave_blocks(BN), 64 * kWavesPerBlock, 0, s>>>(D, lk_row);
    k_dstats<false><<<wave_blocks(BM), 64 * kWavesPerBlock, 0, s>>>(D, lk_col);
    k_dp0<<<stride_blocks(BN * D.M), kBlock, 0, s>>>(D);
    for (int l = 1; l <= D.L; ++l) {
        col_pass<COL_SUM_P>(D, l, s);
        k_drow_step<<<wave_blocks(BN), 64 * kWavesPerBlock, 0, s>>>(D, l);
    }
    k_dcum<<<blocks_for(BN + BM, kBlock), kBlock, 0, s>>>(D);
    k_dloss_rows<<<wave_blocks(BN), 64 * kWavesPerBlock, 0, s>>>(D);
    k_dloss_sum<<<D.B, kBlock, 0, s>>>(D);
}

void launch_dense_backward(const DenseDev &D, hipStream_t s)
{
    const int64_t BN = (int64_t)D.B * D.N;
    // reverse Sinkhorn: row step l, then column step l, for l = L .. 1; each
    // column step's update is applied by the next row step (or at the end)
    for (int l = D.L; l >= 1; --l) {
        k_drow_adj<<<wave_blocks(BN), 64 * kWavesPerBlock, 0, s>>>(D, l, l == D.L, l < D.L);
        col_pass<COL_ADJ_DOT>(D, l, s);
    }
    k_dadj_final<<<stride_blocks(BN * D.M), kBlock, 0, s>>>(D, D.L > 0 ? 1 : 0);
    // softmax and temperature adjoints
    k_drow_softmax_adj<<<wave_blocks(BN), 64 * kWavesPerBlock, 0, s>>>(D);
    col_pass<COL_SIGMA>(D, 0, s);
    col_pass<COL_TBAR>(D, 0, s);
    // distance gradient (Eq. 5)
    k_dgrad_x<<<wave_blocks(BN), 64 * kWavesPerBlock, 0, s>>>(D);
    if (D.grad_y)
        col_pass<COL_GRAD_Y>(D, 0, s);
}

} // namespace apml
