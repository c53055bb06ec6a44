// Temperatures, adaptive softmaxes and the symmetrized plan on the stored
// pairs, and their adjoints. Each row (or column) is handled by a group of
// kGroup lanes that stride over its segment; group sums use a butterfly, so
// results do not depend on scheduling.
//
// Forward (Alg. 1 steps 1-3):
//   k_row_softmax  minimum and second minimum located among the row's stored
//                  pairs by the single-precision distance; C1, C2 in double;
//                  g = max(C2 - C1 + delta, eps_gap); T = L_K / g (Eq. 1);
//                  s = exp(-T (C - C1)), kept iff s >= tau (Sec. III-B);
//                  P_row = s / (sum of kept s) (Sec. III-C). Stores C per pair.
//   k_col_softmax  the same per column, then P0 = (P_row + P_col)/2
//                  (Sec. III-A) on the union of both kept sets.
// Backward (Sec. III-D; reverse mode of the above):
//   k_bwd_col_softmax, k_bwd_row_softmax: with P = s/Z over the kept set,
//     abar = P (Pbar - sum P Pbar); Cbar -= T abar; Tbar -= sum abar (C - C1);
//     T = L_K / g: gbar = -Tbar T / g reaches C of the second minimum (+) and
//     of the minimum (-) unless the gap was clamped; plus the direct term
//     grad_loss * v of loss = sum v C; the row kernel turns Cbar into grad_x
//     with Eq. 5, k_bwd_grad_y into grad_y.
#include "apml_internal.h"
#include "device_common.h"

namespace apml {
namespace {

constexpr int G = kGroup;

__global__ __launch_bounds__(kBlock) void k_row_softmax(DevPlan d, Params p)
{
    const int gid = blockIdx.x * kBlock + threadIdx.x;
    const int r = gid / G, lg = gid % G;
    if (r >= d.B * d.N)
        return;
    const int b = r / d.N;
    const float *xr = d.x + (size_t)r * 3;
    const float x0 = xr[0], x1 = xr[1], x2 = xr[2];
    const float *yb = d.y + (size_t)b * d.M * 3;
    const float2 m = d.m12_row[r];
    const int t0 = d.row_ptr[r], t1 = d.row_ptr[r + 1];
    Argmins<G> am;
    for (int t = t0 + lg; t < t1; t += G) {
        const float *yj = yb + 3 * (size_t)d.csr_col[t];
        am.see(t, sqdist_f32(x0, x1, x2, yj[0], yj[1], yj[2]), m);
    }
    int q1, q2;
    am.resolve(&q1, &q2);
    if (q1 == INT_MAX || q2 == INT_MAX) { // cannot happen: both minima are always emitted
        if (lg == 0) {
            atomicOr(&d.ctr->error, 1u);
            d.T_row[r] = 0.0;
            d.C1_row[r] = 0.0;
            d.g_row[r] = 1.0;
            d.pos_row[2 * (size_t)r] = d.pos_row[2 * (size_t)r + 1] = -1;
            d.clamp_row[r] = 1;
        }
        for (int t = t0 + lg; t < t1; t += G) {
            d.cost[t] = 0.0;
            d.p_row[t] = 0.0f;
            d.flags[t] = 0;
        }
        return;
    }
    const double c1 = dist_f64(xr, yb + 3 * (size_t)d.csr_col[q1]);
    const double c2 = dist_f64(xr, yb + 3 * (size_t)d.csr_col[q2]);
    const double gap = (c2 - c1) + p.delta;
    const bool clamped = gap < p.eps_gap;
    const double g = clamped ? p.eps_gap : gap;
    const double T = p.lk_row / g;
    double z = 0.0;
    for (int t = t0 + lg; t < t1; t += G) {
        const double c = dist_f64(xr, yb + 3 * (size_t)d.csr_col[t]);
        d.cost[t] = c;
        const double s = exp(-T * (c - c1));
        if (s >= p.tau)
            z += s;
    }
    z = group_sum<G>(z);
    for (int t = t0 + lg; t < t1; t += G) {
        const double s = exp(-T * (d.cost[t] - c1));
        const bool keep = s >= p.tau;
        d.p_row[t] = keep ? (float)(s / z) : 0.0f;
        d.flags[t] = keep ? 1 : 0;
    }
    if (lg == 0) {
        d.T_row[r] = T;
        d.C1_row[r] = c1;
        d.g_row[r] = g;
        d.pos_row[2 * (size_t)r] = q1;
        d.pos_row[2 * (size_t)r + 1] = q2;
        d.clamp_row[r] = clamped;
    }
}

// Columns of at most G * kColCache pairs keep their pairs in registers (one
// pass over the column's data instead of three); the cost of a pair is
// recomputed from the coordinates, bitwise as the row kernel computed it,
// instead of being gathered from the row-major array.
constexpr int kColCache = 4;

__global__ __launch_bounds__(kBlock) void k_col_softmax(DevPlan d, Params p)
{
    const int gid = blockIdx.x * kBlock + threadIdx.x;
    const int gc = gid / G, lg = gid % G;
    if (gc >= d.B * d.M)
        return;
    const int b = gc / d.M;
    const float *yc = d.y + (size_t)gc * 3;
    const float y0 = yc[0], y1 = yc[1], y2 = yc[2];
    const float *xb = d.x + (size_t)b * d.N * 3;
    const float2 m = d.m12_col[gc];
    const int s0 = d.col_ptr[gc], s1 = d.col_ptr[gc + 1];
    const bool cached = s1 - s0 <= G * kColCache; // the same for the whole group
    Argmins<G> am;
    int tq[kColCache];
    double cq[kColCache];
    if (cached) {
#pragma unroll
        for (int k = 0; k < kColCache; ++k) {
            const int q = s0 + lg + G * k;
            tq[k] = -1;
            cq[k] = 0.0;
            if (q < s1) {
                const float *xi = xb + 3 * (size_t)d.csc_row[q];
                am.see(q, sqdist_f32(y0, y1, y2, xi[0], xi[1], xi[2]), m);
                cq[k] = dist_f64(xi, yc);
                tq[k] = d.csc_perm[q];
            }
        }
    } else {
        for (int q = s0 + lg; q < s1; q += G) {
            const float *xi = xb + 3 * (size_t)d.csc_row[q];
            am.see(q, sqdist_f32(y0, y1, y2, xi[0], xi[1], xi[2]), m);
        }
    }
    int q1, q2;
    am.resolve(&q1, &q2);
    if (q1 == INT_MAX || q2 == INT_MAX) {
        if (lg == 0) {
            atomicOr(&d.ctr->error, 2u);
            d.T_col[gc] = 0.0;
            d.C1_col[gc] = 0.0;
            d.g_col[gc] = 1.0;
            d.pos_col[2 * (size_t)gc] = d.pos_col[2 * (size_t)gc + 1] = -1;
            d.clamp_col[gc] = 1;
        }
        for (int q = s0 + lg; q < s1; q += G) {
            const int t = d.csc_perm[q];
            d.p_col[q] = 0.0f;
            d.p0c[q] = d.p0r[t] = 0.5f * d.p_row[t];
        }
        return;
    }
    double c1, c2;
    if (cached) {
        double a1 = 0.0, a2 = 0.0;
#pragma unroll
        for (int k = 0; k < kColCache; ++k) {
            const int q = s0 + lg + G * k;
            a1 += q == q1 ? cq[k] : 0.0;
            a2 += q == q2 ? cq[k] : 0.0;
        }
        c1 = group_sum<G>(a1); // one lane holds it, the others add zeros
        c2 = group_sum<G>(a2);
    } else {
        c1 = d.cost[d.csc_perm[q1]];
        c2 = d.cost[d.csc_perm[q2]];
    }
    const double gap = (c2 - c1) + p.delta;
    const bool clamped = gap < p.eps_gap;
    const double g = clamped ? p.eps_gap : gap;
    const double T = p.lk_col / g;
    double z = 0.0;
    if (cached) {
#pragma unroll
        for (int k = 0; k < kColCache; ++k)
            if (tq[k] >= 0) {
                const double s = exp(-T * (cq[k] - c1));
                if (s >= p.tau)
                    z += s;
            }
    } else {
        for (int q = s0 + lg; q < s1; q += G) {
            const double s = exp(-T * (d.cost[d.csc_perm[q]] - c1));
            if (s >= p.tau)
                z += s;
        }
    }
    z = group_sum<G>(z);
    auto write = [&](int q, int t, double c) {
        const double s = exp(-T * (c - c1));
        const bool keep = s >= p.tau;
        const double pc = keep ? s / z : 0.0;
        d.flags[t] = (uint8_t)(d.flags[t] | (keep ? 2 : 0));
        const float p0 = (float)(0.5 * ((double)d.p_row[t] + pc));
        d.p_col[q] = (float)pc;
        d.p0c[q] = p0;
        d.p0r[t] = p0;
    };
    if (cached) {
#pragma unroll
        for (int k = 0; k < kColCache; ++k)
            if (tq[k] >= 0)
                write(s0 + lg + G * k, tq[k], cq[k]);
    } else {
        for (int q = s0 + lg; q < s1; q += G) {
            const int t = d.csc_perm[q];
            write(q, t, d.cost[t]);
        }
    }
    if (lg == 0) {
        d.T_col[gc] = T;
        d.C1_col[gc] = c1;
        d.g_col[gc] = g;
        d.pos_col[2 * (size_t)gc] = q1;
        d.pos_col[2 * (size_t)gc + 1] = q2;
        d.clamp_col[gc] = clamped;
    }
}

// dLoss/dP0 of stored pair t: the Sinkhorn adjoint, or grad_loss * C when
// there are no Sinkhorn iterations.
__device__ __forceinline__ double p0bar(const DevPlan &d, int t, double gl)
{
    return d.L == 0 ? gl * d.cost[t] : d.adj[t];
}

__global__ __launch_bounds__(kBlock) void k_bwd_col_softmax(DevPlan d, Params p)
{
    const int gid = blockIdx.x * kBlock + threadIdx.x;
    const int gc = gid / G, lg = gid % G;
    if (gc >= d.B * d.M)
        return;
    const int b = gc / d.M;
    const double gl = d.grad_loss[b];
    const int s0 = d.col_ptr[gc], s1 = d.col_ptr[gc + 1];
    const double T = d.T_col[gc], c1 = d.C1_col[gc];
    const double gapbar_scale = d.clamp_col[gc] ? 0.0 : -T / d.g_col[gc];
    const int q1 = d.pos_col[2 * (size_t)gc], q2 = d.pos_col[2 * (size_t)gc + 1];
    if (s1 - s0 <= G * kColCache) {
        // one pass over the column's data: kept pairs' P_col, dL/dP0 and cost in registers
        const float *yc = d.y + (size_t)gc * 3;
        const float *xb = d.x + (size_t)b * d.N * 3;
        int tq[kColCache];
        double pq[kColCache], aq[kColCache], cq[kColCache];
        double sigma = 0.0;
#pragma unroll
        for (int k = 0; k < kColCache; ++k) {
            const int q = s0 + lg + G * k;
            tq[k] = -1;
            pq[k] = aq[k] = cq[k] = 0.0;
            if (q < s1) {
                const int t = d.csc_perm[q];
                tq[k] = t;
                if (d.flags[t] & 2) {
                    pq[k] = (double)d.p_col[q];
                    aq[k] = 0.5 * p0bar(d, t, gl);
                    cq[k] = dist_f64(xb + 3 * (size_t)d.csc_row[q], yc);
                    sigma += pq[k] * aq[k];
                }
            }
        }
        sigma = group_sum<G>(sigma);
        double tbar = 0.0;
#pragma unroll
        for (int k = 0; k < kColCache; ++k)
            tbar -= pq[k] * (aq[k] - sigma) * (cq[k] - c1); // zero for pairs not kept
        tbar = group_sum<G>(tbar);
        const double gapbar = gapbar_scale * tbar;
#pragma unroll
        for (int k = 0; k < kColCache; ++k) {
            const int q = s0 + lg + G * k;
            if (tq[k] >= 0) {
                double cb = -T * pq[k] * (aq[k] - sigma);
                if (q == q2)
                    cb += gapbar;
                if (q == q1)
                    cb -= gapbar;
                d.cbar[tq[k]] = cb;
            }
        }
        return;
    }
    double sigma = 0.0;
    for (int q = s0 + lg; q < s1; q += G) {
        const int t = d.csc_perm[q];
        if (d.flags[t] & 2)
            sigma += (double)d.p_col[q] * 0.5 * p0bar(d, t, gl);
    }
    sigma = group_sum<G>(sigma);
    double tbar = 0.0;
    for (int q = s0 + lg; q < s1; q += G) {
        const int t = d.csc_perm[q];
        if (d.flags[t] & 2) {
            const double ab = (double)d.p_col[q] * (0.5 * p0bar(d, t, gl) - sigma);
            tbar -= ab * (d.cost[t] - c1);
        }
    }
    tbar = group_sum<G>(tbar);
    const double gapbar = gapbar_scale * tbar;
    for (int q = s0 + lg; q < s1; q += G) {
        const int t = d.csc_perm[q];
        double cb = 0.0;
        if (d.flags[t] & 2)
            cb = -T * (double)d.p_col[q] * (0.5 * p0bar(d, t, gl) - sigma);
        if (q == q2)
            cb += gapbar;
        if (q == q1)
            cb -= gapbar;
        d.cbar[t] = cb;
    }
}

__global__ __launch_bounds__(kBlock) void k_bwd_row_softmax(DevPlan d, Params p, int keep_cbar)
{
    const int gid = blockIdx.x * kBlock + threadIdx.x;
    const int r = gid / G, lg = gid % G;
    if (r >= d.B * d.N)
        return;
    const int b = r / d.N;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * d.M;
    const float *xr = d.x + (size_t)r * 3;
    const float *yb = d.y + (size_t)b * d.M * 3;
    const double gl = d.grad_loss[b];
    const int t0 = d.row_ptr[r], t1 = d.row_ptr[r + 1];
    double sigma = 0.0;
    for (int t = t0 + lg; t < t1; t += G)
        if (d.flags[t] & 1)
            sigma += (double)d.p_row[t] * 0.5 * p0bar(d, t, gl);
    sigma = group_sum<G>(sigma);
    const double T = d.T_row[r], c1 = d.C1_row[r];
    double tbar = 0.0;
    for (int t = t0 + lg; t < t1; t += G)
        if (d.flags[t] & 1) {
            const double ab = (double)d.p_row[t] * (0.5 * p0bar(d, t, gl) - sigma);
            tbar -= ab * (d.cost[t] - c1);
        }
    tbar = group_sum<G>(tbar);
    const double gapbar = d.clamp_row[r] ? 0.0 : -tbar * T / d.g_row[r];
    const int q1 = d.pos_row[2 * (size_t)r], q2 = d.pos_row[2 * (size_t)r + 1];
    const double al = d.alpha[(size_t)d.L * BN + r];
    const double *bl = d.beta + (size_t)d.L * BM + (size_t)b * d.M;
    double gx = 0.0, gy = 0.0, gz = 0.0;
    for (int t = t0 + lg; t < t1; t += G) {
        const int j = d.csr_col[t];
        const float *yj = yb + 3 * (size_t)j;
        const double c = d.cost[t];
        double cb = d.cbar[t] + gl * (al * (double)d.p0r[t] * bl[j]);
        if (d.flags[t] & 1)
            cb -= T * (double)d.p_row[t] * (0.5 * p0bar(d, t, gl) - sigma);
        if (t == q2)
            cb += gapbar;
        if (t == q1)
            cb -= gapbar;
        const double w = cb / (c + p.eps_dist); // Eq. 5
        gx += w * ((double)xr[0] - (double)yj[0]);
        gy += w * ((double)xr[1] - (double)yj[1]);
        gz += w * ((double)xr[2] - (double)yj[2]);
        if (keep_cbar)
            d.cbar[t] = cb;
    }
    gx = group_sum<G>(gx);
    gy = group_sum<G>(gy);
    gz = group_sum<G>(gz);
    if (lg == 0) {
        float *o = d.grad_x + (size_t)r * 3;
        o[0] = (float)gx;
        o[1] = (float)gy;
        o[2] = (float)gz;
    }
}

__global__ __launch_bounds__(kBlock) void k_bwd_grad_y(DevPlan d, Params p)
{
    const int gid = blockIdx.x * kBlock + threadIdx.x;
    const int gc = gid / G, lg = gid % G;
    if (gc >= d.B * d.M)
        return;
    const int b = gc / d.M;
    const float *yc = d.y + (size_t)gc * 3;
    const float *xb = d.x + (size_t)b * d.N * 3;
    double gx = 0.0, gy = 0.0, gz = 0.0;
    for (int q = d.col_ptr[gc] + lg; q < d.col_ptr[gc + 1]; q += G) {
        const int t = d.csc_perm[q];
        const float *xi = xb + 3 * (size_t)d.csc_row[q];
        const double w = d.cbar[t] / (d.cost[t] + p.eps_dist);
        gx -= w * ((double)xi[0] - (double)yc[0]);
        gy -= w * ((double)xi[1] - (double)yc[1]);
        gz -= w * ((double)xi[2] - (double)yc[2]);
    }
    gx = group_sum<G>(gx);
    gy = group_sum<G>(gy);
    gz = group_sum<G>(gz);
    if (lg == 0) {
        float *o = d.grad_y + (size_t)gc * 3;
        o[0] = (float)gx;
        o[1] = (float)gy;
        o[2] = (float)gz;
    }
}

} // namespace

void launch_softmax(const DevPlan &d, const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(k_row_softmax, dim3(blocks_for((int64_t)d.B * d.N * G, kBlock)), dim3(kBlock), 0, s,
                       d, p);
    hipLaunchKernelGGL(k_col_softmax, dim3(blocks_for((int64_t)d.B * d.M * G, kBlock)), dim3(kBlock), 0, s,
                       d, p);
}

void launch_bwd_softmax(const DevPlan &d, const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(k_bwd_col_softmax, dim3(blocks_for((int64_t)d.B * d.M * G, kBlock)), dim3(kBlock), 0,
                       s, d, p);
    hipLaunchKernelGGL(k_bwd_row_softmax, dim3(blocks_for((int64_t)d.B * d.N * G, kBlock)), dim3(kBlock), 0,
                       s, d, p, d.grad_y != nullptr ? 1 : 0);
    if (d.grad_y)
        hipLaunchKernelGGL(k_bwd_grad_y, dim3(blocks_for((int64_t)d.B * d.M * G, kBlock)), dim3(kBlock), 0, s,
                           d, p);
}

} // namespace apml
