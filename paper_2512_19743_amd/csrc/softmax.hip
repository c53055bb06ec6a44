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
#include <type_traits>

#include "apml_internal.h"
#include "device_common.h"
#include "pieces.h"

namespace apml {
namespace {

// G lanes per owner: the larger of two rules. By grid: 8 where the grid of 8
// stays within 2^21 lanes and that of 4 would hold fewer than 2^19 + 1
// (measured: 8 lanes were 45 us faster on 4 x 65536 points and 100 us slower
// on 64 x 8192 points, where they double an already full grid; on 32 x 2048
// points no faster), else 4. By pairs: the largest power of two up to the
// owners' mean pair count, at most 16 (rows of 18 pairs at the unequal
// workload: forward softmax 187 -> 112 us and its adjoint 183 -> 136 us with
// 16 lanes instead of 4).
__host__ inline int softmax_lanes(int64_t owners, int64_t pairs)
{
    int g = owners * 8 <= (int64_t(1) << 21) && owners * 4 > (int64_t(1) << 19) ? 8 : kGroup;
    while (g < 16 && 2 * g * owners <= pairs)
        g *= 2;
    return g;
}

// The forward softmax of one owner (a row, or a column) by its group of G
// lanes. Lane lg sees pairs k = lg, lg + G, ... of the owner's segment; the
// first kSmCache of them are loaded up front (index, the other point's
// coordinates and, for columns, P_row and the flags of the pair) and their
// distances and similarities kept in registers, so the segment is read once.
// Longer segments read the rest again in each step.
constexpr int kSmCache = 8;

// Pair t (row-major position; row i, column j of sample b, the k-th entry of
// its column) with P0 into the per-sample Sinkhorn pieces of both orders.
__device__ __forceinline__ void pack_pair(const DevPlan &d, int b, int j, int k, int i, int t, float p0)
{
    const int roff = t - d.row_ptr[(size_t)b * d.N + i];
    pieces::pack_row_pair(d, d.sink_place, b, i, roff, j, p0);
    pieces::pack_col_pair(d, d.sink_place, b, j, k, i, roff, p0);
}

// dP0/dP_row and dP0/dP_col of a pair with these flags (bit 0: the row
// softmax keeps it, bit 1: the column softmax): P0 = (P_row + P_col)/2 with
// an absent side 0 (Sec. III-A), or, averaging duplicates literally
// (Sec. III-C), the one present value where only one direction keeps it.
__device__ __forceinline__ double sym_weight(const Params &p, uint8_t flags)
{
    return p.sym_mode == kSymMeanDup && flags != 3 ? 1.0 : 0.5;
}

__device__ __forceinline__ double dist3(float ax, float ay, float az, float bx, float by, float bz)
{
    const double dx = (double)ax - (double)bx;
    const double dy = (double)ay - (double)by;
    const double dz = (double)az - (double)bz;
    return sqrt(dx * dx + dy * dy + dz * dz);
}

// ROWS: owner r = b*N + i over row-major pairs t (the other index is the
// column j); else owner gc = b*M + j over column-major entries q (the other
// index is the row i, the row-major position t = csc_perm[q]).
template <bool ROWS, int G>
__device__ __forceinline__ void owner_softmax(const DevPlan &d, const Params &p, int o, int lg)
{
    const int n_own = ROWS ? d.N : d.M, n_oth = ROWS ? d.M : d.N;
    const int b = o / n_own;
    const float *own = (ROWS ? d.x : d.y) + (size_t)o * 3;
    const float *oth = (ROWS ? d.y : d.x) + (size_t)b * n_oth * 3;
    const int32_t *ptr = ROWS ? d.row_ptr : d.col_ptr;
    const int32_t *idx = ROWS ? d.csr_col : d.csc_row;
    const int s0 = ptr[o], n = ptr[o + 1] - s0;
    const float a0 = own[0], a1 = own[1], a2 = own[2];
    const float2 m = ROWS ? d.m12_row[o] : d.m12_col[o];
    const double lk = ROWS ? p.lk_row : p.lk_col;

    int oi[kSmCache], tt[kSmCache];
    float ox[kSmCache], oy[kSmCache], oz[kSmCache], prow[kSmCache];
    uint8_t fl[kSmCache];
#pragma unroll
    for (int c = 0; c < kSmCache; ++c) {
        const int k = lg + G * c;
        oi[c] = k < n ? idx[s0 + k] : 0;
        tt[c] = ROWS ? s0 + k : (k < n ? d.csc_perm[s0 + k] : 0);
    }
#pragma unroll
    for (int c = 0; c < kSmCache; ++c) {
        const int k = lg + G * c;
        const float *q = oth + 3 * (size_t)oi[c];
        ox[c] = q[0];
        oy[c] = q[1];
        oz[c] = q[2];
        if (!ROWS) {
            prow[c] = k < n ? d.p_row[tt[c]] : 0.0f;
            fl[c] = k < n ? d.flags[tt[c]] : 0;
        }
    }
    auto other = [&](int k, float &x, float &y, float &z) {
        const float *q = oth + 3 * (size_t)idx[s0 + k];
        x = q[0];
        y = q[1];
        z = q[2];
    };

    // minimum and second minimum among the stored pairs (single precision)
    Argmins<G> am;
#pragma unroll
    for (int c = 0; c < kSmCache; ++c)
        if (lg + G * c < n)
            am.see(s0 + lg + G * c, sqdist_f32(a0, a1, a2, ox[c], oy[c], oz[c]), m);
    for (int k = lg + G * kSmCache; k < n; k += G) {
        float x, y, z;
        other(k, x, y, z);
        am.see(s0 + k, sqdist_f32(a0, a1, a2, x, y, z), m);
    }
    int q1, q2;
    am.resolve(&q1, &q2);
    if (q1 == INT_MAX || q2 == INT_MAX) { // cannot happen: both minima are always emitted
        if (lg == 0) {
            atomicOr(&d.ctr->error, ROWS ? 1u : 2u);
            (ROWS ? d.T_row : d.T_col)[o] = 0.0;
            (ROWS ? d.C1_row : d.C1_col)[o] = 0.0;
            (ROWS ? d.g_row : d.g_col)[o] = 1.0;
            (ROWS ? d.pos_row : d.pos_col)[2 * (size_t)o] = -1;
            (ROWS ? d.pos_row : d.pos_col)[2 * (size_t)o + 1] = -1;
            (ROWS ? d.clamp_row : d.clamp_col)[o] = 1;
        }
        for (int k = lg; k < n; k += G) {
            if (ROWS) {
                d.cost[s0 + k] = 0.0;
                d.p_row[s0 + k] = 0.0f;
                d.flags[s0 + k] = 0;
            } else {
                const int t = d.csc_perm[s0 + k];
                d.p_col[s0 + k] = 0.0f;
                const float p0 = (float)(sym_weight(p, d.flags[t]) * d.p_row[t]);
                d.p0c[s0 + k] = d.p0r[t] = p0;
                if (d.sink_place)
                    pack_pair(d, b, (int)(o - (int64_t)b * n_own), k, idx[s0 + k], t, p0);
            }
        }
        return;
    }
    double dc[kSmCache];
#pragma unroll
    for (int c = 0; c < kSmCache; ++c) // only where the lane holds a pair: slots past the segment cost nothing
        dc[c] = lg + G * c < n ? dist3(a0, a1, a2, ox[c], oy[c], oz[c]) : 0.0;
    auto dist_at = [&](int q) { // distance of the pair at position q of the segment array
        const int k = q - s0;
        if (k < G * kSmCache) { // held by one lane of the group
            double v = 0.0;
#pragma unroll
            for (int c = 0; c < kSmCache; ++c)
                v += lg + G * c == k ? dc[c] : 0.0;
            return group_sum<G>(v);
        }
        float x, y, z;
        other(k, x, y, z);
        return dist3(a0, a1, a2, x, y, z);
    };
    const double c1 = dist_at(q1), c2 = dist_at(q2);
    const double gap = (c2 - c1) + p.delta;
    // uniform fallback (Sec. III-A): T = 0 makes s = 1 on every pair, all
    // kept, P = 1/K (the emission stored all K pairs of such an owner); like
    // a clamped gap it carries no temperature gradient
    const bool fallback = p.gap_mode == kGapFallback && (c2 - c1) < p.eps_gap;
    const bool clamped = gap < p.eps_gap || fallback;
    const double g = !fallback && clamped ? p.eps_gap : gap;
    const double T = fallback ? 0.0 : lk / g;

    // kept similarities and their sum
    double sv[kSmCache], zsum = 0.0;
#pragma unroll
    for (int c = 0; c < kSmCache; ++c) {
        sv[c] = 0.0;
        if (lg + G * c < n) {
            const double s = exp(-T * (dc[c] - c1));
            sv[c] = s;
            if (s >= p.tau)
                zsum += s;
        }
    }
    for (int k = lg + G * kSmCache; k < n; k += G) {
        float x, y, z;
        other(k, x, y, z);
        const double s = exp(-T * (dist3(a0, a1, a2, x, y, z) - c1));
        if (s >= p.tau)
            zsum += s;
    }
    zsum = group_sum<G>(zsum);

    // P = s / Z on the kept pairs; rows store C, columns P0 = (P_row + P_col)/2
    auto write = [&](int k, int t, double c, double s, float pr, uint8_t f) {
        const bool keep = s >= p.tau;
        const double pk = keep ? s / zsum : 0.0;
        if (ROWS) {
            d.cost[t] = c;
            d.p_row[t] = (float)pk;
            d.flags[t] = keep ? 1 : 0;
        } else {
            const int q = s0 + k;
            d.flags[t] = (uint8_t)(f | (keep ? 2 : 0));
            const float p0 = (float)(sym_weight(p, (uint8_t)(f | (keep ? 2 : 0))) * ((double)pr + pk));
            d.p_col[q] = (float)pk;
            d.p0c[q] = p0;
            d.p0r[t] = p0;
            if (d.sink_place)
                pack_pair(d, b, (int)(o - (int64_t)b * n_own), k, idx[q], t, p0);
        }
    };
#pragma unroll
    for (int c = 0; c < kSmCache; ++c)
        if (lg + G * c < n)
            write(lg + G * c, tt[c], dc[c], sv[c], prow[c], fl[c]);
    for (int k = lg + G * kSmCache; k < n; k += G) {
        float x, y, z;
        other(k, x, y, z);
        const double c = dist3(a0, a1, a2, x, y, z);
        const int t = ROWS ? s0 + k : d.csc_perm[s0 + k];
        write(k, t, c, exp(-T * (c - c1)), ROWS ? 0.0f : d.p_row[t], ROWS ? 0 : d.flags[t]);
    }
    if (lg == 0) {
        (ROWS ? d.T_row : d.T_col)[o] = T;
        (ROWS ? d.C1_row : d.C1_col)[o] = c1;
        (ROWS ? d.g_row : d.g_col)[o] = g;
        (ROWS ? d.pos_row : d.pos_col)[2 * (size_t)o] = q1;
        (ROWS ? d.pos_row : d.pos_col)[2 * (size_t)o + 1] = q2;
        (ROWS ? d.clamp_row : d.clamp_col)[o] = clamped;
    }
}

template <int G> __global__ __launch_bounds__(kBlock) void k_row_softmax(DevPlan d, Params p)
{
    const int gid = xcd_contiguous(blockIdx.x, gridDim.x) * kBlock + threadIdx.x; // a sample's owners share an L2
    const int r = gid / G;
    if (r < d.B * d.N)
        owner_softmax<true, G>(d, p, r, gid % G);
}

template <int G> __global__ __launch_bounds__(kBlock) void k_col_softmax(DevPlan d, Params p)
{
    const int gid = xcd_contiguous(blockIdx.x, gridDim.x) * kBlock + threadIdx.x; // a sample's owners share an L2
    const int gc = gid / G;
    if (gc < d.B * d.M)
        owner_softmax<false, G>(d, p, gc, gid % G);
}

// Column-major view of columns [j0, j1) of sample b in one workgroup: every
// pair of the sample is read and those in the range take a slot of their
// column segment through an LDS counter; the final place of an entry in its
// segment is its rank by row among the segment's entries (one thread per
// entry, so long segments do not serialize a lane). Entries are
// row << 16 | position of the pair in the sample.
constexpr int kCscT = kSinkLanes;

__device__ __forceinline__ void csc_sample(const DevPlan &d, int b, int j0, int j1, uint32_t *lds_csc)
{
    const int tid = threadIdx.x, N = d.N, mc = j1 - j0;
    int *cp = reinterpret_cast<int *>(lds_csc), *fill = cp + (mc + 1);
    const int lo = d.row_ptr[(size_t)b * N], n = d.row_ptr[(size_t)(b + 1) * N] - lo;
    uint32_t *ent = reinterpret_cast<uint32_t *>(fill + mc);
    uint16_t *colof = reinterpret_cast<uint16_t *>(ent + n); // column of each slot, from j0
    for (int k = tid; k <= mc; k += kCscT)
        cp[k] = d.col_ptr[(size_t)b * d.M + j0 + k] - lo; // the sample starts at lo in both orders
    for (int k = tid; k < mc; k += kCscT)
        fill[k] = 0;
    __syncthreads();
    const int c0 = cp[0], nc = cp[mc] - c0; // slots of the range start at c0
    constexpr int kBatch = 8;               // pairs per thread whose loads are in flight together
    for (int t0 = 0; t0 < n; t0 += kBatch * kCscT) {
        int j[kBatch], i[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int t = t0 + u * kCscT + tid;
            j[u] = t < n ? d.csr_col[lo + t] - j0 : -1;
            i[u] = t < n ? d.csr_row[lo + t] - b * N : 0;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int t = t0 + u * kCscT + tid;
            if ((unsigned)j[u] < (unsigned)mc) {
                const int q = cp[j[u]] - c0 + atomicAdd(&fill[j[u]], 1);
                ent[q] = (uint32_t)i[u] << 16 | (uint32_t)t;
                colof[q] = (uint16_t)j[u];
            }
        }
    }
    __syncthreads();
    for (int q = tid; q < nc; q += kCscT) {
        const uint32_t e = ent[q];
        const int j = colof[q], s0 = cp[j], s1 = cp[j + 1];
        int rank = 0;
        for (int u = s0 - c0; u < s1 - c0; ++u)
            rank += ent[u] < e;
        d.csc_row[lo + s0 + rank] = (int)(e >> 16);
        d.csc_perm[lo + s0 + rank] = lo + (int)(e & 0xFFFFu);
        d.csc_col[lo + s0 + rank] = b * d.M + j0 + j;
    }
}

// The column-major view of each sample (first B * parts blocks, `parts`
// column ranges per sample) and the row softmax (the other blocks, kCscT / G
// rows each): independent work in one launch, so the row softmax runs on the
// CUs the per-sample blocks leave free.
template <int G> __global__ __launch_bounds__(kCscT) void k_csc_rows(DevPlan d, Params p, int parts)
{
    extern __shared__ uint32_t lds_csc[];
    if ((int)blockIdx.x < d.B * parts) {
        const int b = blockIdx.x / parts, part = blockIdx.x % parts;
        csc_sample(d, b, (int)((int64_t)d.M * part / parts), (int)((int64_t)d.M * (part + 1) / parts), lds_csc);
        return;
    }
    const int gid = (blockIdx.x - d.B * parts) * kCscT + threadIdx.x;
    const int r = gid / G;
    if (r < d.B * d.N)
        owner_softmax<true, G>(d, p, r, gid % G);
}

__host__ inline size_t csc_sample_lds(int M, int64_t max_pairs)
{
    return 4 * (2 * (size_t)M + 1) + 6 * (size_t)max_pairs + 16;
}

// dLoss/dP0 of stored pair t: the Sinkhorn adjoint, or grad_loss * C when
// there are no Sinkhorn iterations.
__device__ __forceinline__ double p0bar(const DevPlan &d, int t, double gl)
{
    return d.L == 0 ? gl * d.cost[t] : d.adj[t];
}

// Backward of one owner's softmax by its group of G lanes, with the first
// pairs of each lane loaded up front (as in the forward).
//   columns: cbar_t = -T P_col (Pbar_t - sigma) on kept pairs, plus the gap
//            term at the two argmins; written per pair (cbar).
//   rows:    the same for P_row, plus cbar from the columns and the direct
//            term grad_loss * v; then Eq. 5 turns cbar into grad_x.
// DP: P in double, formed again as the forward formed it before storing it in
// single precision (same operations and lane order, so the same sum Z). The
// temperature adjoint cancels, and it reaches the argmins multiplied by T / g,
// large for a small gap: with stored single-precision P the gradient error
// reached 5e-4 there, and 9e-6 on 16 x 4096 x 16384 points (1.2e-7 with DP).
// Taken where the reverse sweeps keep the adjoint in double (or there are
// none); the sweeps that keep it in LDS store it in single precision, which
// then bounds the error as much (32 samples of 2048 points: 6.7e-6 either
// way), and P is read as stored. Both cache 4 pairs per lane (the forward 8):
// four or more waves per SIMD instead of three (the row kernel held 158
// registers with 8), and owners rarely have more than 4 pairs per lane
// (64 samples of 8192 points: adjoint 0.157 -> 0.134 ms; 32 of 2048:
// 0.0338 -> 0.0331 ms).
constexpr int kBwdCache = 4;

template <bool DP> struct BwdP {
    static constexpr int kCache = kBwdCache;
    using T = std::conditional_t<DP, double, float>; // type of the cached P
};

template <int G, bool DP> __global__ __launch_bounds__(kBlock) void k_bwd_col_softmax(DevPlan d, Params p)
{
    constexpr int NC = BwdP<DP>::kCache;
    using PT = typename BwdP<DP>::T;
    const int gid = xcd_contiguous(blockIdx.x, gridDim.x) * kBlock + threadIdx.x; // a sample's owners share an L2
    const int gc = gid / G, lg = gid % G;
    if (gc >= d.B * d.M)
        return;
    const int b = gc / d.M;
    const double gl = d.grad_loss[b];
    const int s0 = d.col_ptr[gc], n = d.col_ptr[gc + 1] - s0;
    const double T = d.T_col[gc], c1 = d.C1_col[gc];
    const double gapbar_scale = d.clamp_col[gc] || p.tgrad_mode == kTgradDetached ? 0.0 : -T / d.g_col[gc];
    const int q1 = d.pos_col[2 * (size_t)gc], q2 = d.pos_col[2 * (size_t)gc + 1];
    const float *yc = d.y + (size_t)gc * 3;
    const float y0 = yc[0], y1 = yc[1], y2 = yc[2];
    const float *xb = d.x + (size_t)b * d.N * 3;

    int tq[NC], iq[NC];
    PT pq[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int k = lg + G * c;
        tq[c] = k < n ? d.csc_perm[s0 + k] : 0;
        iq[c] = k < n ? d.csc_row[s0 + k] : 0;
        if constexpr (!DP)
            pq[c] = k < n ? d.p_col[s0 + k] : 0.0f;
    }
    double aq[NC], cq[NC];
    bool kq[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int k = lg + G * c;
        const uint8_t f = k < n ? d.flags[tq[c]] : 0;
        kq[c] = (f & 2) != 0;
        aq[c] = kq[c] ? sym_weight(p, f) * p0bar(d, tq[c], gl) : 0.0;
        const float *xi = xb + 3 * (size_t)iq[c];
        cq[c] = kq[c] ? dist3(xi[0], xi[1], xi[2], y0, y1, y2) : 0.0;
    }
    double zsum = 0.0;
    if constexpr (DP) {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            pq[c] = kq[c] ? exp(-T * (cq[c] - c1)) : 0.0;
            zsum += pq[c];
        }
        for (int k = lg + G * NC; k < n; k += G) {
            const int t = d.csc_perm[s0 + k];
            if (d.flags[t] & 2)
                zsum += exp(-T * (d.cost[t] - c1));
        }
        zsum = group_sum<G>(zsum);
#pragma unroll
        for (int c = 0; c < NC; ++c)
            pq[c] = kq[c] ? pq[c] / zsum : 0.0;
    }
    // P of a kept pair past the cached ones (column-major entry q, row-major position t)
    auto p_at = [&](int q, int t) -> double {
        if constexpr (DP)
            return exp(-T * (d.cost[t] - c1)) / zsum;
        else
            return (double)d.p_col[q];
    };
    double sigma = 0.0;
#pragma unroll
    for (int c = 0; c < NC; ++c)
        sigma += kq[c] ? (double)pq[c] * aq[c] : 0.0;
    for (int k = lg + G * NC; k < n; k += G) {
        const int t = d.csc_perm[s0 + k];
        const uint8_t f = d.flags[t];
        if (f & 2)
            sigma += p_at(s0 + k, t) * (sym_weight(p, f) * p0bar(d, t, gl));
    }
    sigma = group_sum<G>(sigma);
    double tbar = 0.0;
#pragma unroll
    for (int c = 0; c < NC; ++c)
        tbar -= kq[c] ? (double)pq[c] * (aq[c] - sigma) * (cq[c] - c1) : 0.0;
    for (int k = lg + G * NC; k < n; k += G) {
        const int t = d.csc_perm[s0 + k];
        const uint8_t f = d.flags[t];
        if (f & 2)
            tbar -= p_at(s0 + k, t) * (sym_weight(p, f) * p0bar(d, t, gl) - sigma) * (d.cost[t] - c1);
    }
    tbar = group_sum<G>(tbar);
    const double gapbar = gapbar_scale * tbar;
    auto gap_terms = [&](int q, double cb) {
        if (q == q2)
            cb += gapbar;
        if (q == q1)
            cb -= gapbar;
        return cb;
    };
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int k = lg + G * c;
        if (k < n)
            d.cbar[tq[c]] = gap_terms(s0 + k, kq[c] ? -T * (double)pq[c] * (aq[c] - sigma) : 0.0);
    }
    for (int k = lg + G * NC; k < n; k += G) {
        const int t = d.csc_perm[s0 + k];
        const uint8_t f = d.flags[t];
        const double cb = (f & 2) ? -T * p_at(s0 + k, t) * (sym_weight(p, f) * p0bar(d, t, gl) - sigma) : 0.0;
        d.cbar[t] = gap_terms(s0 + k, cb);
    }
}

template <int G, bool DP>
__global__ __launch_bounds__(kBlock) void k_bwd_row_softmax(DevPlan d, Params p, int keep_cbar)
{
    constexpr int NC = BwdP<DP>::kCache;
    using PT = typename BwdP<DP>::T;
    const int gid = xcd_contiguous(blockIdx.x, gridDim.x) * kBlock + threadIdx.x; // a sample's owners share an L2
    const int r = gid / G, lg = gid % G;
    if (r >= d.B * d.N)
        return;
    const int b = r / d.N;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * d.M;
    const float *xr = d.x + (size_t)r * 3;
    const float x0 = xr[0], x1 = xr[1], x2 = xr[2];
    const float *yb = d.y + (size_t)b * d.M * 3;
    const double gl = d.grad_loss[b];
    const int t0 = d.row_ptr[r], n = d.row_ptr[r + 1] - t0;
    const double T = d.T_row[r], c1 = d.C1_row[r];
    const double gscale = d.clamp_row[r] || p.tgrad_mode == kTgradDetached ? 0.0 : -T / d.g_row[r];
    const int q1 = d.pos_row[2 * (size_t)r], q2 = d.pos_row[2 * (size_t)r + 1];
    const double al = d.alpha[(size_t)d.L * BN + r];
    const double *bl = d.beta + (size_t)d.L * BM + (size_t)b * d.M;

    int jq[NC];
    bool kq[NC];
    float p0q[NC];
    PT pq[NC];
    double aq[NC], cq[NC], cbq[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int k = lg + G * c, t = t0 + k;
        const bool in = k < n;
        jq[c] = in ? d.csr_col[t] : 0;
        const uint8_t f = in ? d.flags[t] : 0;
        kq[c] = (f & 1) != 0;
        if constexpr (!DP) {
            pq[c] = in ? d.p_row[t] : 0.0f;
            cbq[c] = in ? d.cbar[t] : 0.0; // DP reads it where it is used
        }
        p0q[c] = in ? d.p0r[t] : 0.0f;
        aq[c] = in ? sym_weight(p, f) * p0bar(d, t, gl) : 0.0;
        cq[c] = in ? d.cost[t] : 1.0;
    }
    double zsum = 0.0;
    if constexpr (DP) {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            pq[c] = kq[c] ? exp(-T * (cq[c] - c1)) : 0.0;
            zsum += pq[c];
        }
        for (int k = lg + G * NC; k < n; k += G)
            if (d.flags[t0 + k] & 1)
                zsum += exp(-T * (d.cost[t0 + k] - c1));
        zsum = group_sum<G>(zsum);
#pragma unroll
        for (int c = 0; c < NC; ++c)
            pq[c] = kq[c] ? pq[c] / zsum : 0.0;
    }
    // P of a kept pair past the cached ones
    auto p_at = [&](int t) -> double {
        if constexpr (DP)
            return exp(-T * (d.cost[t] - c1)) / zsum;
        else
            return (double)d.p_row[t];
    };
    double sigma = 0.0;
#pragma unroll
    for (int c = 0; c < NC; ++c)
        sigma += kq[c] ? (double)pq[c] * aq[c] : 0.0;
    for (int k = lg + G * NC; k < n; k += G) {
        const int t = t0 + k;
        const uint8_t f = d.flags[t];
        if (f & 1)
            sigma += p_at(t) * (sym_weight(p, f) * p0bar(d, t, gl));
    }
    sigma = group_sum<G>(sigma);
    double tbar = 0.0;
#pragma unroll
    for (int c = 0; c < NC; ++c)
        tbar -= kq[c] ? (double)pq[c] * (aq[c] - sigma) * (cq[c] - c1) : 0.0;
    for (int k = lg + G * NC; k < n; k += G) {
        const int t = t0 + k;
        const uint8_t f = d.flags[t];
        if (f & 1)
            tbar -= p_at(t) * (sym_weight(p, f) * p0bar(d, t, gl) - sigma) * (d.cost[t] - c1);
    }
    tbar = group_sum<G>(tbar);
    const double gapbar = gscale * tbar;
    double gx = 0.0, gy = 0.0, gz = 0.0;
    // cbar of pair t (column part cb0, P_row, dL/dP0, cost, P0, column j) into grad_x (Eq. 5)
    auto add = [&](int t, int j, double cb0, bool kept, double prow, double a, double c, float p0) {
        double cb = cb0 + gl * (al * (double)p0 * bl[j]);
        if (kept)
            cb -= T * prow * (a - sigma);
        if (t == q2)
            cb += gapbar;
        if (t == q1)
            cb -= gapbar;
        const float *yj = yb + 3 * (size_t)j;
        const double w = cb / (c + p.eps_dist); // Eq. 5
        gx += w * ((double)x0 - (double)yj[0]);
        gy += w * ((double)x1 - (double)yj[1]);
        gz += w * ((double)x2 - (double)yj[2]);
        if (keep_cbar)
            d.cbar[t] = cb;
    };
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int k = lg + G * c;
        if (k < n)
            add(t0 + k, jq[c], DP ? d.cbar[t0 + k] : cbq[c], kq[c], (double)pq[c], aq[c], cq[c], p0q[c]);
    }
    for (int k = lg + G * NC; k < n; k += G) {
        const int t = t0 + k;
        const uint8_t f = d.flags[t];
        const bool kept = (f & 1) != 0;
        add(t, d.csr_col[t], d.cbar[t], kept, kept ? p_at(t) : 0.0, sym_weight(p, f) * p0bar(d, t, gl), d.cost[t],
            d.p0r[t]);
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

template <int G> __global__ __launch_bounds__(kBlock) void k_bwd_grad_y(DevPlan d, Params p)
{
    const int gid = xcd_contiguous(blockIdx.x, gridDim.x) * kBlock + threadIdx.x; // a sample's owners share an L2
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

bool csc_sample_fits(int N, int M, int64_t max_pairs)
{
    return N <= 65536 && max_pairs <= 65536 && csc_sample_lds(M, max_pairs) <= 160 * 1024;
}

// Launches kernel template K with the lanes per owner of `owners`.
#define APML_LAUNCH_G(K, owners, pairs, per_block, shmem, s, ...)                                                   \
    do {                                                                                                           \
        const int g_ = softmax_lanes(owners, pairs);                                                               \
        const dim3 grid_(blocks_for((int64_t)(owners) * g_, per_block));                                           \
        if (g_ == 16)                                                                                              \
            hipLaunchKernelGGL(K<16>, grid_, dim3(per_block), shmem, s, __VA_ARGS__);                              \
        else if (g_ == 8)                                                                                          \
            hipLaunchKernelGGL(K<8>, grid_, dim3(per_block), shmem, s, __VA_ARGS__);                               \
        else                                                                                                       \
            hipLaunchKernelGGL(K<kGroup>, grid_, dim3(per_block), shmem, s, __VA_ARGS__);                          \
    } while (0)

// The same for a kernel template with a second, boolean parameter X.
#define APML_LAUNCH_GP(K, X, owners, pairs, s, ...)                                                                 \
    do {                                                                                                           \
        const int g_ = softmax_lanes(owners, pairs);                                                               \
        const dim3 grid_(blocks_for((int64_t)(owners) * g_, kBlock));                                              \
        if (g_ == 16)                                                                                              \
            hipLaunchKernelGGL((K<16, X>), grid_, dim3(kBlock), 0, s, __VA_ARGS__);                                \
        else if (g_ == 8)                                                                                          \
            hipLaunchKernelGGL((K<8, X>), grid_, dim3(kBlock), 0, s, __VA_ARGS__);                                 \
        else                                                                                                       \
            hipLaunchKernelGGL((K<kGroup, X>), grid_, dim3(kBlock), 0, s, __VA_ARGS__);                            \
    } while (0)

hipError_t launch_csc_and_softmax(const DevPlan &d, const Params &p, int64_t max_pairs, hipStream_t s)
{
    const size_t bytes = csc_sample_lds(d.M, max_pairs);
    const int64_t BN = (int64_t)d.B * d.N;
    const int gr = softmax_lanes(BN, d.nnz);
    const void *k = gr == 16  ? (const void *)k_csc_rows<16>
                    : gr == 8 ? (const void *)k_csc_rows<8>
                              : (const void *)k_csc_rows<kGroup>;
    hipError_t e = set_dynamic_lds(k, bytes);
    if (e != hipSuccess)
        return e;
    const unsigned rows = blocks_for(BN * gr, kCscT);
    // Two column ranges per sample while that still leaves CUs for the row
    // softmax: at 32 samples of 2048 points this took this launch and the
    // column softmax together from 44.5 to 42.0 us (four ranges: 42.8); each
    // range reads all of its sample's pairs.
    const int parts = 2 * d.B <= 256 ? 2 : 1;
    const dim3 grid(d.B * parts + rows);
    if (gr == 16)
        hipLaunchKernelGGL(k_csc_rows<16>, grid, dim3(kCscT), bytes, s, d, p, parts);
    else if (gr == 8)
        hipLaunchKernelGGL(k_csc_rows<8>, grid, dim3(kCscT), bytes, s, d, p, parts);
    else
        hipLaunchKernelGGL(k_csc_rows<kGroup>, grid, dim3(kCscT), bytes, s, d, p, parts);
    APML_LAUNCH_G(k_col_softmax, (int64_t)d.B * d.M, d.nnz, kBlock, 0, s, d, p);
    return hipGetLastError();
}

void launch_softmax(const DevPlan &d, const Params &p, hipStream_t s)
{
    APML_LAUNCH_G(k_row_softmax, (int64_t)d.B * d.N, d.nnz, kBlock, 0, s, d, p);
    APML_LAUNCH_G(k_col_softmax, (int64_t)d.B * d.M, d.nnz, kBlock, 0, s, d, p);
}

void launch_bwd_softmax(const DevPlan &d, const Params &p, bool double_p, hipStream_t s)
{
    const int keep = d.grad_y != nullptr ? 1 : 0;
    if (double_p) {
        APML_LAUNCH_GP(k_bwd_col_softmax, true, (int64_t)d.B * d.M, d.nnz, s, d, p);
        APML_LAUNCH_GP(k_bwd_row_softmax, true, (int64_t)d.B * d.N, d.nnz, s, d, p, keep);
    } else {
        APML_LAUNCH_GP(k_bwd_col_softmax, false, (int64_t)d.B * d.M, d.nnz, s, d, p);
        APML_LAUNCH_GP(k_bwd_row_softmax, false, (int64_t)d.B * d.N, d.nnz, s, d, p, keep);
    }
    if (d.grad_y)
        APML_LAUNCH_G(k_bwd_grad_y, (int64_t)d.B * d.M, d.nnz, kBlock, 0, s, d, p);
}

#undef APML_LAUNCH_G
#undef APML_LAUNCH_GP

} // namespace apml
