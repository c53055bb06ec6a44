// Sinkhorn normalisation on the stored pairs (Eq. 3, Eq. 4; Alg. 1 steps
// 4-7), the loss (Sec. III-D) and the reverse Sinkhorn sweeps.
//
// Scaling form. Every column step of Eq. 3 divides a whole column by one
// factor and every row step of Eq. 4 a whole row, so after iteration l the
// plan is v = alpha^l_i P0_ij beta^l_j with
//   beta^l_j  = beta^(l-1)_j  / (beta^(l-1)_j  sum_i alpha^(l-1)_i P0_ij + eps)
//   alpha^l_i = alpha^(l-1)_i / (alpha^(l-1)_i sum_j P0_ij beta^l_j     + eps)
// which is Eq. 3 / Eq. 4 exactly, including eps. A sweep reads P0 and the
// indices once and writes no per-pair values.
//
// Per-sample kernels (N, M <= kCover): one workgroup per sample runs all 2L
// sweeps. Each lane owns SL rows and SL columns. The first kMax pairs of each
// are kept in registers for the whole kernel and the rest in an LDS tail
// buffer, so a lane sums its rows (or columns) sequentially in pair order and
// applies the scaling itself: one workgroup barrier per sweep, no cross-lane
// reduction, bitwise reproducible. The scalings live in LDS; the saved
// scalings of the reverse pass are prefetched one phase ahead.
//
// Reverse sweeps: for u = w/(R + eps) with R = sum over the row of w,
//   wbar = (ubar - sum_row ubar*u) / (R + eps),
// and likewise for the columns. The per-pair plan adjoint lives in LDS
// (indexed by row-major position within the sample) when it fits; the lane
// owning a row (or column) reads its pairs' adjoints, forms the sum and
// rewrites them.
#include <algorithm>

#include "apml_internal.h"
#include "device_common.h"

namespace apml {
namespace {

constexpr int kCover = 2048;   // rows or columns a per-sample workgroup covers
constexpr int kMax = 8;        // pairs per owner kept in registers
constexpr int kTailCap = 2048; // LDS tail entries per order
constexpr int kFwdT = 1024;    // forward: 1024 lanes x 2 owners
constexpr int kBwdT = 512;     // reverse: 512 lanes x 4 owners (more registers per lane)
constexpr int kMaxWaves = 16;

// One order of a sample's pairs: owners are rows (row-major) or columns
// (column-major).
struct LOrder {
    const int32_t *ptr;    // [n_own + 1]: global positions of the owners' segments
    const int32_t *gather; // per pair: index of the other side, within the sample
    const float *val;      // per pair: P0
    const int32_t *perm;   // per pair: row-major position (column-major order) or nullptr
    int n_own;
};

// The pairs beyond kMax of long owners, in LDS.
struct Tail {
    uint32_t *gp; // gathered index | (row-major position within the sample) << 16
    float *p0;
};

// A lane's SL owners: the first kMax pairs of each in registers. Gathered
// indices and positions are packed two per word.
template <int SL, bool POS> struct LCache {
    float p0[SL][kMax];
    uint32_t gi[SL][kMax / 2];
    uint32_t pos[POS ? SL : 1][POS ? kMax / 2 : 1];
    int own[SL];   // owner index within the sample (-1: none)
    int start[SL]; // global position of the owner's first pair
    int len[SL];   // its number of pairs (0: no owner)
    int toff[SL];  // its first tail entry
    int wmax[SL];  // the longest len[s] in the wave (wave-uniform)
};

__device__ __forceinline__ int h16(uint32_t w, int k) { return (int)((w >> (16 * (k & 1))) & 0xFFFFu); }

// A copy of v that the compiler cannot see through.
template <typename V> __device__ __forceinline__ V opaque(V v)
{
    asm volatile("" : "+v"(v));
    return v;
}

// Workgroup-wide exclusive scan of one int per thread (T threads, part holds
// T/64 ints).
template <int T> __device__ int block_scan(int v, int *part)
{
    const int lane = lane_id(), wave = threadIdx.x >> 6;
    int inc = v;
    for (int off = 1; off < 64; off <<= 1) {
        const int n = __shfl_up(inc, off);
        if (lane >= off)
            inc += n;
    }
    if (lane == 63)
        part[wave] = inc;
    lds_barrier();
    int base = 0;
    for (int w = 0; w < wave; ++w)
        base += part[w];
    lds_barrier();
    return base + inc - v;
}

constexpr int kBuckets = 16;

// Loads the lane's owners of one order. Owners are dealt to lanes in order of
// decreasing length (counting sort on min(len, kBuckets - 1)), so the lanes
// of a wave have similar lengths and a wave visits only as many cached entries
// as its longest owner has. The result does not depend on this assignment:
// each owner's sums are formed by one lane in pair order. Long owners' extra
// pairs go to the LDS tail (capacity kTailCap; entries beyond it stay in
// global memory). Padding entries of the cache get P0 = 0, gathered index 0
// and position 0. scratch: kCover + kBuckets ints of LDS.
template <int T, int SL, bool POS>
__device__ void lload(LCache<SL, POS> &c, const LOrder &o, int lo, Tail tl, int *part, int *scratch)
{
    int *order = scratch, *hist = scratch + kCover;
    if (threadIdx.x < kBuckets)
        hist[threadIdx.x] = 0;
    lds_barrier();
    int bk[SL], rk[SL];
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        const int own = threadIdx.x + s * T;
        if (own < o.n_own) {
            const int n = o.ptr[own + 1] - o.ptr[own];
            bk[s] = kBuckets - 1 - min(n, kBuckets - 1);
            rk[s] = atomicAdd(&hist[bk[s]], 1);
        }
    }
    lds_barrier();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int k = 0; k < kBuckets; ++k) {
            const int h = hist[k];
            hist[k] = run;
            run += h;
        }
    }
    lds_barrier();
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        const int own = threadIdx.x + s * T;
        if (own < o.n_own)
            order[hist[bk[s]] + rk[s]] = own;
    }
    lds_barrier();

    int tails = 0;
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        const int k = threadIdx.x + s * T;
        const int own = k < o.n_own ? order[k] : -1;
        int st = 0, n = 0;
        if (own >= 0) {
            st = o.ptr[own];
            n = o.ptr[own + 1] - st;
        }
        c.own[s] = own;
        c.start[s] = st;
        c.len[s] = n;
        int m = n;
        for (int off = 32; off > 0; off >>= 1)
            m = max(m, __shfl_xor(m, off));
        c.wmax[s] = __builtin_amdgcn_readfirstlane(m);
#pragma unroll
        for (int e = 0; e < kMax; e += 2) {
            uint32_t w = 0, wp = 0;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const bool v = e + h < n;
                const int t = st + e + h;
                w |= (uint32_t)(v ? o.gather[t] : 0) << (16 * h);
                c.p0[s][e + h] = v ? o.val[t] : 0.0f;
                if (POS)
                    wp |= ((uint32_t)(v ? o.perm[t] - lo : 0) & 0xFFFFu) << (16 * h);
            }
            c.gi[s][e / 2] = w;
            if (POS)
                c.pos[s][e / 2] = wp;
        }
        tails += max(0, n - kMax);
    }
    int base = block_scan<T>(tails, part);
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        c.toff[s] = base;
        for (int e = kMax; e < c.len[s]; ++e, ++base)
            if (base < kTailCap) {
                const int t = c.start[s] + e;
                tl.gp[base] = (uint32_t)o.gather[t] | (((uint32_t)(POS ? o.perm[t] - lo : t - lo) & 0xFFFFu) << 16);
                tl.p0[base] = o.val[t];
            }
    }
}

// Number of slot s's pairs beyond kMax that sit in the LDS tail; the rest of
// them are read from global memory.
template <int SL, bool POS> __device__ __forceinline__ int tail_in_lds(const LCache<SL, POS> &c, int s)
{
    return max(0, min(c.len[s] - kMax, kTailCap - c.toff[s]));
}

// Visits the pairs of slot s in order: f(gathered, p0, row-major position,
// real). The kMax cached entries are visited unconditionally: padding entries
// (real == false) carry P0 = 0, gathered index 0 and position 0, all valid, so
// they add exact zeros to sums; f must skip stores for them.
template <int SL, bool POS, class F>
__device__ __forceinline__ void leach(const LCache<SL, POS> &c, const LOrder &o, int lo, Tail tl, int s, F f)
{
    // The cached words pass through opaque() at each use: values derived from
    // them (widened P0, unpacked indices, positions) are loop invariants of
    // the sweep loop, and hoisting them would multiply the registers held.
    const int st = opaque(c.start[s] - lo), n = opaque(c.len[s]);
#pragma unroll
    for (int e = 0; e < kMax; ++e) {
        if (e < c.wmax[s]) { // wave-uniform
            const float p0 = opaque(c.p0[s][e]);
            const bool real = e < n;
            const int pos = POS ? h16(opaque(c.pos[s][e / 2]), e) : (real ? st + e : 0);
            f(h16(opaque(c.gi[s][e / 2]), e), p0, pos, real);
        }
    }
    const int nl = tail_in_lds(c, s);
    for (int k = c.toff[s]; k < c.toff[s] + nl; ++k) {
        const uint32_t w = tl.gp[k];
        f((int)(w & 0xFFFFu), tl.p0[k], (int)(w >> 16), true);
    }
    for (int t = c.start[s] + kMax + nl; t < c.start[s] + c.len[s]; ++t)
        f(o.gather[t], o.val[t], POS ? o.perm[t] - lo : t - lo, true);
}

// Sum over the pairs of slot s, in order, of f(gathered, p0, row-major position).
template <int SL, bool POS, class F>
__device__ __forceinline__ double lsum(const LCache<SL, POS> &c, const LOrder &o, int lo, Tail tl, int s, F f)
{
    double acc = 0.0;
    leach(c, o, lo, tl, s, [&](int g, float p0, int pos, bool) { acc += f(g, p0, pos); });
    return acc;
}

// LDS: va [kCover], vb [kCover], part [2 kMaxWaves ints], row tail, column
// tail, then a region that holds the loader's scratch during set-up and
// afterwards (reverse, adjoint in LDS) the plan adjoint.
struct LShared {
    double *va, *vb, *adj;
    int *part;
    Tail tr, tc;
    __device__ explicit LShared(double *lds)
    {
        va = lds;
        vb = va + kCover;
        part = reinterpret_cast<int *>(vb + kCover);
        tr.gp = reinterpret_cast<uint32_t *>(part + 2 * kMaxWaves);
        tr.p0 = reinterpret_cast<float *>(tr.gp + kTailCap);
        tc.gp = reinterpret_cast<uint32_t *>(tr.p0 + kTailCap);
        tc.p0 = reinterpret_cast<float *>(tc.gp + kTailCap);
        adj = reinterpret_cast<double *>(tc.p0 + kTailCap);
        scratch = reinterpret_cast<int *>(adj);
    }
    int *scratch;
};
constexpr size_t kLSharedBytes = 8 * 2 * (size_t)kCover + 8 * kMaxWaves + 4 * 4 * (size_t)kTailCap;
constexpr size_t kLoadScratchBytes = 4 * (size_t)(kCover + kBuckets);

__global__ __launch_bounds__(kFwdT) void k_sinkhorn_fwd(DevPlan d, double eps)
{
    constexpr int T = kFwdT, SL = kCover / kFwdT;
    extern __shared__ double lds[];
    LShared sh(lds);
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const LOrder orow{d.row_ptr + (size_t)b * N, d.csr_col, d.p0r, nullptr, N};
    const LOrder ocol{d.col_ptr + (size_t)b * M, d.csc_row, d.p0c, nullptr, M};
    const int lo = d.row_ptr[(size_t)b * N], hi = d.row_ptr[(size_t)(b + 1) * N];
    LCache<SL, false> cr, cc;
    lload<T>(cr, orow, lo, sh.tr, sh.part, sh.scratch);
    lload<T>(cc, ocol, lo, sh.tc, sh.part, sh.scratch);
    for (int k = tid; k < N; k += T) {
        sh.va[k] = 1.0;
        d.alpha[(size_t)b * N + k] = 1.0;
    }
    for (int k = tid; k < M; k += T) {
        sh.vb[k] = 1.0;
        d.beta[(size_t)b * M + k] = 1.0;
    }
    lds_barrier();

    for (int l = 1; l <= L; ++l) {
        // column scaling (Eq. 3): beta_j /= beta_j sum_i alpha_i P0_ij + eps
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            const int j = cc.own[s];
            if (j >= 0) {
                const double S = lsum(cc, ocol, lo, sh.tc, s, [&](int i, float p0, int) { return (double)p0 * sh.va[i]; });
                const double o = sh.vb[j];
                const double den = o * S + eps;
                const double v = o / den;
                sh.vb[j] = v;
                d.beta[l * BM + (size_t)b * M + j] = v;
                d.sden[(l - 1) * BM + (size_t)b * M + j] = den;
            }
        }
        lds_barrier();
        // row scaling (Eq. 4): alpha_i /= alpha_i sum_j P0_ij beta_j + eps
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            const int i = cr.own[s];
            if (i >= 0) {
                const double R = lsum(cr, orow, lo, sh.tr, s, [&](int j, float p0, int) { return (double)p0 * sh.vb[j]; });
                const double o = sh.va[i];
                const double den = o * R + eps;
                const double v = o / den;
                sh.va[i] = v;
                d.alpha[l * BN + (size_t)b * N + i] = v;
                d.rden[(l - 1) * BN + (size_t)b * N + i] = den;
            }
        }
        lds_barrier();
    }

    // loss = sum_t v_t C_t (Sec. III-D), over the sample's pairs in row-major order
    double acc = 0.0;
    for (int t = lo + tid; t < hi; t += T)
        acc += sh.va[d.csr_row[t] - b * N] * (double)d.p0r[t] * sh.vb[d.csr_col[t]] * d.cost[t];
    acc = wave_sum(acc);
    double *part = reinterpret_cast<double *>(sh.tc.p0); // the tails are no longer read
    if (lane_id() == 0)
        part[tid >> 6] = acc;
    lds_barrier();
    if (tid == 0) {
        double s = 0.0;
        for (int w = 0; w < T / 64; ++w)
            s += part[w];
        d.loss[b] = (float)s;
    }
}

// Reverse sweeps, last iteration first. The plan adjoint starts as
// grad_loss * C (loss = sum v C) and ends as dLoss/dP0 in d.adj. ADJ_LDS keeps
// it in LDS (indexed by row-major position within the sample).
template <bool ADJ_LDS> __global__ __launch_bounds__(kBwdT) void k_sinkhorn_bwd(DevPlan d)
{
    constexpr int T = kBwdT, SL = kCover / kBwdT;
    extern __shared__ double lds[];
    LShared sh(lds);
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const int lo = d.row_ptr[(size_t)b * N], hi = d.row_ptr[(size_t)(b + 1) * N];
    const LOrder orow{d.row_ptr + (size_t)b * N, d.csr_col, d.p0r, nullptr, N};
    const LOrder ocol{d.col_ptr + (size_t)b * M, d.csc_row, d.p0c, d.csc_perm, M};
    LCache<SL, false> cr;
    LCache<SL, true> cc;
    lload<T>(cr, orow, lo, sh.tr, sh.part, sh.scratch);
    lload<T>(cc, ocol, lo, sh.tc, sh.part, sh.scratch);
    double *adj = ADJ_LDS ? sh.adj : d.adj + lo; // indexed by position within the sample
    const double gl = d.grad_loss[b];
    for (int t = lo + tid; t < hi; t += T)
        adj[t - lo] = gl * d.cost[t];
    // own scalings, loaded one phase ahead
    double a_own[SL], b_own[SL];
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        const int i = cr.own[s], j = cc.own[s];
        a_own[s] = i >= 0 ? d.alpha[L * BN + (size_t)b * N + i] : 0.0;
        b_own[s] = j >= 0 ? d.beta[L * BM + (size_t)b * M + j] : 0.0;
    }

    for (int l = L; l >= 1; --l) {
        double a_prev[SL], r_own[SL], s_own[SL];
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            const int i = cr.own[s], j = cc.own[s];
            r_own[s] = i >= 0 ? d.rden[(l - 1) * BN + (size_t)b * N + i] : 1.0;
            a_prev[s] = i >= 0 ? d.alpha[(l - 1) * BN + (size_t)b * N + i] : 0.0;
            s_own[s] = j >= 0 ? d.sden[(l - 1) * BM + (size_t)b * M + j] : 1.0;
            if (j >= 0)
                sh.vb[j] = b_own[s];
        }
        // orders the previous column step's adjoint updates (or the initial
        // adjoint) before this row step, and publishes vb = beta^l
        wg_barrier<ADJ_LDS>();
        // adjoint of the row scaling: d_i = sum_row ubar alpha^l_i P0 beta^l_j;
        // ubar <- (ubar - d_i) / (R_i + eps) on the row's pairs
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            if (cr.own[s] >= 0) {
                const double ai = a_own[s];
                const double dsum =
                    lsum(cr, orow, lo, sh.tr, s, [&](int j, float p0, int p) { return adj[p] * (ai * (double)p0 * sh.vb[j]); });
                const double ri = 1.0 / r_own[s], q = dsum * ri;
                leach(cr, orow, lo, sh.tr, s, [&](int, float, int p, bool real) {
                    if (real)
                        adj[p] = adj[p] * ri - q;
                });
            }
        }
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            const int i = cr.own[s];
            if (i >= 0)
                sh.va[i] = a_prev[s];
        }
        wg_barrier<ADJ_LDS>();
        // adjoint of the column scaling: e_j = sum_col wbar alpha^(l-1)_i P0 beta^l_j
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            if (cc.own[s] >= 0) {
                const double bj = b_own[s];
                const double esum =
                    lsum(cc, ocol, lo, sh.tc, s, [&](int i, float p0, int p) { return adj[p] * (sh.va[i] * (double)p0 * bj); });
                const double ri = 1.0 / s_own[s], q = esum * ri;
                leach(cc, ocol, lo, sh.tc, s, [&](int, float, int p, bool real) {
                    if (real)
                        adj[p] = adj[p] * ri - q;
                });
            }
        }
        // the next iteration's own values; vb is rewritten at the top of the
        // next iteration, after every lane has passed this iteration's second
        // barrier, the last point where it was read
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            const int j = cc.own[s];
            a_own[s] = a_prev[s];
            if (l > 1)
                b_own[s] = j >= 0 ? d.beta[(l - 1) * BM + (size_t)b * M + j] : 0.0;
        }
    }
    if (ADJ_LDS) {
        lds_barrier();
        for (int t = lo + tid; t < hi; t += T)
            d.adj[t] = adj[t - lo];
    }
}

// per-iteration fallback (any N, M): one launch per sweep
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_fill_ones(double *a, int n)
{
    const int k = blockIdx.x * kBlock + threadIdx.x;
    if (k < n)
        a[k] = 1.0;
}

__global__ __launch_bounds__(kBlock) void k_sink_col(DevPlan d, int l, double eps)
{
    const int gc = blockIdx.x * kBlock + threadIdx.x;
    if (gc >= d.B * d.M)
        return;
    const int b = gc / d.M;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * d.M;
    const double *alpha_prev = d.alpha + (size_t)(l - 1) * BN + (size_t)b * d.N;
    double acc = 0.0;
    for (int q = d.col_ptr[gc]; q < d.col_ptr[gc + 1]; ++q)
        acc += (double)d.p0c[q] * alpha_prev[d.csc_row[q]];
    const double bprev = d.beta[(size_t)(l - 1) * BM + gc];
    const double den = bprev * acc + eps;
    d.beta[(size_t)l * BM + gc] = bprev / den;
    d.sden[(size_t)(l - 1) * BM + gc] = den;
}

__global__ __launch_bounds__(kBlock) void k_sink_row(DevPlan d, int l, double eps)
{
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= d.B * d.N)
        return;
    const int b = r / d.N;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * d.M;
    const double *beta_cur = d.beta + (size_t)l * BM + (size_t)b * d.M;
    double acc = 0.0;
    for (int t = d.row_ptr[r]; t < d.row_ptr[r + 1]; ++t)
        acc += (double)d.p0r[t] * beta_cur[d.csr_col[t]];
    const double aprev = d.alpha[(size_t)(l - 1) * BN + r];
    const double den = aprev * acc + eps;
    d.alpha[(size_t)l * BN + r] = aprev / den;
    d.rden[(size_t)(l - 1) * BN + r] = den;
}

__global__ __launch_bounds__(kBlock) void k_loss_rows(DevPlan d, double *loss_rows)
{
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= d.B * d.N)
        return;
    const int b = r / d.N;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * d.M;
    const double *beta = d.beta + (size_t)d.L * BM + (size_t)b * d.M;
    double acc = 0.0;
    for (int t = d.row_ptr[r]; t < d.row_ptr[r + 1]; ++t)
        acc += (double)d.p0r[t] * beta[d.csr_col[t]] * d.cost[t];
    loss_rows[r] = d.alpha[(size_t)d.L * BN + r] * acc;
}

__global__ __launch_bounds__(kBlock) void k_loss_reduce(DevPlan d, const double *loss_rows)
{
    __shared__ double part[kBlock / 64];
    const int b = blockIdx.x;
    double s = 0.0;
    for (int i = threadIdx.x; i < d.N; i += kBlock)
        s += loss_rows[(size_t)b * d.N + i];
    s = wave_sum(s);
    if (lane_id() == 0)
        part[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = 0.0;
        for (int w = 0; w < kBlock / 64; ++w)
            t += part[w];
        d.loss[b] = (float)t;
    }
}

__global__ __launch_bounds__(kBlock) void k_bwd_sink_row(DevPlan d, int l)
{
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= d.B * d.N)
        return;
    const int b = r / d.N;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * d.M;
    const double al = d.alpha[(size_t)l * BN + r];
    const double *bl = d.beta + (size_t)l * BM + (size_t)b * d.M;
    const bool last = l == d.L;
    const double gl = d.grad_loss[b];
    const int t0 = d.row_ptr[r], t1 = d.row_ptr[r + 1];
    double dsum = 0.0;
    for (int t = t0; t < t1; ++t) {
        const double ub = last ? gl * d.cost[t] : d.adj[t];
        dsum += ub * (al * (double)d.p0r[t] * bl[d.csr_col[t]]);
    }
    const double den = d.rden[(size_t)(l - 1) * BN + r];
    for (int t = t0; t < t1; ++t) {
        const double ub = last ? gl * d.cost[t] : d.adj[t];
        d.adj[t] = (ub - dsum) / den;
    }
}

__global__ __launch_bounds__(kBlock) void k_bwd_sink_col(DevPlan d, int l)
{
    const int gc = blockIdx.x * kBlock + threadIdx.x;
    if (gc >= d.B * d.M)
        return;
    const int b = gc / d.M;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * d.M;
    const double *ap = d.alpha + (size_t)(l - 1) * BN + (size_t)b * d.N;
    const double bl = d.beta[(size_t)l * BM + gc];
    const int s0 = d.col_ptr[gc], s1 = d.col_ptr[gc + 1];
    double e = 0.0;
    for (int q = s0; q < s1; ++q)
        e += d.adj[d.csc_perm[q]] * (ap[d.csc_row[q]] * (double)d.p0c[q] * bl);
    const double den = d.sden[(size_t)(l - 1) * BM + gc];
    for (int q = s0; q < s1; ++q) {
        const int t = d.csc_perm[q];
        d.adj[t] = (d.adj[t] - e) / den;
    }
}

} // namespace

bool sinkhorn_per_sample_ok(int N, int M) { return N <= kCover && M <= kCover; }

bool sinkhorn_bwd_per_sample_ok(int N, int M, int64_t max_pairs)
{
    return sinkhorn_per_sample_ok(N, M) && max_pairs <= 65536; // positions are packed in 16 bits
}

hipError_t launch_sinkhorn_fwd(const DevPlan &d, double eps, hipStream_t s)
{
    const size_t bytes = kLSharedBytes + kLoadScratchBytes;
    hipError_t e = hipFuncSetAttribute((const void *)k_sinkhorn_fwd,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_sinkhorn_fwd, dim3(d.B), dim3(kFwdT), bytes, s, d, eps);
    return hipGetLastError();
}

hipError_t launch_sinkhorn_bwd(const DevPlan &d, int64_t max_pairs, hipStream_t s)
{
    const size_t budget = 160 * 1024;
    const size_t adj_bytes = 8 * (size_t)max_pairs;
    const bool adj_lds = kLSharedBytes + std::max(adj_bytes, kLoadScratchBytes) <= budget;
    const size_t bytes = kLSharedBytes + (adj_lds ? std::max(adj_bytes, kLoadScratchBytes) : kLoadScratchBytes);
    const void *k = adj_lds ? (const void *)k_sinkhorn_bwd<true> : (const void *)k_sinkhorn_bwd<false>;
    hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess)
        return e;
    if (adj_lds)
        hipLaunchKernelGGL(k_sinkhorn_bwd<true>, dim3(d.B), dim3(kBwdT), bytes, s, d);
    else
        hipLaunchKernelGGL(k_sinkhorn_bwd<false>, dim3(d.B), dim3(kBwdT), bytes, s, d);
    return hipGetLastError();
}

void launch_sinkhorn_fwd_steps(const DevPlan &d, double eps, hipStream_t s)
{
    const int BN = d.B * d.N, BM = d.B * d.M;
    hipLaunchKernelGGL(k_fill_ones, dim3(blocks_for(BN, kBlock)), dim3(kBlock), 0, s, d.alpha, BN);
    hipLaunchKernelGGL(k_fill_ones, dim3(blocks_for(BM, kBlock)), dim3(kBlock), 0, s, d.beta, BM);
    for (int l = 1; l <= d.L; ++l) {
        hipLaunchKernelGGL(k_sink_col, dim3(blocks_for(BM, kBlock)), dim3(kBlock), 0, s, d, l, eps);
        hipLaunchKernelGGL(k_sink_row, dim3(blocks_for(BN, kBlock)), dim3(kBlock), 0, s, d, l, eps);
    }
    // the backward scratch is free during the forward pass: use it for the row losses
    hipLaunchKernelGGL(k_loss_rows, dim3(blocks_for(BN, kBlock)), dim3(kBlock), 0, s, d, d.dvec);
    hipLaunchKernelGGL(k_loss_reduce, dim3(d.B), dim3(kBlock), 0, s, d, (const double *)d.dvec);
}

void launch_sinkhorn_bwd_steps(const DevPlan &d, hipStream_t s)
{
    const int BN = d.B * d.N, BM = d.B * d.M;
    for (int l = d.L; l >= 1; --l) {
        hipLaunchKernelGGL(k_bwd_sink_row, dim3(blocks_for(BN, kBlock)), dim3(kBlock), 0, s, d, l);
        hipLaunchKernelGGL(k_bwd_sink_col, dim3(blocks_for(BM, kBlock)), dim3(kBlock), 0, s, d, l);
    }
}

} // namespace apml
