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
// sweeps with workgroup barriers only. A group of kG lanes owns kKC rows (and
// kKC columns); each lane keeps kC pairs of each in registers for the whole
// kernel (zero padded; longer rows stream the rest), so a row sum is kC
// multiply-adds per lane and a fixed butterfly over the group. The sums land
// in LDS and a per-owner pass applies the division. Scalings, sums and (in
// reverse) the per-pair plan adjoint live in LDS. Global memory is only read
// at setup and for the saved scalings, which are prefetched into registers
// one phase ahead; layer stores are not waited for.
//
// Reverse sweeps: for u = w/(R + eps) with R = sum over the row of w,
//   wbar = (ubar - sum_row ubar*u) / (R + eps) = ubar r - (sum_row ubar*u) r,
// r = 1/(R + eps), and likewise for the columns.
#include "apml_internal.h"
#include "device_common.h"

namespace apml {
namespace {

constexpr int kT = 1024;          // threads of a per-sample workgroup
constexpr int kG = 4;             // lanes per row / column
constexpr int kNG = kT / kG;      // groups
constexpr int kKC = 8;            // rows (and columns) per group
constexpr int kC = 2;             // pairs per lane and row kept in registers
constexpr int kCover = kKC * kNG; // rows or columns a workgroup covers
constexpr int kPer = kCover / kT; // owners per thread in the per-owner passes

// One order of a sample's pairs: owners are rows (row-major) or columns
// (column-major).
struct VOrder {
    const int32_t *ptr;    // [n_own + 1]: global positions of the owners' segments
    const int32_t *gather; // per pair: index of the other side, within the sample
    const float *val;      // per pair: P0
    const int32_t *perm;   // per pair: row-major position (column-major order) or nullptr
    int n_own;
};

// A lane's share of one order: kKC owners, kC pairs each, zero padded.
template <bool POS> struct VCache {
    uint32_t gi[kKC];     // the kC gathered indices, 16 bits each
    float p0[kKC][kC];
    uint32_t pos[POS ? kKC : 1]; // the kC row-major positions within the sample, 16 bits each
    uint32_t start[kKC / 2];     // first pair of owner k, within the sample, 16 bits each
    uint32_t longm;       // bit k: owner k has more than kG*kC pairs
    uint32_t validm;      // bit k*kC + c: cached pair c of owner k exists
};

__device__ __forceinline__ int lane_g() { return threadIdx.x % kG; }
__device__ __forceinline__ int group() { return threadIdx.x / kG; }
__device__ __forceinline__ int gidx(uint32_t w, int c) { return (int)((w >> (16 * c)) & 0xFFFFu); }

template <bool POS> __device__ void vload(VCache<POS> &c, const VOrder &o, int lo)
{
    c.longm = 0;
    c.validm = 0;
#pragma unroll
    for (int k = 0; k < kKC; ++k) {
        const int own = group() + k * kNG;
        int s = 0, e = 0;
        if (own < o.n_own) {
            s = o.ptr[own];
            e = o.ptr[own + 1];
        }
        if (k % 2 == 0)
            c.start[k / 2] = 0;
        c.start[k / 2] |= ((uint32_t)(s - lo) & 0xFFFFu) << (16 * (k % 2));
        if (e - s > kG * kC)
            c.longm |= 1u << k;
        uint32_t w = 0, wp = 0;
#pragma unroll
        for (int cc = 0; cc < kC; ++cc) {
            const int t = s + lane_g() + kG * cc;
            const bool v = t < e;
            w |= (uint32_t)(v ? o.gather[t] : 0) << (16 * cc);
            c.p0[k][cc] = v ? o.val[t] : 0.0f;
            if (POS)
                wp |= ((uint32_t)(v ? o.perm[t] - lo : 0) & 0xFFFFu) << (16 * cc);
            if (v)
                c.validm |= 1u << (k * kC + cc);
        }
        c.gi[k] = w;
        if (POS)
            c.pos[k] = wp;
    }
}

// For every owner of this lane's group: total = group sum of
// contrib(gathered, p0, row-major position, owner) over its pairs; the
// first lane stores it to tot[owner]. Cached pairs first (one owner slot at a
// time), then the pairs of long owners beyond the cache.
template <bool POS, class Contrib>
__device__ __forceinline__ void vsum(const VCache<POS> &c, const VOrder &o, int lo, double *tot, Contrib contrib)
{
#pragma unroll
    for (int k = 0; k < kKC; ++k) {
        const int own = group() + k * kNG;
        double acc = 0.0;
#pragma unroll
        for (int cc = 0; cc < kC; ++cc)
            acc += contrib(gidx(c.gi[k], cc), c.p0[k][cc],
                           POS ? gidx(c.pos[k], cc) : gidx(c.start[k / 2], k % 2) + lane_g() + kG * cc, own);
        acc = group_sum<kG>(acc);
        if (lane_g() == 0 && own < o.n_own)
            tot[own] = acc;
        __builtin_amdgcn_sched_barrier(0);
    }
    for (uint32_t m = c.longm; m; m &= m - 1) { // uniform within the group
        const int own = group() + (__builtin_ctz(m)) * kNG;
        const int e = o.ptr[own + 1];
        double acc = 0.0;
        for (int t = o.ptr[own] + lane_g() + kG * kC; t < e; t += kG)
            acc += contrib(o.gather[t], o.val[t], POS ? o.perm[t] - lo : t - lo, own);
        acc = group_sum<kG>(acc);
        if (lane_g() == 0)
            tot[own] += acc;
    }
}

// adj[position] = adj[position] * r[owner] - q[owner] for every pair of the
// lane's owners (positions within the sample, row-major).
template <bool POS>
__device__ __forceinline__ void vupdate(const VCache<POS> &c, const VOrder &o, int lo, double *adj, const double *r,
                                        const double *q)
{
#pragma unroll
    for (int k = 0; k < kKC; ++k) {
        const int own = group() + k * kNG;
        if (own < o.n_own) {
            const double rr = r[own], qq = q[own];
#pragma unroll
            for (int cc = 0; cc < kC; ++cc)
                if (c.validm & (1u << (k * kC + cc))) {
                    const int p = POS ? gidx(c.pos[k], cc) : gidx(c.start[k / 2], k % 2) + lane_g() + kG * cc;
                    adj[p] = adj[p] * rr - qq;
                }
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    for (uint32_t m = c.longm; m; m &= m - 1) {
        const int own = group() + (__builtin_ctz(m)) * kNG;
        const double rr = r[own], qq = q[own];
        const int e = o.ptr[own + 1];
        for (int t = o.ptr[own] + lane_g() + kG * kC; t < e; t += kG) {
            const int p = POS ? o.perm[t] - lo : t - lo;
            adj[p] = adj[p] * rr - qq;
        }
    }
}

// Values of a length-n vector at this thread's owner-pass indices tid, tid+kT.
__device__ __forceinline__ void prefetch(const double *v, int n, double out[kPer])
{
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
        const int k = threadIdx.x + u * kT;
        out[u] = k < n ? v[k] : 0.0;
    }
}

__device__ __forceinline__ void to_lds(double *lds, int n, const double in[kPer])
{
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
        const int k = threadIdx.x + u * kT;
        if (k < n)
            lds[k] = in[u];
    }
}

// LDS: va [kCover], vb [kCover], vc [kCover], part [kT/64], then (reverse,
// ADJ_LDS) the plan adjoint of the largest sample.
struct VShared {
    double *va, *vb, *vc, *part, *adj;
    __device__ explicit VShared(double *lds)
    {
        va = lds;
        vb = va + kCover;
        vc = vb + kCover;
        part = vc + kCover;
        adj = part + kT / 64;
    }
};
constexpr size_t kVSharedBytes = 8 * (3 * (size_t)kCover + kT / 64);

__global__ __launch_bounds__(kT) void k_sinkhorn_fwd(DevPlan d, double eps)
{
    extern __shared__ double lds[];
    VShared sh(lds);
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const VOrder orow{d.row_ptr + (size_t)b * N, d.csr_col, d.p0r, nullptr, N};
    const VOrder ocol{d.col_ptr + (size_t)b * M, d.csc_row, d.p0c, nullptr, M};
    VCache<false> cr, cc;
    vload(cr, orow, 0);
    vload(cc, ocol, 0);
    for (int k = tid; k < N; k += kT) {
        sh.va[k] = 1.0;
        d.alpha[(size_t)b * N + k] = 1.0;
    }
    for (int k = tid; k < M; k += kT) {
        sh.vb[k] = 1.0;
        d.beta[(size_t)b * M + k] = 1.0;
    }
    lds_barrier();

    for (int l = 1; l <= L; ++l) {
        // column scaling (Eq. 3): S_j = sum_i alpha_i P0_ij, beta_j /= beta_j S_j + eps
        vsum(cc, ocol, 0, sh.vc, [&](int i, float p0, int, int) { return (double)p0 * sh.va[i]; });
        lds_barrier();
        for (int j = tid; j < M; j += kT) {
            const double o = sh.vb[j];
            const double den = o * sh.vc[j] + eps;
            const double v = o / den;
            sh.vb[j] = v;
            d.beta[l * BM + (size_t)b * M + j] = v;
            d.sden[(l - 1) * BM + (size_t)b * M + j] = den;
        }
        lds_barrier();
        // row scaling (Eq. 4): R_i = sum_j P0_ij beta_j, alpha_i /= alpha_i R_i + eps
        vsum(cr, orow, 0, sh.vc, [&](int j, float p0, int, int) { return (double)p0 * sh.vb[j]; });
        lds_barrier();
        for (int i = tid; i < N; i += kT) {
            const double o = sh.va[i];
            const double den = o * sh.vc[i] + eps;
            const double v = o / den;
            sh.va[i] = v;
            d.alpha[l * BN + (size_t)b * N + i] = v;
            d.rden[(l - 1) * BN + (size_t)b * N + i] = den;
        }
        lds_barrier();
    }

    // loss = sum_t v_t C_t (Sec. III-D)
    const int lo = d.row_ptr[(size_t)b * N], hi = d.row_ptr[(size_t)(b + 1) * N];
    double acc = 0.0;
    for (int t = lo + tid; t < hi; t += kT)
        acc += sh.va[d.csr_row[t] - b * N] * (double)d.p0r[t] * sh.vb[d.csr_col[t]] * d.cost[t];
    acc = wave_sum(acc);
    if (lane_id() == 0)
        sh.part[tid >> 6] = acc;
    lds_barrier();
    if (tid == 0) {
        double s = 0.0;
        for (int w = 0; w < kT / 64; ++w)
            s += sh.part[w];
        d.loss[b] = (float)s;
    }
}

// Reverse sweeps, last iteration first. The plan adjoint starts as
// grad_loss * C (loss = sum v C) and ends as dLoss/dP0 in d.adj. ADJ_LDS keeps
// it in LDS (indexed by row-major position within the sample).
template <bool ADJ_LDS> __global__ __launch_bounds__(kT) void k_sinkhorn_bwd(DevPlan d)
{
    extern __shared__ double lds[];
    VShared sh(lds);
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const int lo = d.row_ptr[(size_t)b * N], hi = d.row_ptr[(size_t)(b + 1) * N];
    const VOrder orow{d.row_ptr + (size_t)b * N, d.csr_col, d.p0r, nullptr, N};
    const VOrder ocol{d.col_ptr + (size_t)b * M, d.csc_row, d.p0c, d.csc_perm, M};
    VCache<false> cr;
    VCache<true> cc;
    vload(cr, orow, lo);
    vload(cc, ocol, lo);
    double *adj = ADJ_LDS ? sh.adj : d.adj + lo; // indexed by position within the sample
    const double gl = d.grad_loss[b];
    for (int t = lo + tid; t < hi; t += kT)
        adj[t - lo] = gl * d.cost[t];
    // saved scalings, one phase ahead: alpha^L into LDS now, beta^L, rden^L,
    // alpha^(L-1), sden^L in registers
    double nb[kPer], nr[kPer], na[kPer], ns[kPer];
    {
        double a0[kPer];
        prefetch(d.alpha + L * BN + (size_t)b * N, N, a0);
        to_lds(sh.va, N, a0);
    }
    prefetch(d.beta + L * BM + (size_t)b * M, M, nb);
    wg_barrier<ADJ_LDS>();

    for (int l = L; l >= 1; --l) {
        prefetch(d.rden + (l - 1) * BN + (size_t)b * N, N, nr);
        prefetch(d.alpha + (l - 1) * BN + (size_t)b * N, N, na);
        prefetch(d.sden + (l - 1) * BM + (size_t)b * M, M, ns);
        to_lds(sh.vb, M, nb); // beta^l (alpha^l is in va)
        lds_barrier();
        // adjoint of the row scaling: d_i = sum_row ubar alpha_i P0 beta_j
        vsum(cr, orow, lo, sh.vc, [&](int j, float p0, int p, int i) { return adj[p] * (sh.va[i] * (double)p0 * sh.vb[j]); });
        lds_barrier();
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int i = tid + u * kT;
            if (i < N) {
                const double r = 1.0 / nr[u];
                sh.va[i] = r;
                sh.vc[i] *= r;
            }
        }
        lds_barrier();
        vupdate(cr, orow, lo, adj, sh.va, sh.vc);
        wg_barrier<ADJ_LDS>();
        // adjoint of the column scaling: e_j = sum_col wbar alpha^(l-1)_i P0 beta_j
        to_lds(sh.va, N, na);
        if (l > 1)
            prefetch(d.beta + (l - 1) * BM + (size_t)b * M, M, nb);
        lds_barrier();
        vsum(cc, ocol, lo, sh.vc, [&](int i, float p0, int p, int j) { return adj[p] * (sh.va[i] * (double)p0 * sh.vb[j]); });
        lds_barrier();
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int j = tid + u * kT;
            if (j < M) {
                const double r = 1.0 / ns[u];
                sh.vb[j] = r;
                sh.vc[j] *= r;
            }
        }
        lds_barrier();
        vupdate(cc, ocol, lo, adj, sh.vb, sh.vc);
        wg_barrier<ADJ_LDS>();
    }
    if (ADJ_LDS)
        for (int t = lo + tid; t < hi; t += kT)
            d.adj[t] = adj[t - lo];
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

// The packed 16-bit positions of the reverse kernel need samples below 65536 pairs.
static_assert(kCover <= 65536, "gathered indices are packed in 16 bits");

hipError_t launch_sinkhorn_fwd(const DevPlan &d, double eps, hipStream_t s)
{
    const size_t bytes = kVSharedBytes;
    hipError_t e = hipFuncSetAttribute((const void *)k_sinkhorn_fwd,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_sinkhorn_fwd, dim3(d.B), dim3(kT), bytes, s, d, eps);
    return hipGetLastError();
}

hipError_t launch_sinkhorn_bwd(const DevPlan &d, int64_t max_pairs, hipStream_t s)
{
    const size_t budget = 160 * 1024;
    const bool adj_lds = kVSharedBytes + 8 * (size_t)max_pairs <= budget;
    const size_t bytes = adj_lds ? kVSharedBytes + 8 * (size_t)max_pairs : kVSharedBytes;
    const void *k = adj_lds ? (const void *)k_sinkhorn_bwd<true> : (const void *)k_sinkhorn_bwd<false>;
    hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess)
        return e;
    if (adj_lds)
        hipLaunchKernelGGL(k_sinkhorn_bwd<true>, dim3(d.B), dim3(kT), bytes, s, d);
    else
        hipLaunchKernelGGL(k_sinkhorn_bwd<false>, dim3(d.B), dim3(kT), bytes, s, d);
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
