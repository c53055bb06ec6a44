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
// Per-sample kernels: one workgroup per sample runs all 2L sweeps with
// workgroup barriers only. The sample's pairs are split into equal contiguous
// slices, one per thread (row-major slices for row sweeps, column-major
// slices for column sweeps); a slice that fits the register cache is loaded
// once for the whole kernel. Sums over a row or column are taken in a fixed
// order: each thread sums the runs of equal owner in its slice; a run that
// continues into the following threads is completed by its first thread from
// their partial sums, in thread order. Each round gathers all of its loads
// before any store. The scalings (and, backward, the plan adjoint) live in
// LDS when the sample fits.
//
// Reverse sweeps: for u = w/(R + eps) with R = sum over the row of w,
//   wbar = (ubar - sum_row ubar*u) / (R + eps),
// and likewise for the columns; the adjoint of the plan is a per-pair array.
#include "apml_internal.h"
#include "device_common.h"

namespace apml {
namespace {

// forward: 1024 threads, 12 pairs per thread and order in registers
constexpr int kFwdThreads = 1024, kFwdCache = 12;
// backward (also keeps the row-major position of column-major pairs):
// 512 threads, 24 pairs per thread and order
constexpr int kBwdThreads = 512, kBwdCache = 24;

template <int T> constexpr int header_doubles() { return (T * 8 + 2 * T + 7) / 8; }

// One ordering of a sample's pairs and this thread's slice of it.
struct Slice {
    int a, b;    // this thread's slice, global positions
    bool head;   // its first run continues the previous thread's last run
    bool tail;   // its last run continues into the next thread
    bool cached; // the slice fits the register cache
};

template <int T, int R> __device__ Slice make_slice(const int32_t *owner, int lo, int hi)
{
    Slice s;
    const int64_t n = hi - lo, e = (n + T - 1) / T;
    s.a = (int)min((int64_t)hi, lo + (int64_t)threadIdx.x * e);
    s.b = (int)min((int64_t)hi, s.a + e);
    s.head = s.a < s.b && s.a > lo && owner[s.a - 1] == owner[s.a];
    s.tail = s.a < s.b && s.b < hi && owner[s.b] == owner[s.b - 1];
    s.cached = e <= R;
    return s;
}

__device__ bool through(const Slice &s, const int32_t *owner)
{
    return s.head && s.tail && owner[s.a] == owner[s.b - 1];
}

// Up to R pairs of a slice: owner and gathered index (local, 16 bits each),
// P0, and optionally the row-major position.
template <int R, bool POS> struct Cache {
    uint32_t key[R];
    float val[R];
    int pos[POS ? R : 1];
    int n;
};

// Where the pairs of one ordering live in the plan.
struct Order {
    const int32_t *owner; // global owner index per pair
    int owner_base;       // b*N or b*M
    const int32_t *gather;
    const float *val;
    const int32_t *perm;  // row-major position (column-major order), or nullptr
};

template <int R, bool POS>
__device__ __forceinline__ void load(Cache<R, POS> &c, const Order &o, int at, int end)
{
    c.n = min(R, end - at);
#pragma unroll
    for (int e = 0; e < R; ++e)
        if (e < c.n) {
            c.key[e] = ((uint32_t)(o.owner[at + e] - o.owner_base) << 16) | (uint32_t)o.gather[at + e];
            c.val[e] = o.val[at + e];
            if (POS)
                c.pos[e] = o.perm[at + e];
        }
}

template <int R, bool POS>
__device__ __forceinline__ void refill(Cache<R, POS> &c, const Slice &s, const Order &o, int at)
{
    if (!s.cached)
        load(c, o, at, s.b);
}

template <int R> __device__ __forceinline__ int pair_pos(const Cache<R, true> &c, int e, int at)
{
    return c.pos[e];
}
template <int R> __device__ __forceinline__ int pair_pos(const Cache<R, false> &c, int e, int at)
{
    return at + e;
}

// Sum of contrib over the pairs of every owner that starts in this thread's
// slice, handed to fin(owner, sum). Ends with the workgroup synchronised.
template <int T, int R, bool POS, class Contrib, class Fin>
__device__ void seg_pass(Cache<R, POS> &c, const Slice &s, const Order &o, double *part,
                         const uint8_t *thr, Contrib contrib, Fin fin)
{
    int cur = -1, pend = -1;
    double acc = 0.0, pend_sum = 0.0;
    bool first = true;
    for (int at = s.a; at < s.b; at += R) {
        refill(c, s, o, at);
        double vals[R]; // all loads of the round first: none waits behind a store of fin
#pragma unroll
        for (int e = 0; e < R; ++e)
            if (e < c.n)
                vals[e] = contrib((int)(c.key[e] >> 16), (int)(c.key[e] & 0xFFFFu), c.val[e],
                                  pair_pos(c, e, at));
#pragma unroll
        for (int e = 0; e < R; ++e) {
            if (e < c.n) {
                const int own = (int)(c.key[e] >> 16);
                if (own != cur) {
                    if (cur >= 0) {
                        if (first && s.head)
                            part[threadIdx.x] = acc;
                        else
                            fin(cur, acc);
                        first = false;
                    }
                    cur = own;
                    acc = vals[e];
                } else {
                    acc += vals[e];
                }
            }
        }
    }
    if (cur >= 0) {
        if (first && s.head)
            part[threadIdx.x] = acc;
        else if (s.tail) {
            pend = cur;
            pend_sum = acc;
        } else
            fin(cur, acc);
    }
    __syncthreads();
    if (pend >= 0) {
        double t = pend_sum;
        for (int k = threadIdx.x + 1; k < T; ++k) {
            t += part[k];
            if (!thr[k])
                break;
        }
        fin(pend, t);
    }
    __syncthreads();
}

// Visits every pair of this thread's slice: f(owner, gathered, p0, position).
template <int R, bool POS, class F>
__device__ __forceinline__ void for_each(Cache<R, POS> &c, const Slice &s, const Order &o, F f)
{
    for (int at = s.a; at < s.b; at += R) {
        refill(c, s, o, at);
#pragma unroll
        for (int e = 0; e < R; ++e)
            if (e < c.n)
                f((int)(c.key[e] >> 16), (int)(c.key[e] & 0xFFFFu), c.val[e], pair_pos(c, e, at));
    }
}

// Per pair of the slice: v = compute(owner, gathered, p0, position), then
// store(position, v), all computes of a round before its stores.
template <int R, bool POS, class Compute, class Store>
__device__ __forceinline__ void update_each(Cache<R, POS> &c, const Slice &s, const Order &o,
                                            Compute compute, Store store)
{
    for (int at = s.a; at < s.b; at += R) {
        refill(c, s, o, at);
        double nv[R];
#pragma unroll
        for (int e = 0; e < R; ++e)
            if (e < c.n)
                nv[e] = compute((int)(c.key[e] >> 16), (int)(c.key[e] & 0xFFFFu), c.val[e],
                                pair_pos(c, e, at));
#pragma unroll
        for (int e = 0; e < R; ++e)
            if (e < c.n)
                store(pair_pos(c, e, at), nv[e]);
    }
}

// LDS layout: partial sums [T], through flags [2T] (row-major, column-major),
// then the scalings [N], [M] if they fit, then the plan adjoint if it fits.
template <int T> struct Shared {
    double *part;
    uint8_t *thr;
    double *va, *vb, *adj;
    __device__ Shared(double *lds, int N, int M, int vec_lds)
    {
        part = lds;
        thr = reinterpret_cast<uint8_t *>(lds + T);
        va = lds + header_doubles<T>();
        vb = va + N;
        adj = vec_lds ? vb + M : va;
    }
};

__global__ __launch_bounds__(kFwdThreads) void k_sinkhorn_fwd(DevPlan d, double eps, int vec_lds)
{
    constexpr int T = kFwdThreads, R = kFwdCache;
    extern __shared__ double lds[];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    Shared<T> sh(lds, N, M, vec_lds);
    const Order orow{d.csr_row, b * N, d.csr_col, d.p0r, nullptr};
    const Order ocol{d.csc_col, b * M, d.csc_row, d.p0c, nullptr};
    const Slice sr = make_slice<T, R>(d.csr_row, d.row_ptr[(size_t)b * N], d.row_ptr[(size_t)(b + 1) * N]);
    const Slice sc = make_slice<T, R>(d.csc_col, d.col_ptr[(size_t)b * M], d.col_ptr[(size_t)(b + 1) * M]);
    sh.thr[tid] = through(sr, d.csr_row);
    sh.thr[T + tid] = through(sc, d.csc_col);
    double *alpha0 = d.alpha + (size_t)b * N, *beta0 = d.beta + (size_t)b * M;
    for (int k = tid; k < N; k += T) {
        alpha0[k] = 1.0;
        if (vec_lds)
            sh.va[k] = 1.0;
    }
    for (int k = tid; k < M; k += T) {
        beta0[k] = 1.0;
        if (vec_lds)
            sh.vb[k] = 1.0;
    }
    Cache<R, false> cr, cc;
    if (sr.cached)
        load(cr, orow, sr.a, sr.b);
    if (sc.cached)
        load(cc, ocol, sc.a, sc.b);
    __syncthreads();

    for (int l = 1; l <= L; ++l) {
        // column scaling (Eq. 3)
        const double *a_prev = vec_lds ? sh.va : d.alpha + (l - 1) * BN + (size_t)b * N;
        const double *b_prev = vec_lds ? sh.vb : d.beta + (l - 1) * BM + (size_t)b * M;
        double *beta_l = d.beta + l * BM + (size_t)b * M;
        double *sden_l = d.sden + (l - 1) * BM + (size_t)b * M;
        seg_pass<T>(
            cc, sc, ocol, sh.part, sh.thr + T,
            [&](int j, int i, float p0, int) { return (double)p0 * a_prev[i]; },
            [&](int j, double tot) {
                const double bo = b_prev[j];
                const double den = bo * tot + eps;
                const double bn = bo / den;
                beta_l[j] = bn;
                sden_l[j] = den;
                if (vec_lds)
                    sh.vb[j] = bn;
            });
        // row scaling (Eq. 4)
        const double *b_cur = vec_lds ? sh.vb : beta_l;
        double *alpha_l = d.alpha + l * BN + (size_t)b * N;
        double *rden_l = d.rden + (l - 1) * BN + (size_t)b * N;
        seg_pass<T>(
            cr, sr, orow, sh.part, sh.thr,
            [&](int i, int j, float p0, int) { return (double)p0 * b_cur[j]; },
            [&](int i, double tot) {
                const double ao = a_prev[i];
                const double den = ao * tot + eps;
                const double an = ao / den;
                alpha_l[i] = an;
                rden_l[i] = den;
                if (vec_lds)
                    sh.va[i] = an;
            });
    }

    // loss = sum_t v_t C_t (Sec. III-D)
    const double *aL = vec_lds ? sh.va : d.alpha + L * BN + (size_t)b * N;
    const double *bL = vec_lds ? sh.vb : d.beta + L * BM + (size_t)b * M;
    double acc = 0.0;
    for_each(cr, sr, orow, [&](int i, int j, float p0, int t) { acc += aL[i] * (double)p0 * bL[j] * d.cost[t]; });
    acc = wave_sum(acc);
    __syncthreads();
    if (lane_id() == 0)
        sh.part[tid >> 6] = acc;
    __syncthreads();
    if (tid == 0) {
        double s = 0.0;
        for (int w = 0; w < T / 64; ++w)
            s += sh.part[w];
        d.loss[b] = (float)s;
    }
}

// Reverse sweeps, last iteration first. The plan adjoint starts as
// grad_loss * C (loss = sum v C) and ends as dLoss/dP0 in d.adj. ADJ_LDS keeps
// it in LDS for the whole kernel (indexed by row-major position in the sample).
template <bool ADJ_LDS>
__global__ __launch_bounds__(kBwdThreads) void k_sinkhorn_bwd(DevPlan d, int vec_lds)
{
    constexpr int T = kBwdThreads, R = kBwdCache;
    extern __shared__ double lds[];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    Shared<T> sh(lds, N, M, vec_lds);
    const Order orow{d.csr_row, b * N, d.csr_col, d.p0r, nullptr};
    const Order ocol{d.csc_col, b * M, d.csc_row, d.p0c, d.csc_perm};
    const int lo = d.row_ptr[(size_t)b * N], hi = d.row_ptr[(size_t)(b + 1) * N];
    const Slice sr = make_slice<T, R>(d.csr_row, lo, hi);
    const Slice sc = make_slice<T, R>(d.csc_col, d.col_ptr[(size_t)b * M], d.col_ptr[(size_t)(b + 1) * M]);
    sh.thr[tid] = through(sr, d.csr_row);
    sh.thr[T + tid] = through(sc, d.csc_col);
    Cache<R, false> cr;
    Cache<R, true> cc;
    if (sr.cached)
        load(cr, orow, sr.a, sr.b);
    if (sc.cached)
        load(cc, ocol, sc.a, sc.b);
    // adjoint storage: LDS slot t - lo, or the global array
    double *adj = ADJ_LDS ? sh.adj - lo : d.adj;
    const double gl = d.grad_loss[b];
    for (int t = lo + tid; t < hi; t += T)
        adj[t] = gl * d.cost[t];
    __syncthreads();

    for (int l = L; l >= 1; --l) {
        // adjoint of the row scaling of iteration l
        const double *al = d.alpha + l * BN + (size_t)b * N;
        const double *bl = d.beta + l * BM + (size_t)b * M;
        if (vec_lds) {
            for (int k = tid; k < N; k += T)
                sh.va[k] = al[k];
            for (int k = tid; k < M; k += T)
                sh.vb[k] = bl[k];
            __syncthreads();
        }
        const double *A = vec_lds ? sh.va : al;
        const double *Bv = vec_lds ? sh.vb : bl;
        double *dv = vec_lds ? sh.va : d.dvec + (size_t)b * N;
        seg_pass<T>(
            cr, sr, orow, sh.part, sh.thr,
            [&](int i, int j, float p0, int t) { return adj[t] * (A[i] * (double)p0 * Bv[j]); },
            [&](int i, double tot) { dv[i] = tot; });
        const double *rd = d.rden + (l - 1) * BN + (size_t)b * N;
        update_each(
            cr, sr, orow, [&](int i, int j, float p0, int t) { return (adj[t] - dv[i]) / rd[i]; },
            [&](int t, double v) { adj[t] = v; });
        __syncthreads();
        // adjoint of the column scaling of iteration l
        const double *ap = d.alpha + (l - 1) * BN + (size_t)b * N;
        if (vec_lds) {
            for (int k = tid; k < N; k += T)
                sh.va[k] = ap[k];
            __syncthreads();
        }
        const double *A2 = vec_lds ? sh.va : ap;
        double *ev = vec_lds ? sh.vb : d.evec + (size_t)b * M;
        seg_pass<T>(
            cc, sc, ocol, sh.part, sh.thr + T,
            [&](int j, int i, float p0, int t) { return adj[t] * (A2[i] * (double)p0 * Bv[j]); },
            [&](int j, double tot) { ev[j] = tot; });
        const double *sd = d.sden + (l - 1) * BM + (size_t)b * M;
        update_each(
            cc, sc, ocol, [&](int j, int i, float p0, int t) { return (adj[t] - ev[j]) / sd[j]; },
            [&](int t, double v) { adj[t] = v; });
        __syncthreads();
    }
    if (ADJ_LDS)
        for (int t = lo + tid; t < hi; t += T)
            d.adj[t] = adj[t];
}

// ---------------------------------------------------------------------------
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

bool sinkhorn_per_sample_ok(int N, int M) { return N <= 65536 && M <= 65536; }

namespace {

// LDS of a per-sample kernel with T threads: header, the scalings if N + M
// fit, and (max_pairs >= 0) the plan adjoint of the largest sample if it fits.
template <int T>
size_t lds_bytes(int N, int M, int64_t max_pairs, bool *vectors_in_lds, bool *adj_in_lds)
{
    const size_t header = 8 * (size_t)header_doubles<T>();
    const size_t budget = 160 * 1024;
    const size_t vec = 8 * ((size_t)N + M);
    *vectors_in_lds = header + vec <= budget;
    const size_t used = header + (*vectors_in_lds ? vec : 0);
    *adj_in_lds = max_pairs >= 0 && used + 8 * (size_t)max_pairs <= budget;
    return used + (*adj_in_lds ? 8 * (size_t)max_pairs : 0);
}

} // namespace

hipError_t launch_sinkhorn_fwd(const DevPlan &d, double eps, hipStream_t s)
{
    bool vec_lds = false, unused = false;
    const size_t bytes = lds_bytes<kFwdThreads>(d.N, d.M, -1, &vec_lds, &unused);
    hipError_t e = hipFuncSetAttribute((const void *)k_sinkhorn_fwd,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_sinkhorn_fwd, dim3(d.B), dim3(kFwdThreads), bytes, s, d, eps, vec_lds ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_sinkhorn_bwd(const DevPlan &d, int64_t max_pairs, hipStream_t s)
{
    bool vec_lds = false, adj_lds = false;
    const size_t bytes = lds_bytes<kBwdThreads>(d.N, d.M, max_pairs, &vec_lds, &adj_lds);
    const void *k = adj_lds ? (const void *)k_sinkhorn_bwd<true> : (const void *)k_sinkhorn_bwd<false>;
    hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess)
        return e;
    if (adj_lds)
        hipLaunchKernelGGL(k_sinkhorn_bwd<true>, dim3(d.B), dim3(kBwdThreads), bytes, s, d, vec_lds ? 1 : 0);
    else
        hipLaunchKernelGGL(k_sinkhorn_bwd<false>, dim3(d.B), dim3(kBwdThreads), bytes, s, d, vec_lds ? 1 : 0);
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
