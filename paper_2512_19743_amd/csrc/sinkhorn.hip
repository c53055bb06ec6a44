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
// sweeps with the sample's pairs held in registers. Each row's (column's)
// pairs are cut into pieces of kP consecutive pairs; piece k sits in lane
// k mod kT, slot k / kT, for the whole kernel. A sweep is two phases:
//   piece phase  each lane forms the partial sum of each of its pieces
//                (gathering the other side's scalings from LDS) and stores it
//                in LDS;
//   owner phase  the lane owning a row (column) adds its pieces' partials in
//                piece order and applies the scaling.
// Every sum has a fixed order, so the result is bitwise reproducible, and no
// lane walks a long row alone.
//
// Reverse sweeps: for u = w/(R + eps) with R = sum over the row of w,
//   wbar = (ubar - sum_row ubar*u) / (R + eps),
// and likewise for the columns. The per-pair adjoint lives in global memory
// (it stays in L2). An update is applied lazily: the owner phase of a row step
// only publishes 1/(R + eps) and q = (sum_row ubar*u)/(R + eps) per row, and
// the next piece phase, which visits the pairs in column order, applies
// wbar = ubar/(R + eps) - q to each pair it reads and writes the result back.
// So each pair's adjoint is read and written once per sweep.
#include <algorithm>

#include "apml_internal.h"
#include "device_common.h"

namespace apml {
namespace {

constexpr int kT = 1024;            // threads of a per-sample workgroup
constexpr int kSL = 2;              // owners per lane: owner o sits in lane o / kSL
constexpr int kCover = kT * kSL;    // rows or columns a workgroup covers
constexpr int kP = 4;               // pairs per piece
constexpr int kFwdSLP = 6;          // piece slots per lane and order, forward
constexpr int kBwdSLP = 5;          // and reverse

// One order of a sample's pairs: owners are rows (row-major) or columns
// (column-major).
struct POrder {
    const int32_t *ptr;    // [n_own + 1]: global positions of the owners' segments
    const int32_t *gather; // per pair: index of the other side, within the sample
    const float *val;      // per pair: P0
    const int32_t *perm;   // per pair: row-major position (column-major order) or nullptr
    int n_own;
};

enum PosMode { kNoPos, kRunPos, kPairPos };

// A lane's pieces of one order. Per pair: P0, and the gathered index with a
// 'real' bit (bit 15), two per word; padding entries have P0 = 0, index 0.
// kRunPos: the first pair's row-major position within the sample (the pairs of
// a row piece are consecutive); kPairPos: each pair's position, two per word.
template <int SLP, int PM> struct Pieces {
    float p0[SLP][kP];
    uint32_t gi[SLP][kP / 2];
    uint32_t pos[SLP][PM == kPairPos ? kP / 2 : 1];
    int n; // number of pieces of the order in this sample (wave-uniform)
};

// A lane's owners: first piece | piece count << 16.
struct Owners {
    uint32_t pp[kSL];
};

__device__ __forceinline__ int half16(uint32_t w, int e) { return (int)((w >> (16 * (e & 1))) & 0xFFFFu); }
__device__ __forceinline__ int gidx(uint32_t w, int e) { return half16(w, e) & 0x7FFF; }
__device__ __forceinline__ bool greal(uint32_t w, int e) { return (half16(w, e) >> 15) != 0; }

// A copy of v that the compiler cannot see through: keeps values derived from
// the cached words (widened P0, unpacked indices) from being hoisted out of
// the sweep loop, which would multiply the registers held.
template <typename V> __device__ __forceinline__ V opaque(V v)
{
    asm volatile("" : "+v"(v));
    return v;
}

// Workgroup-wide exclusive scan of one int per thread; also returns the total.
// part: kT/64 ints of LDS.
__device__ int block_scan(int v, int *part, int &total)
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
    int base = 0, tot = 0;
    for (int w = 0; w < kT / 64; ++w) {
        const int p = part[w];
        base += w < wave ? p : 0;
        tot += p;
    }
    lds_barrier();
    total = tot;
    return base + inc - v;
}

// Cuts one order into pieces and loads the lane's pieces into registers.
// owner_of: SLP*kT words of LDS scratch (free again on return). Returns false
// when the sample has more pieces than the workgroup holds.
template <int SLP, int PM>
__device__ bool pload(Pieces<SLP, PM> &pc, Owners &ow, const POrder &o, int lo, int *part, uint32_t *owner_of)
{
    const int tid = threadIdx.x;
    constexpr int cap = SLP * kT;
    int np[kSL], local = 0;
#pragma unroll
    for (int s = 0; s < kSL; ++s) {
        const int own = kSL * tid + s;
        const int n = own < o.n_own ? o.ptr[own + 1] - o.ptr[own] : 0;
        np[s] = (n + kP - 1) / kP;
        local += np[s];
    }
    int total;
    int base = block_scan(local, part, total);
#pragma unroll
    for (int s = 0; s < kSL; ++s) {
        ow.pp[s] = (uint32_t)base | ((uint32_t)np[s] << 16);
        for (int q = 0; q < np[s]; ++q)
            if (base + q < cap)
                owner_of[base + q] = (uint32_t)(kSL * tid + s) | ((uint32_t)q << 16);
        base += np[s];
    }
    lds_barrier();
    pc.n = __builtin_amdgcn_readfirstlane(total);
    // all slots' loads are independent: no branches between them
    int t0s[SLP], ns[SLP];
#pragma unroll
    for (int s = 0; s < SLP; ++s) {
        const int k = s * kT + tid;
        const bool v = k < min(total, cap);
        const uint32_t w = owner_of[v ? k : 0];
        const int own = v ? (int)(w & 0xFFFFu) : 0, q = (int)(w >> 16);
        const int a = o.ptr[own], e = o.ptr[own + 1];
        t0s[s] = v ? a + q * kP : 0;
        ns[s] = v ? min(kP, e - (a + q * kP)) : 0;
    }
#pragma unroll
    for (int s = 0; s < SLP; ++s) {
        const int t0 = t0s[s], n = ns[s];
#pragma unroll
        for (int e = 0; e < kP; e += 2) {
            uint32_t g = 0, wp = 0;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const bool v = e + h < n;
                const int t = v ? t0 + e + h : lo; // position lo always exists
                const uint32_t gv = (uint32_t)o.gather[t];
                const float pv = o.val[t];
                g |= (v ? gv | 0x8000u : 0u) << (16 * h);
                pc.p0[s][e + h] = v ? pv : 0.0f;
                if (PM == kPairPos) {
                    const int pp = o.perm[t] - lo;
                    wp |= ((uint32_t)(v ? pp : 0) & 0xFFFFu) << (16 * h);
                }
            }
            pc.gi[s][e / 2] = g;
            if (PM == kPairPos)
                pc.pos[s][e / 2] = wp;
        }
        if (PM == kRunPos)
            pc.pos[s][0] = (uint32_t)(n > 0 ? t0 - lo : 0);
    }
    lds_barrier();
    return total <= cap;
}

// True when slot s of this wave holds at least one piece.
template <int SLP, int PM> __device__ __forceinline__ bool wave_active(const Pieces<SLP, PM> &pc, int s)
{
    return s * kT + (int)(threadIdx.x & ~63u) < pc.n;
}

// Visits the kP entries of piece slot s: f(gathered, p0, position, real).
// Padding entries have real == false, P0 = 0, gathered index 0 and position
// 0: they add exact zeros to sums, and f must not store for them.
template <int SLP, int PM, class F>
__device__ __forceinline__ void pvisit(const Pieces<SLP, PM> &pc, int s, F f)
{
    const int run = PM == kRunPos ? (int)opaque(pc.pos[s][0]) : 0;
#pragma unroll
    for (int e = 0; e < kP; ++e) {
        const uint32_t g = opaque(pc.gi[s][e / 2]);
        const float p0 = opaque(pc.p0[s][e]);
        const int pos = PM == kPairPos ? half16(opaque(pc.pos[s][e / 2]), e) : run + e;
        f(gidx(g, e), p0, pos, greal(g, e));
    }
}

// Sum of the partials of owner slot s, in piece order. The first four are
// loaded together.
__device__ __forceinline__ double owner_sum(const Owners &ow, int s, const double *part)
{
    const int first = (int)(ow.pp[s] & 0xFFFFu), cnt = (int)(ow.pp[s] >> 16);
    double v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
        v[k] = k < cnt ? part[first + k] : 0.0;
    double acc = ((v[0] + v[1]) + v[2]) + v[3];
    for (int k = first + 4; k < first + cnt; ++k)
        acc += part[k];
    return acc;
}

// Most pieces an order of a sample with n_own owners and at most max_pairs
// pairs can have: sum over owners of ceil(len / kP).
inline int64_t max_pieces(int n_own, int64_t max_pairs) { return (max_pairs + (int64_t)(kP - 1) * n_own) / kP; }

constexpr size_t fwd_lds_bytes() { return 8 * (2 * (size_t)kCover + (size_t)kFwdSLP * kT) + 4 * (kT / 64); }
constexpr size_t bwd_lds_bytes() { return 8 * (6 * (size_t)kCover + (size_t)kBwdSLP * kT) + 4 * (kT / 64); }

__global__ __launch_bounds__(kT) void k_sinkhorn_fwd(DevPlan d, double eps)
{
    constexpr int SLP = kFwdSLP;
    extern __shared__ double lds[];
    double *va = lds, *vb = va + kCover, *part = vb + kCover;
    int *scan = reinterpret_cast<int *>(part + SLP * kT);
    uint32_t *owner_of = reinterpret_cast<uint32_t *>(part); // set-up only
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const int lo = d.row_ptr[(size_t)b * N], hi = d.row_ptr[(size_t)(b + 1) * N];
    const POrder orow{d.row_ptr + (size_t)b * N, d.csr_col, d.p0r, nullptr, N};
    const POrder ocol{d.col_ptr + (size_t)b * M, d.csc_row, d.p0c, nullptr, M};
    Pieces<SLP, kNoPos> pr, pc;
    Owners owr, owc;
    bool ok = pload(pr, owr, orow, lo, scan, owner_of);
    ok = pload(pc, owc, ocol, lo, scan, owner_of) && ok;
    if (!ok) { // excluded by the host's capacity check; fail loudly if reached
        if (tid == 0)
            d.loss[b] = __builtin_nanf("");
        return;
    }
    for (int k = tid; k < N; k += kT) {
        va[k] = 1.0;
        d.alpha[(size_t)b * N + k] = 1.0;
    }
    for (int k = tid; k < M; k += kT) {
        vb[k] = 1.0;
        d.beta[(size_t)b * M + k] = 1.0;
    }
    lds_barrier();

    for (int l = 1; l <= L; ++l) {
        // column scaling (Eq. 3): beta_j /= beta_j sum_i alpha_i P0_ij + eps
#pragma unroll
        for (int s = 0; s < SLP; ++s)
            if (wave_active(pc, s)) {
                double acc = 0.0;
                pvisit(pc, s, [&](int i, float p0, int, bool) { acc += (double)p0 * va[i]; });
                part[s * kT + tid] = acc;
            }
        lds_barrier();
#pragma unroll
        for (int s = 0; s < kSL; ++s) {
            const int j = kSL * tid + s;
            if (j < M) {
                const double S = owner_sum(owc, s, part);
                const double o = vb[j];
                const double den = o * S + eps;
                const double v = o / den;
                vb[j] = v;
                d.beta[l * BM + (size_t)b * M + j] = v;
                d.sden[(l - 1) * BM + (size_t)b * M + j] = den;
            }
        }
        lds_barrier();
        // row scaling (Eq. 4): alpha_i /= alpha_i sum_j P0_ij beta_j + eps
#pragma unroll
        for (int s = 0; s < SLP; ++s)
            if (wave_active(pr, s)) {
                double acc = 0.0;
                pvisit(pr, s, [&](int j, float p0, int, bool) { acc += (double)p0 * vb[j]; });
                part[s * kT + tid] = acc;
            }
        lds_barrier();
#pragma unroll
        for (int s = 0; s < kSL; ++s) {
            const int i = kSL * tid + s;
            if (i < N) {
                const double R = owner_sum(owr, s, part);
                const double o = va[i];
                const double den = o * R + eps;
                const double v = o / den;
                va[i] = v;
                d.alpha[l * BN + (size_t)b * N + i] = v;
                d.rden[(l - 1) * BN + (size_t)b * N + i] = den;
            }
        }
        lds_barrier();
    }

    // loss = sum_t v_t C_t (Sec. III-D), over the sample's pairs in row-major order
    double acc = 0.0;
    for (int t = lo + tid; t < hi; t += kT)
        acc += va[d.csr_row[t] - b * N] * (double)d.p0r[t] * vb[d.csr_col[t]] * d.cost[t];
    acc = wave_sum(acc);
    if (lane_id() == 0)
        part[tid >> 6] = acc;
    lds_barrier();
    if (tid == 0) {
        double s = 0.0;
        for (int w = 0; w < kT / 64; ++w)
            s += part[w];
        d.loss[b] = (float)s;
    }
}

// Reverse sweeps, last iteration first. The plan adjoint starts as
// grad_loss * C (loss = sum v C) and ends as dLoss/dP0 in d.adj (row-major).
__global__ __launch_bounds__(kT) void k_sinkhorn_bwd(DevPlan d)
{
    constexpr int SLP = kBwdSLP;
    extern __shared__ double lds[];
    // row side: alpha^(l-1), 1/(R + eps), q; column side: beta^l, 1/(S + eps), q
    double *va = lds, *ri = va + kCover, *qr = ri + kCover;
    double *vb = qr + kCover, *si = vb + kCover, *qc = si + kCover;
    double *part = qc + kCover;
    int *scan = reinterpret_cast<int *>(part + SLP * kT);
    uint32_t *owner_of = reinterpret_cast<uint32_t *>(part); // set-up only
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const int lo = d.row_ptr[(size_t)b * N], hi = d.row_ptr[(size_t)(b + 1) * N];
    const POrder orow{d.row_ptr + (size_t)b * N, d.csr_col, d.p0r, nullptr, N};
    const POrder ocol{d.col_ptr + (size_t)b * M, d.csc_row, d.p0c, d.csc_perm, M};
    Pieces<SLP, kRunPos> pr;
    Pieces<SLP, kPairPos> pc;
    Owners owr, owc;
    bool ok = pload(pr, owr, orow, lo, scan, owner_of);
    ok = pload(pc, owc, ocol, lo, scan, owner_of) && ok;
    double *adj = d.adj + lo; // indexed by row-major position within the sample
    if (!ok) { // excluded by the host's capacity check; fail loudly if reached
        for (int t = lo + tid; t < hi; t += kT)
            adj[t - lo] = __builtin_nan("");
        return;
    }
    const double gl = d.grad_loss[b];
    for (int t = lo + tid; t < hi; t += kT)
        adj[t - lo] = gl * d.cost[t];
    double a_own[kSL], b_own[kSL];
#pragma unroll
    for (int s = 0; s < kSL; ++s) {
        const int i = kSL * tid + s, j = kSL * tid + s;
        a_own[s] = i < N ? d.alpha[L * BN + (size_t)b * N + i] : 0.0;
        b_own[s] = j < M ? d.beta[L * BM + (size_t)b * M + j] : 0.0;
        if (j < M) { // no pending column update before the last iteration
            vb[j] = b_own[s];
            si[j] = 1.0;
            qc[j] = 0.0;
        }
    }
    __syncthreads();

    for (int l = L; l >= 1; --l) {
        // saved values of this iteration, loaded ahead of their use
        double rden[kSL], a_prev[kSL], sden[kSL], b_prev[kSL];
#pragma unroll
        for (int s = 0; s < kSL; ++s) {
            const int k = kSL * tid + s;
            rden[s] = k < N ? d.rden[(l - 1) * BN + (size_t)b * N + k] : 1.0;
            a_prev[s] = k < N ? d.alpha[(l - 1) * BN + (size_t)b * N + k] : 0.0;
            sden[s] = k < M ? d.sden[(l - 1) * BM + (size_t)b * M + k] : 1.0;
            b_prev[s] = (k < M && l > 1) ? d.beta[(l - 1) * BM + (size_t)b * M + k] : 0.0;
        }
        // row pieces: apply the pending column update, then partial sums of
        // ubar * P0 * beta^l over each piece
        // (all adjoint loads of the phase are issued before its first store)
        double m[SLP][kP];
#pragma unroll
        for (int s = 0; s < SLP; ++s)
            if (wave_active(pr, s)) {
                int e = 0;
                pvisit(pr, s, [&](int, float, int p, bool real) { m[s][e++] = real ? adj[p] : 0.0; });
            }
#pragma unroll
        for (int s = 0; s < SLP; ++s)
            if (wave_active(pr, s)) {
                double acc = 0.0;
                int e = 0;
                pvisit(pr, s, [&](int j, float p0, int p, bool real) {
                    const double a = m[s][e++] * si[j] - qc[j];
                    if (real)
                        adj[p] = a;
                    acc += a * ((double)p0 * vb[j]);
                });
                part[s * kT + tid] = acc;
            }
        __syncthreads();
        // row owners (adjoint of Eq. 4): d_i = alpha^l_i * sum; publish
        // 1/(R + eps) and q = d_i/(R + eps), and alpha^(l-1) for the columns
#pragma unroll
        for (int s = 0; s < kSL; ++s) {
            const int i = kSL * tid + s;
            if (i < N) {
                const double dsum = a_own[s] * owner_sum(owr, s, part);
                const double r = 1.0 / rden[s];
                ri[i] = r;
                qr[i] = dsum * r;
                va[i] = a_prev[s];
            }
        }
        lds_barrier();
        // column pieces: apply the row update, then partial sums of
        // wbar * alpha^(l-1) * P0 over each piece
#pragma unroll
        for (int s = 0; s < SLP; ++s)
            if (wave_active(pc, s)) {
                int e = 0;
                pvisit(pc, s, [&](int, float, int p, bool real) { m[s][e++] = real ? adj[p] : 0.0; });
            }
#pragma unroll
        for (int s = 0; s < SLP; ++s)
            if (wave_active(pc, s)) {
                double acc = 0.0;
                int e = 0;
                pvisit(pc, s, [&](int i, float p0, int p, bool real) {
                    const double a = m[s][e++] * ri[i] - qr[i];
                    if (real)
                        adj[p] = a;
                    acc += a * (va[i] * (double)p0);
                });
                part[s * kT + tid] = acc;
            }
        __syncthreads();
        // column owners (adjoint of Eq. 3): e_j = beta^l_j * sum; publish
        // 1/(S + eps), q = e_j/(S + eps), and beta^(l-1) for the next rows
#pragma unroll
        for (int s = 0; s < kSL; ++s) {
            const int j = kSL * tid + s;
            if (j < M) {
                const double esum = b_own[s] * owner_sum(owc, s, part);
                const double r = 1.0 / sden[s];
                si[j] = r;
                qc[j] = esum * r;
                vb[j] = b_prev[s];
            }
            a_own[s] = a_prev[s];
            b_own[s] = b_prev[s];
        }
        lds_barrier();
    }
    // the last column update
    for (int t = lo + tid; t < hi; t += kT) {
        const int j = d.csr_col[t];
        adj[t - lo] = adj[t - lo] * si[j] - qc[j];
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

bool sinkhorn_per_sample_ok(int N, int M, int64_t max_pairs)
{
    return N <= kCover && M <= kCover && max_pieces(std::max(N, M), max_pairs) <= (int64_t)kFwdSLP * kT;
}

bool sinkhorn_bwd_per_sample_ok(int N, int M, int64_t max_pairs)
{
    return N <= kCover && M <= kCover && max_pieces(std::max(N, M), max_pairs) <= (int64_t)kBwdSLP * kT &&
           max_pairs <= 65536; // positions within a sample are packed in 16 bits
}

hipError_t launch_sinkhorn_fwd(const DevPlan &d, double eps, hipStream_t s)
{
    const size_t bytes = fwd_lds_bytes();
    hipError_t e = hipFuncSetAttribute((const void *)k_sinkhorn_fwd,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_sinkhorn_fwd, dim3(d.B), dim3(kT), bytes, s, d, eps);
    return hipGetLastError();
}

hipError_t launch_sinkhorn_bwd(const DevPlan &d, hipStream_t s)
{
    const size_t bytes = bwd_lds_bytes();
    hipError_t e = hipFuncSetAttribute((const void *)k_sinkhorn_bwd,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_sinkhorn_bwd, dim3(d.B), dim3(kT), bytes, s, d);
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
