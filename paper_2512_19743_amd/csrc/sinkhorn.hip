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
// Per-sample kernels: one 1024-lane workgroup per sample runs all 2L sweeps
// with the sample's pairs in registers. k_place and k_pack_pairs cut every
// row's (column's) pairs into pieces of kP and lay them out so that an
// owner's pieces are consecutive lanes of one wave (see PackedOrder). In a
// sweep each lane sums its pieces (gathering the other side's values from
// LDS) and the pieces of one owner are added by a butterfly inside their
// aligned lane group, in a fixed order. In the forward kernel the group's
// first lane then applies its owner's scaling at once (one barrier per
// sweep); in the reverse kernel it stores the sum in LDS for an owner phase
// in which lane t owns rows (columns) 2t and 2t+1.
// Sums have a fixed association, so results are bitwise reproducible.
//
// Reverse sweeps: for u = w/(R + eps) with R = sum over the row of w,
//   wbar = (ubar - sum_row ubar*u) / (R + eps),
// and likewise for the columns. The per-pair adjoint lives in LDS (indexed
// by row-major position within the sample). An update is applied lazily: the
// owner phase of a row step only publishes 1/(R + eps) and
// q = (sum_row ubar*u)/(R + eps) per row, and the next piece phase, which
// visits the pairs in column order, applies wbar = ubar/(R + eps) - q to each
// pair it reads and writes the result back. Each pair's adjoint is read and
// written once per sweep.
#include <algorithm>
#include <atomic>
#include <cstdlib>

#include "apml_internal.h"
#include "device_common.h"
#include "pieces.h"

namespace apml {
namespace {

constexpr int kT = kSinkLanes;
constexpr int kP = kSinkPiece;
constexpr int kSL = kSinkOwners / kSinkLanes; // owners per lane in the owner phase
using pieces::adj_slot;
using pieces::adj_slots;
using pieces::pack_col_pair;
using pieces::pack_row_pair;
using pieces::pk_index;
using pieces::place_order;

__global__ __launch_bounds__(kT) void k_place(DevPlan d, int32_t *place)
{
    __shared__ int hist[8], base[8];
    place_order(d, place, blockIdx.x, blockIdx.y == 0, hist, base);
}

// Writes every stored pair into its piece, one thread per pair and order.
__global__ __launch_bounds__(kBlock) void k_pack_pairs(DevPlan d, const int32_t *place)
{
    const int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const bool rows = g < d.nnz;
    const int64_t t = rows ? g : g - d.nnz;
    if (t >= d.nnz)
        return;
    if (rows) {
        const int r = d.csr_row[t], b = r / d.N;
        pack_row_pair(d, place, b, r - b * d.N, (int)(t - d.row_ptr[r]), d.csr_col[t], d.p0r[t]);
    } else {
        const int gc = d.csc_col[t], b = gc / d.M, i = d.csc_row[t];
        const int roff = d.csc_perm[t] - d.row_ptr[(size_t)b * d.N + i];
        pack_col_pair(d, place, b, gc - b * d.M, (int)(t - d.col_ptr[gc]), i, roff, d.p0c[t]);
    }
}

// ---------------------------------------------------------------------------
// per-sample kernels
// ---------------------------------------------------------------------------

// A lane's positions of one order, in registers for the whole kernel.
template <bool POS, int SLP> struct Pieces {
    float p0[SLP][kP];
    uint32_t gi[SLP][kP / 2];
    uint32_t pos[POS ? SLP : 1][POS ? kP / 2 : 1];
    uint32_t info[SLP];
    int n; // positions used (wave-uniform)
};

template <bool POS, int SLP> __device__ void load_pieces(Pieces<POS, SLP> &pc, const PackedOrder &pk, int b)
{
    const int tid = threadIdx.x;
#pragma unroll
    for (int s = 0; s < SLP; ++s) {
        const int p = s * kT + tid;
#pragma unroll
        for (int e = 0; e < kP; ++e)
            pc.p0[s][e] = pk.p0[pk_index(b, p, e, kP, SLP)];
#pragma unroll
        for (int w = 0; w < kP / 2; ++w) {
            pc.gi[s][w] = pk.gi[pk_index(b, p, w, kP / 2, SLP)];
            if (POS)
                pc.pos[s][w] = pk.pos[pk_index(b, p, w, kP / 2, SLP)];
        }
        pc.info[s] = pk.info[pk_index(b, p, 0, 1, SLP)];
    }
    pc.n = __builtin_amdgcn_readfirstlane(pk.n_pos[b]);
}

// Unpacking of the cached words. Each 16-bit half of a gi word holds the byte
// offset of the gathered 8-byte value, each half of a pos word a row-major
// position; an info word is owner (bits 0-10) | log2 group (11-13) | head (14)
// | valid (15) | first row-major position of a row piece (16-31). Bit fields
// are extracted at a base offset the compiler cannot see through (Unpack,
// renewed every sweep), so the unpacked values and the masks derived from
// them are recomputed inside the sweep loop instead of being hoisted out of
// it, which would multiply the registers held; P0 is widened to double by an
// instruction of its own for the same reason. The loads of a slot are issued
// before any of its arithmetic. Padding pairs carry P0 = 0 and offset or
// position 0: they gather and read real data, add nothing and write nothing.
struct Unpack {
    uint32_t lo; // 0

    __device__ __forceinline__ static Unpack make()
    {
        Unpack u{0u};
        asm volatile("" : "+s"(u.lo));
        return u;
    }
    __device__ __forceinline__ uint32_t bits(uint32_t w, uint32_t pos, uint32_t width) const
    {
        return __builtin_amdgcn_ubfe(w, lo + pos, width);
    }
    __device__ __forceinline__ uint32_t half(uint32_t w, int e) const { return bits(w, (e & 1) ? 16u : 0u, 16u); }
    __device__ __forceinline__ int owner(uint32_t info) const { return (int)bits(info, 0, 11); }
    __device__ __forceinline__ int run(uint32_t info) const { return (int)bits(info, 16, 16); }
};

__device__ __forceinline__ double widen(float f)
{
    double d;
    asm volatile("v_cvt_f64_f32 %0, %1" : "=v"(d) : "v"(f));
    return d;
}

template <typename T> __device__ __forceinline__ T lds_at(const void *base, uint32_t byte_off)
{
    return *reinterpret_cast<const T *>(reinterpret_cast<const char *>(base) + byte_off);
}

// Slot s of this wave holds at least one used position.
template <bool POS, int SLP> __device__ __forceinline__ bool wave_active(const Pieces<POS, SLP> &pc, int s)
{
    return s * kT + (int)(threadIdx.x & ~63u) < pc.n;
}

// Sum over the pairs of slot s of P0 times the gathered value (doubles at
// vals + byte offset), in pair order.
// P0 of slot s in double: widened once per kernel when the registers allow
// (WIDE), else widened at each use.
template <bool POS, int SLP, bool WIDE> struct P0Cache {
    double v[WIDE ? SLP : 1][WIDE ? kP : 1];

    __device__ __forceinline__ void init(const Pieces<POS, SLP> &pc)
    {
        if constexpr (WIDE) {
#pragma unroll
            for (int s = 0; s < SLP; ++s)
#pragma unroll
                for (int e = 0; e < kP; ++e)
                    v[s][e] = (double)pc.p0[s][e];
        }
    }
    __device__ __forceinline__ double get(const Pieces<POS, SLP> &pc, int s, int e) const
    {
        if constexpr (WIDE)
            return v[s][e];
        else
            return widen(pc.p0[s][e]);
    }
};

template <bool POS, int SLP, bool WIDE>
__device__ __forceinline__ double slot_dot(const Pieces<POS, SLP> &pc, const P0Cache<POS, SLP, WIDE> &p0, int s,
                                           const double *vals, const Unpack &u)
{
    double g[kP];
#pragma unroll
    for (int e = 0; e < kP; ++e)
        g[e] = lds_at<double>(vals, u.half(pc.gi[s][e / 2], e));
    double acc = p0.get(pc, s, 0) * g[0];
#pragma unroll
    for (int e = 1; e < kP; ++e)
        acc = __builtin_fma(p0.get(pc, s, e), g[e], acc);
    return acc;
}

// v from the partner lane of butterfly step K. Steps 0 and 1 pair lane i with
// i ^ 1 and i ^ 2 (quad_perm); from step 2 on, all lanes of an aligned block
// of 2^K lanes already hold the same value, so any lane of the neighbouring
// block will do: step 2 uses row_half_mirror (i -> 7 - i within 8), step 3
// row_mirror (i -> 15 - i within 16), both DPP moves; steps 4 and 5 use lane
// permutes across rows.
template <int K> __device__ __forceinline__ double partner(double v)
{
    int2 w = __builtin_bit_cast(int2, v);
    if constexpr (K == 0) {
        w.x = __builtin_amdgcn_update_dpp(0, w.x, 0xB1, 0xF, 0xF, true); // quad_perm [1,0,3,2]
        w.y = __builtin_amdgcn_update_dpp(0, w.y, 0xB1, 0xF, 0xF, true);
    } else if constexpr (K == 1) {
        w.x = __builtin_amdgcn_update_dpp(0, w.x, 0x4E, 0xF, 0xF, true); // quad_perm [2,3,0,1]
        w.y = __builtin_amdgcn_update_dpp(0, w.y, 0x4E, 0xF, 0xF, true);
    } else if constexpr (K == 2) {
        w.x = __builtin_amdgcn_update_dpp(0, w.x, 0x141, 0xF, 0xF, true); // row_half_mirror
        w.y = __builtin_amdgcn_update_dpp(0, w.y, 0x141, 0xF, 0xF, true);
    } else if constexpr (K == 3) {
        w.x = __builtin_amdgcn_update_dpp(0, w.x, 0x140, 0xF, 0xF, true); // row_mirror
        w.y = __builtin_amdgcn_update_dpp(0, w.y, 0x140, 0xF, 0xF, true);
    } else {
        w.x = __shfl_xor(w.x, 1 << K);
        w.y = __shfl_xor(w.y, 1 << K);
    }
    return __builtin_bit_cast(double, w);
}

template <int K> __device__ __forceinline__ void bfly_step(double &acc, int lg, int lgmax)
{
    if (K < lgmax) { // wave-uniform
        const double y = partner<K>(acc);
        if (K < lg)
            acc += y;
    }
}

// Adds the partial sums of each aligned group of 2^lg lanes (lg from info);
// every lane of a group ends with the same bits (each step adds two values
// that are the same on both sides, and addition commutes). Groups are sorted
// by size, so the wave's first lane has the largest.
__device__ __forceinline__ double group_reduce(double acc, uint32_t info, const Unpack &u)
{
    const int lg = (int)u.bits(info, 11, 3);
    const int lgmax = __builtin_amdgcn_readfirstlane(lg);
    bfly_step<0>(acc, lg, lgmax);
    bfly_step<1>(acc, lg, lgmax);
    bfly_step<2>(acc, lg, lgmax);
    bfly_step<3>(acc, lg, lgmax);
    bfly_step<4>(acc, lg, lgmax);
    bfly_step<5>(acc, lg, lgmax);
    return acc;
}

// Stores a group's sum at its owner (first lane of the group).
__device__ __forceinline__ void store_sum(double acc, uint32_t info, double *sums, const Unpack &u)
{
    if (u.bits(info, 14, 2) == 3u) // head and valid
        sums[u.owner(info)] = acc;
}

constexpr size_t bwd_fixed_lds_bytes() { return (8 + 8 + 4 + 4) * (size_t)kSinkOwners; }


// a / b for positive normal a, b: the hardware reciprocal refined by two
// Newton steps, then one correction of the quotient (within an ulp of the
// correctly rounded quotient; no scaling for denormals or overflow).
__device__ __forceinline__ double quotient(double a, double b)
{
    double r = __builtin_amdgcn_rcp(b);
    r = __builtin_fma(r, __builtin_fma(-b, r, 1.0), r);
    r = __builtin_fma(r, __builtin_fma(-b, r, 1.0), r);
    const double q = a * r;
    return __builtin_fma(r, __builtin_fma(-b, q, a), q);
}

// Up to this many slots the forward kernel keeps P0 in double in registers.
constexpr int kFwdWideSlots = 4;

// The head lane of an owner's group applies the owner's scaling as soon as
// the group has its sum: v = cur / (cur * sum + eps) (Eq. 3 or Eq. 4), into
// the owner's side array in LDS (which the phase does not gather from) and
// into the saved scalings.
__device__ __forceinline__ void apply_scaling(double acc, uint32_t info, double *own, double eps, double *g_val,
                                              const Unpack &u)
{
    if (u.bits(info, 14, 2) == 3u) { // head and valid
        const int o = u.owner(info);
        const double cur = own[o];
        const double den = cur * acc + eps;
        const double v = quotient(cur, den);
        own[o] = v;
        g_val[o] = v;
    }
}

// loss = sum_t v_t C_t (Sec. III-D) of sample b, with v = alpha P0 beta from
// the final scalings va, vb in LDS, over the sample's pairs [lo, hi) in
// row-major order, four pairs per lane in flight; part: kT / 64 doubles of LDS.
__device__ void sample_loss(const DevPlan &d, int b, int lo, int hi, const double *va, const double *vb, double *part)
{
    const int tid = threadIdx.x, N = d.N;
    double acc = 0.0;
    for (int t0 = lo + tid; t0 < hi; t0 += 4 * kT) {
        int r[4], c[4];
        float p[4];
        double C[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int t = t0 + u * kT < hi ? t0 + u * kT : lo;
            r[u] = d.csr_row[t] - b * N;
            c[u] = d.csr_col[t];
            p[u] = d.p0r[t];
            C[u] = d.cost[t];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (t0 + u * kT < hi)
                acc += va[r[u]] * (double)p[u] * vb[c[u]] * C[u];
    }
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

template <int SLP> __global__ __launch_bounds__(kT) void k_sinkhorn_fwd(DevPlan d, double eps)
{
    // static arrays: their addresses are constants folded into the LDS instructions
    __shared__ double va[kSinkOwners], vb[kSinkOwners], part[kT / 64];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const int lo = d.row_ptr[(size_t)b * N], hi = d.row_ptr[(size_t)(b + 1) * N];
    Pieces<false, SLP> pr, pc;
    load_pieces(pr, d.pk_row, b);
    load_pieces(pc, d.pk_col, b);
    constexpr bool kWide = SLP <= kFwdWideSlots;
    P0Cache<false, SLP, kWide> prw, pcw;
    prw.init(pr);
    pcw.init(pc);
#pragma unroll
    for (int s = 0; s < kSL; ++s) {
        const int k = kSL * tid + s;
        if (k < N) {
            va[k] = 1.0;
            d.alpha[(size_t)b * N + k] = 1.0;
        }
        if (k < M) {
            vb[k] = 1.0;
            d.beta[(size_t)b * M + k] = 1.0;
        }
    }
    lds_barrier();

    for (int l = 1; l <= L; ++l) {
        const Unpack u = Unpack::make();
        // column scaling (Eq. 3): beta_j /= beta_j sum_i alpha_i P0_ij + eps
        double *gb = d.beta + l * BM + (size_t)b * M;
#pragma unroll
        for (int s = 0; s < SLP; ++s)
            if (wave_active(pc, s)) {
                const double acc = slot_dot(pc, pcw, s, va, u);
                apply_scaling(group_reduce(acc, pc.info[s], u), pc.info[s], vb, eps, gb, u);
            }
        lds_barrier();
        // row scaling (Eq. 4): alpha_i /= alpha_i sum_j P0_ij beta_j + eps
        double *ga = d.alpha + l * BN + (size_t)b * N;
#pragma unroll
        for (int s = 0; s < SLP; ++s)
            if (wave_active(pr, s)) {
                const double acc = slot_dot(pr, prw, s, vb, u);
                apply_scaling(group_reduce(acc, pr.info[s], u), pr.info[s], va, eps, ga, u);
            }
        lds_barrier();
    }

    sample_loss(d, b, lo, hi, va, vb, part);
}

// Reverse sweeps, last iteration first. The plan adjoint starts as
// grad_loss * C (loss = sum v C) and ends as dLoss/dP0 in d.adj (row-major).
//
// Scaled representation. With the lazy updates above a row piece would need
// three per-column values (the pending 1/(S + eps), q and beta) and a column
// piece three per-row values. Storing instead z = adjoint * alpha^l_i before
// a row phase and z = adjoint * beta^l_j before a column phase, each phase
// needs two values of the other side, X and Y, and one value of its own
// owner, 1/alpha or 1/beta:
//   row phase l:    z' = (z / alpha^l_i) X_j - Y_j,  X_j = beta^l_j / (S_j + eps),
//                   Y_j = beta^l_j e_j / (S_j + eps)     (pending column update)
//   column phase l: z' = (z / beta^l_j) X_i - Y_i,   X_i = alpha^(l-1)_i / (R_i + eps),
//                   Y_i = alpha^(l-1)_i d_i / (R_i + eps)
// and the row sum d_i / alpha^l_i (column sum e_j / beta^l_j) is just the sum
// of z' P0 over the row's (column's) pairs. X, Y and the reciprocals are kept
// in single precision, the adjoint and all sums in double.
// A row piece that holds pairs: valid and either the row's first piece or one
// with a position (a padding piece of a group has neither; a later real
// piece starts at least kP pairs into its row).
__device__ __forceinline__ bool real_piece(uint32_t info, const Unpack &u)
{
    return (info & 0x8000u) != 0 && (u.bits(info, 14, 1) != 0 || u.run(info) != 0);
}

template <int SLP> __global__ __launch_bounds__(kT) void k_sinkhorn_bwd(DevPlan d)
{
    // fixed arrays static (constant addresses), the adjoints (single
    // precision, row-piece layout) dynamic
    __shared__ double sums[kSinkOwners];
    __shared__ float2 xy[kSinkOwners]; // one side at a time
    __shared__ float inv_a[kSinkOwners], inv_b[kSinkOwners];
    extern __shared__ float adj[];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const int lo = d.row_ptr[(size_t)b * N];
    Pieces<false, SLP> pr;
    Pieces<true, SLP> pc;
    load_pieces(pr, d.pk_row, b);
    load_pieces(pc, d.pk_col, b);
    const double gl = d.grad_loss[b];
    const double *alpha_L = d.alpha + L * BN;
    {
        const Unpack u = Unpack::make();
        // the plan adjoint starts as grad_loss * C, held as adjoint * alpha^L_i
#pragma unroll
        for (int s = 0; s < SLP; ++s) {
            const int i = u.owner(pr.info[s]), run = u.run(pr.info[s]);
            const bool piece = real_piece(pr.info[s], u);
            const int rend = piece ? d.row_ptr[(size_t)b * N + i + 1] - lo : 0;
            const double al = piece ? alpha_L[(size_t)b * N + i] : 0.0;
#pragma unroll
            for (int e = 0; e < kP; ++e) {
                const bool real = piece && run + e < rend;
                const bool mass = pr.p0[s][e] != 0.0f; // only pairs with mass carry an adjoint
                adj[adj_slot(s * kT + tid, e)] = real && mass ? (float)(gl * d.cost[lo + run + e] * al) : 0.0f;
            }
        }
        if (tid == 0)
            adj[adj_slots(SLP)] = 0.0f;
    }
    double a_own[kSL], b_own[kSL];
#pragma unroll
    for (int s = 0; s < kSL; ++s) {
        const int k = kSL * tid + s;
        a_own[s] = k < N ? alpha_L[(size_t)b * N + k] : 1.0;
        b_own[s] = k < M ? d.beta[L * BM + (size_t)b * M + k] : 1.0;
        if (k < N)
            inv_a[k] = (float)(1.0 / a_own[s]);
        if (k < M) { // no pending column update before the last iteration
            xy[k] = make_float2((float)b_own[s], 0.0f);
            inv_b[k] = (float)(1.0 / b_own[s]);
        }
    }
    lds_barrier();

    for (int l = L; l >= 1; --l) {
        // scalings of the previous iteration for the row owners, loaded ahead
        // of their use (those of the column owners after the row owners)
        double a_prev[kSL], b_prev[kSL];
#pragma unroll
        for (int s = 0; s < kSL; ++s) {
            const int k = kSL * tid + s;
            a_prev[s] = k < N ? d.alpha[(l - 1) * BN + (size_t)b * N + k] : 1.0;
        }
        // row phase: the lane's own adjoint words, consecutive across lanes
        const Unpack u = Unpack::make();
#pragma unroll
        for (int s = 0; s < SLP; ++s)
            if (wave_active(pr, s)) {
                const double inv = (double)inv_a[u.owner(pr.info[s])];
                float m[kP];
                float2 w[kP];
#pragma unroll
                for (int e = 0; e < kP; ++e) {
                    m[e] = adj[adj_slot(s * kT + tid, e)];
                    w[e] = lds_at<float2>(xy, u.half(pr.gi[s][e / 2], e));
                }
                double acc = 0.0;
#pragma unroll
                for (int e = 0; e < kP; ++e) {
                    const double z = __builtin_fma((double)m[e] * inv, (double)w[e].x, -(double)w[e].y);
                    const double p0 = widen(pr.p0[s][e]);
                    // pairs without mass (padding) keep 0, so their values stay bounded
                    adj[adj_slot(s * kT + tid, e)] = p0 != 0.0 ? (float)z : 0.0f;
                    acc = e == 0 ? z * p0 : __builtin_fma(z, p0, acc);
                }
                store_sum(group_reduce(acc, pr.info[s], u), pr.info[s], sums, u);
            }
        lds_barrier();
        // row owners (adjoint of Eq. 4): d_i = alpha^l_i * sum; the pending
        // factor alpha^(l-1)_i / (R_i + eps) is alpha^l_i itself
#pragma unroll
        for (int s = 0; s < kSL; ++s) {
            const int i = kSL * tid + s;
            const double al = a_own[s];
            const double dsum = al * sums[min(i, N - 1)];
            if (i < N) {
                xy[i] = make_float2((float)al, (float)(dsum * al));
                inv_a[i] = __builtin_amdgcn_rcpf((float)a_prev[s]);
            }
            a_own[s] = a_prev[s];
        }
#pragma unroll
        for (int s = 0; s < kSL; ++s) {
            const int k = kSL * tid + s;
            b_prev[s] = k < M ? d.beta[(l - 1) * BM + (size_t)b * M + k] : 1.0;
        }
        lds_barrier();
        // column phase: the adjoints of the column's pairs at their row-piece
        // places (padding at the spare entry)
#pragma unroll
        for (int s = 0; s < SLP; ++s)
            if (wave_active(pc, s)) {
                const double inv = (double)inv_b[u.owner(pc.info[s])];
                uint32_t ps[kP];
                float m[kP];
                float2 w[kP];
#pragma unroll
                for (int e = 0; e < kP; ++e) {
                    ps[e] = u.half(pc.pos[s][e / 2], e);
                    m[e] = adj[ps[e]];
                    w[e] = lds_at<float2>(xy, u.half(pc.gi[s][e / 2], e));
                }
                double acc = 0.0;
#pragma unroll
                for (int e = 0; e < kP; ++e) {
                    const double z = __builtin_fma((double)m[e] * inv, (double)w[e].x, -(double)w[e].y);
                    const double p0 = widen(pc.p0[s][e]);
                    if (p0 != 0.0) // padding leaves the spare entry at 0
                        adj[ps[e]] = (float)z;
                    acc = e == 0 ? z * p0 : __builtin_fma(z, p0, acc);
                }
                store_sum(group_reduce(acc, pc.info[s], u), pc.info[s], sums, u);
            }
        lds_barrier();
        // column owners (adjoint of Eq. 3): e_j = beta^l_j * sum; the pending
        // factor beta^(l-1)_j / (S_j + eps) is beta^l_j
#pragma unroll
        for (int s = 0; s < kSL; ++s) {
            const int j = kSL * tid + s;
            const double bl = b_own[s];
            const double esum = bl * sums[min(j, M - 1)];
            if (j < M) {
                xy[j] = make_float2((float)bl, (float)(esum * bl));
                inv_b[j] = __builtin_amdgcn_rcpf((float)b_prev[s]);
            }
            b_own[s] = b_prev[s];
        }
        lds_barrier();
    }
    // the last column update (alpha^0 = beta^0 = 1), written out in row-major order
    {
        const Unpack u = Unpack::make();
#pragma unroll
        for (int s = 0; s < SLP; ++s) {
            const int i = u.owner(pr.info[s]), run = u.run(pr.info[s]);
            const bool piece = real_piece(pr.info[s], u);
            const int rend = piece ? d.row_ptr[(size_t)b * N + i + 1] - lo : 0;
#pragma unroll
            for (int e = 0; e < kP; ++e)
                if (piece && run + e < rend) {
                    const float2 w = lds_at<float2>(xy, u.half(pr.gi[s][e / 2], e));
                    d.adj[lo + run + e] = (double)adj[adj_slot(s * kT + tid, e)] * (double)w.x - (double)w.y;
                }
        }
    }
}

// ---------------------------------------------------------------------------
// streamed per-sample kernels (samples of up to kSinkOwnersW points per side)
// ---------------------------------------------------------------------------
//
// One 1024-lane workgroup per sample runs all 2L sweeps, as above, but the
// pieces (too many for registers) are read from memory in every sweep, a slot
// at a time with the next slot's loads in flight. The forward kernel keeps
// both scaling vectors in LDS in double precision (2 x 64 KB). The reverse
// kernel keeps the plan adjoint twice, in the row pieces' and in the column
// pieces' layout in memory (coalesced, each read and written once per phase
// by the lane that owns the position), and exchanges two single-precision
// factors per owner and phase through LDS. With the plan after row step l
// equal to alpha^l_i P0 beta^l_j, after column step l to alpha^(l-1)_i P0
// beta^l_j, and 1/(R^l_i + eps) = alpha^l_i / alpha^(l-1)_i, 1/(S^l_j + eps)
// = beta^l_j / beta^(l-1)_j (r: row copy, c: column copy):
//   row phase l:    rho = r - Yc_j (the adjoint after the reverse of Eq. 3
//                   of iteration l+1, times beta^l_j); d_i = alpha^l_i
//                   sum_j rho P0; r' = (rho - d_i beta^l_j) alpha^l_i /
//                   alpha^(l-1)_i; publishes Yr_i = d_i alpha^l_i and
//                   alpha^(l-1)_i
//   column phase l: kappa = c - Yr_i; e_j = beta^l_j sum_i kappa P0;
//                   c' = (kappa - e_j alpha^(l-1)_i) beta^l_j / beta^(l-1)_j;
//                   publishes Yc_j = e_j beta^l_j and beta^(l-1)_j
// from r = grad_loss C beta^L_j, c = grad_loss C alpha^L_i and Yc = 0; after
// column phase 1 the adjoint with respect to P0 is r - Yc_j. Copies and
// published factors are single precision, sums and updates double; pairs
// without mass keep 0.
constexpr int kSLW = kSinkOwnersW / kT; // owners per thread in the placement

// Placement of one order of sample b (grid B x 2): as place_order, for up to
// kSinkOwnersW owners and the wide info word.
__global__ __launch_bounds__(kT) void k_place_w(DevPlan d, int32_t *place)
{
    __shared__ int hist[8], base[8];
    const int b = blockIdx.x, tid = threadIdx.x;
    const bool rows = blockIdx.y == 0;
    const int n_own = rows ? d.N : d.M;
    const int32_t *ptr = rows ? d.row_ptr + (size_t)b * d.N : d.col_ptr + (size_t)b * d.M;
    const WideOrder pk = rows ? d.wk_row : d.wk_col;
    const int slots = pk.slots, cap = slots * kT;
    {
        const size_t np0 = (size_t)slots * kP * kT, ngi = np0 / 2;
        for (size_t k = tid; k < np0; k += kT)
            pk.p0[(size_t)b * np0 + k] = 0.0f;
        for (size_t k = tid; k < ngi; k += kT)
            pk.gi[(size_t)b * ngi + k] = 0u;
    }
    if (tid < 8)
        hist[tid] = 0;
    __syncthreads();
    int lg[kSLW], rk[kSLW];
#pragma unroll
    for (int s = 0; s < kSLW; ++s) {
        const int k = kSLW * tid + s;
        lg[s] = -1;
        if (k < n_own) {
            lg[s] = sink_log2_group(sink_pieces(ptr[k + 1] - ptr[k]));
            rk[s] = atomicAdd(&hist[lg[s]], 1);
        }
    }
    __syncthreads();
    if (tid == 0) {
        int run = 0;
        for (int c = 6; c >= 0; --c) { // largest groups first: every group is aligned to its size
            base[c] = run;
            run += hist[c] << c;
        }
        base[7] = run;
        pk.n_pos[b] = run;
    }
    __syncthreads();
    for (int p = base[7] + tid; p < cap; p += kT) // unused positions: invalid
        pk.info[pk_index(b, p, 0, 1, slots)] = 0u;
#pragma unroll
    for (int s = 0; s < kSLW; ++s) {
        if (lg[s] < 0)
            continue;
        const int k = kSLW * tid + s, first = base[lg[s]] + (rk[s] << lg[s]);
        place[((size_t)b * 2 + (rows ? 0 : 1)) * kSinkOwnersW + k] = first;
        for (int q = 0; q < (1 << lg[s]); ++q)
            pk.info[pk_index(b, first + q, 0, 1, slots)] =
                (uint32_t)k | ((uint32_t)lg[s] << 13) | ((q == 0 ? 1u : 0u) << 16) | (1u << 17);
    }
}

// Writes every stored pair into its streamed piece, one thread per pair and order.
__global__ __launch_bounds__(kBlock) void k_pack_w(DevPlan d, const int32_t *place)
{
    const int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const bool rows = g < d.nnz;
    const int64_t t = rows ? g : g - d.nnz;
    if (t >= d.nnz)
        return;
    int b, owner, off, other;
    float p0;
    if (rows) {
        const int r = d.csr_row[t];
        b = r / d.N;
        owner = r - b * d.N;
        off = (int)(t - d.row_ptr[r]);
        other = d.csr_col[t];
        p0 = d.p0r[t];
    } else {
        const int gc = d.csc_col[t];
        b = gc / d.M;
        owner = gc - b * d.M;
        off = (int)(t - d.col_ptr[gc]);
        other = d.csc_row[t];
        p0 = d.p0c[t];
    }
    const WideOrder &pk = rows ? d.wk_row : d.wk_col;
    const int p = place[((size_t)b * 2 + (rows ? 0 : 1)) * kSinkOwnersW + owner] + off / kP, e = off % kP;
    pk.p0[pk_index(b, p, e, kP, pk.slots)] = p0;
    reinterpret_cast<uint16_t *>(pk.gi + pk_index(b, p, e / 2, kP / 2, pk.slots))[e & 1] = (uint16_t)(other << 3);
}

// One streamed position of a lane: P0 of its pairs, the byte offsets of the
// gathered values, the info word.
struct WSlot {
    float p0[kP];
    uint32_t gi[kP / 2];
    uint32_t info;
};

template <class Order> __device__ __forceinline__ WSlot load_wslot(const Order &pk, int b, int s)
{
    WSlot w;
    const int p = s * kT + (int)threadIdx.x;
#pragma unroll
    for (int e = 0; e < kP; ++e)
        w.p0[e] = pk.p0[pk_index(b, p, e, kP, pk.slots)];
#pragma unroll
    for (int q = 0; q < kP / 2; ++q)
        w.gi[q] = pk.gi[pk_index(b, p, q, kP / 2, pk.slots)];
    w.info = pk.info[pk_index(b, p, 0, 1, pk.slots)];
    return w;
}

__device__ __forceinline__ double group_reduce_lg(double acc, int lg)
{
    const int lgmax = __builtin_amdgcn_readfirstlane(lg);
    bfly_step<0>(acc, lg, lgmax);
    bfly_step<1>(acc, lg, lgmax);
    bfly_step<2>(acc, lg, lgmax);
    bfly_step<3>(acc, lg, lgmax);
    bfly_step<4>(acc, lg, lgmax);
    bfly_step<5>(acc, lg, lgmax);
    return acc;
}

// Slots of the calling wave that hold used positions (wave-uniform).
__device__ __forceinline__ int wave_slots(int n_used)
{
    const int wave_base = (int)(threadIdx.x & ~63u);
    return wave_base < n_used ? (n_used - wave_base + kT - 1) / kT : 0;
}

// Slots whose loads are issued together before any of them is used: the
// streamed words come from the last-level cache, whose latency a single slot
// of work does not cover.
constexpr int kWBatch = 4;

// Split kernels: how a sample's workgroups exchange 64-bit words. When they
// all run on one XCD (local), through that XCD's L2: plain stores (the CU's
// cache writes through to the L2) and loads that skip only the CU's cache
// (sc0). Otherwise through memory: relaxed device-scope atomics, which skip
// the per-XCD L2s. Measured with 4 workgroups exchanging 8192 words: 2.3 us
// per meeting and exchange through the L2, 15.7 us through memory.
__device__ __forceinline__ void publish64(void *p, uint64_t v, bool local)
{
    if (local)
        *reinterpret_cast<uint64_t *>(p) = v;
    else
        __hip_atomic_store(reinterpret_cast<uint64_t *>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A 32-bit word published as in publish64.
__device__ __forceinline__ void publish32(float *p, float v, bool local)
{
    if (local)
        *p = v;
    else
        __hip_atomic_store(reinterpret_cast<uint32_t *>(p), __builtin_bit_cast(uint32_t, v), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// One forward sweep: every owner's sum of P0 times the other side's scaling
// (vals) over its pieces, then its own scaling v = cur / (cur sum + eps)
// (Eq. 3 or Eq. 4) into own (LDS) and g_val (the saved scalings). With SPLIT
// the calling workgroup takes the slots s0, s0 + step, ... of each wave, and
// v goes to g_val only (published for the other workgroups of the sample);
// every owner's sum is formed by the same lanes as in the one-workgroup
// kernel, so both give the same bits.
template <bool SPLIT>
__device__ void wide_sweep(const WideOrder &pk, int b, int n_used, const double *vals, double *own, double eps,
                           double *g_val, int s0_first = 0, int step = 1, bool local = false)
{
    const int ns = wave_slots(n_used);
    for (int s0 = s0_first; s0 < ns; s0 += kWBatch * step) {
        WSlot w[kWBatch];
#pragma unroll
        for (int k = 0; k < kWBatch; ++k)
            if (s0 + k * step < ns)
                w[k] = load_wslot(pk, b, s0 + k * step);
#pragma unroll
        for (int k = 0; k < kWBatch; ++k) {
            if (s0 + k * step >= ns)
                break;
            const Unpack u = Unpack::make();
            double g[kP];
#pragma unroll
            for (int e = 0; e < kP; ++e)
                g[e] = lds_at<double>(vals, u.half(w[k].gi[e / 2], e));
            double acc = (double)w[k].p0[0] * g[0];
#pragma unroll
            for (int e = 1; e < kP; ++e)
                acc = __builtin_fma((double)w[k].p0[e], g[e], acc);
            acc = group_reduce_lg(acc, (int)u.bits(w[k].info, 13, 3));
            if (u.bits(w[k].info, 16, 2) == 3u) { // head and valid
                const int o = (int)u.bits(w[k].info, 0, 13);
                const double c = own[o];
                const double v = quotient(c, c * acc + eps);
                if constexpr (SPLIT) {
                    publish64(g_val + o, __builtin_bit_cast(uint64_t, v), local);
                } else {
                    own[o] = v;
                    g_val[o] = v;
                }
            }
        }
    }
}

__global__ __launch_bounds__(kT) void k_sinkhorn_fwd_w(DevPlan d, double eps)
{
    __shared__ double va[kSinkOwnersW], vb[kSinkOwnersW], part[kT / 64];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const int lo = d.row_ptr[(size_t)b * N], hi = d.row_ptr[(size_t)(b + 1) * N];
    const int n_row = __builtin_amdgcn_readfirstlane(d.wk_row.n_pos[b]);
    const int n_col = __builtin_amdgcn_readfirstlane(d.wk_col.n_pos[b]);
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
        // column scaling (Eq. 3), then row scaling (Eq. 4)
        wide_sweep<false>(d.wk_col, b, n_col, va, vb, eps, d.beta + l * BM + (size_t)b * M);
        lds_barrier();
        wide_sweep<false>(d.wk_row, b, n_row, vb, va, eps, d.alpha + l * BN + (size_t)b * N);
        lds_barrier();
    }
    sample_loss(d, b, lo, hi, va, vb, part);
}

// One reverse phase over the pieces of one order: copy (this order's adjoint
// copy) is brought up to date with the other direction's pending step
// (factors fin, gathered), the owners' sums formed, this direction's step
// applied, and the owners' factors published in fout (see above). own:
// the saved scalings of this direction at iteration l (own_l) and l - 1.
// With SPLIT the calling workgroup takes the slots s0, s0 + step, ... and
// the factors go to fout in global memory for the sample's other workgroups.
template <bool SPLIT>
__device__ void wide_reverse(const WideOrder &pk, int b, int n_used, float *copy, const float2 *fin, float2 *fout,
                             const double *own_l, const double *own_prev, int s0_first = 0, int step = 1,
                             bool local = false, float *yout = nullptr)
{
    const int ns = wave_slots(n_used);
    for (int s0 = s0_first; s0 < ns; s0 += kWBatch * step) {
        WSlot w[kWBatch];
        float cv[kWBatch][kP];
        double al[kWBatch], alp[kWBatch];
#pragma unroll
        for (int k = 0; k < kWBatch; ++k)
            if (s0 + k * step < ns) {
                w[k] = load_wslot(pk, b, s0 + k * step);
                const int p = (s0 + k * step) * kT + (int)threadIdx.x;
#pragma unroll
                for (int e = 0; e < kP; ++e)
                    cv[k][e] = copy[pk_index(b, p, e, kP, pk.slots)];
            }
#pragma unroll
        for (int k = 0; k < kWBatch; ++k)
            if (s0 + k * step < ns) {
                const int o = (int)(w[k].info & 0x1FFFu);
                al[k] = own_l[o];
                alp[k] = own_prev[o];
            }
#pragma unroll
        for (int k = 0; k < kWBatch; ++k) {
            if (s0 + k * step >= ns)
                break;
            const Unpack u = Unpack::make();
            const int o = (int)u.bits(w[k].info, 0, 13);
            const int p = (s0 + k * step) * kT + (int)threadIdx.x;
            float2 f[kP];
#pragma unroll
            for (int e = 0; e < kP; ++e)
                f[e] = lds_at<float2>(fin, u.half(w[k].gi[e / 2], e));
            double rho[kP], acc = 0.0;
#pragma unroll
            for (int e = 0; e < kP; ++e) {
                rho[e] = (double)cv[k][e] - (double)f[e].x;
                const double p0 = (double)w[k].p0[e];
                acc = e == 0 ? rho[e] * p0 : __builtin_fma(rho[e], p0, acc);
            }
            const double dsum = al[k] * group_reduce_lg(acc, (int)u.bits(w[k].info, 13, 3));
            const double q = quotient(al[k], alp[k]);
#pragma unroll
            for (int e = 0; e < kP; ++e)
                copy[pk_index(b, p, e, kP, pk.slots)] =
                    w[k].p0[e] != 0.0f ? (float)((rho[e] - dsum * (double)f[e].y) * q) : 0.0f;
            if (u.bits(w[k].info, 16, 2) == 3u) { // head and valid
                if constexpr (SPLIT) // the other word, alp, is a saved scaling the readers load themselves
                    publish32(yout + o, (float)(dsum * al[k]), local);
                else
                    fout[o] = make_float2((float)(dsum * al[k]), (float)alp[k]);
            }
        }
    }
}

// The two adjoint copies of sample b start as grad_loss C beta^L_j (rows) and
// grad_loss C alpha^L_i (columns), over the slots s0, s0 + step, ...
__device__ void wide_reverse_start(const DevPlan &d, int b, int n_row, int n_col, int s0_first, int step)
{
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const float *xb = d.x + (size_t)b * N * 3, *yb = d.y + (size_t)b * M * 3;
    const double *alpha = d.alpha + (size_t)b * N, *beta = d.beta + (size_t)b * M;
    const double gl = d.grad_loss[b];
    for (int order = 0; order < 2; ++order) {
        const WideOrder &pk = order == 0 ? d.wk_row : d.wk_col;
        float *copy = order == 0 ? d.wr : d.wc;
        const int ns = wave_slots(order == 0 ? n_row : n_col);
        for (int s = s0_first; s < ns; s += step) {
            const WSlot w = load_wslot(pk, b, s);
            const Unpack u = Unpack::make();
            const int o = (int)u.bits(w.info, 0, 13), p = s * kT + (int)threadIdx.x;
#pragma unroll
            for (int e = 0; e < kP; ++e) {
                const int k = (int)(u.half(w.gi[e / 2], e) >> 3);
                const int i = order == 0 ? o : k, j = order == 0 ? k : o;
                const double sc = order == 0 ? beta[(size_t)L * BM + j] : alpha[(size_t)L * BN + i];
                copy[pk_index(b, p, e, kP, pk.slots)] =
                    w.p0[e] != 0.0f ? (float)(gl * dist_f64(xb + 3 * i, yb + 3 * j) * sc) : 0.0f;
            }
        }
    }
}

// After column phase 1: the adjoint with respect to P0, r - Yc_j, written in
// row-major order for the row slots s0, s0 + step, ... (fc: the column
// factors of that phase).
__device__ void wide_reverse_end(const DevPlan &d, int b, int n_row, const float2 *fc, int s0_first, int step)
{
    const int N = d.N;
    const int ns = wave_slots(n_row);
    for (int s = s0_first; s < ns; s += step) {
        const WSlot w = load_wslot(d.wk_row, b, s);
        const Unpack u = Unpack::make();
        if (u.bits(w.info, 17, 1) == 0u)
            continue;
        const int i = (int)u.bits(w.info, 0, 13), lg = (int)u.bits(w.info, 13, 3);
        const int p = s * kT + (int)threadIdx.x, q = p & ((1 << lg) - 1); // groups are aligned to their size
        const int r0 = d.row_ptr[(size_t)b * N + i], len = d.row_ptr[(size_t)b * N + i + 1] - r0;
#pragma unroll
        for (int e = 0; e < kP; ++e)
            if (q * kP + e < len) {
                const float2 f = lds_at<float2>(fc, u.half(w.gi[e / 2], e));
                d.adj[r0 + q * kP + e] = (double)d.wr[pk_index(b, p, e, kP, d.wk_row.slots)] - (double)f.x;
            }
    }
}

__global__ __launch_bounds__(kT) void k_sinkhorn_bwd_w(DevPlan d)
{
    __shared__ float2 fr[kSinkOwnersW]; // row factors (Yr_i, alpha^(l-1)_i)
    __shared__ float2 fc[kSinkOwnersW]; // column factors (Yc_j, beta^(l-1)_j)
    const int b = blockIdx.x, tid = threadIdx.x;
    const int M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * M;
    const double *alpha = d.alpha + (size_t)b * d.N, *beta = d.beta + (size_t)b * M; // + l * BN, + l * BM
    const int n_row = __builtin_amdgcn_readfirstlane(d.wk_row.n_pos[b]);
    const int n_col = __builtin_amdgcn_readfirstlane(d.wk_col.n_pos[b]);
    wide_reverse_start(d, b, n_row, n_col, 0, 1);
    for (int k = tid; k < M; k += kT) // no pending column update before row phase L
        fc[k] = make_float2(0.0f, (float)beta[(size_t)L * BM + k]);
    lds_barrier();
    for (int l = L; l >= 1; --l) {
        // reverse of Eq. 4, then of Eq. 3, of iteration l
        wide_reverse<false>(d.wk_row, b, n_row, d.wr, fc, fr, alpha + l * BN, alpha + (l - 1) * BN);
        lds_barrier();
        wide_reverse<false>(d.wk_col, b, n_col, d.wc, fr, fc, beta + l * BM, beta + (l - 1) * BM);
        lds_barrier();
    }
    wide_reverse_end(d, b, n_row, fc, 0, 1);
}

// ---------------------------------------------------------------------------
// split streamed kernels: K workgroups per sample
// ---------------------------------------------------------------------------
//
// The streamed kernels above leave most CUs idle when the batch has fewer
// samples than the chip has CUs. Here K workgroups (one per CU) share a
// sample: workgroup k takes the slots k, k + K, ... of every wave, so each
// owner's sum is formed by the same lanes in the same order as in the
// one-workgroup kernels (same bits). After each half-sweep the owners' new
// values (the saved scalings, or the two reverse factors) are published to
// global memory and the K workgroups meet (split_meet), then every workgroup
// reads the whole vector into its LDS. The grid is launched cooperatively:
// all its workgroups are resident at once, so a meeting always completes.

constexpr unsigned kSplitSpinLimit = 1u << 20; // polls of one meeting (about a second) before giving up

// Sample and member of workgroup g, or false for a workgroup without one.
// Workgroups are dispatched to the eight XCDs in turn, so sample b takes
// XCD b % 8 and the ids x + 8 ((b / 8) K + k) on it: a sample's K workgroups
// share an XCD (their meetings stay within one L2's reach). The grid is
// split_grid(B, K) workgroups; those past the last sample end at once.
__device__ __forceinline__ bool split_member(int g, int B, int K, int &b, int &k)
{
    const int x = g % 8, slot = g / 8;
    b = (slot / K) * 8 + x;
    k = slot % K;
    return b < B;
}

// Meeting t of a sample's K workgroups (t = 1, 2, ...): each waits until its
// own stores have completed (s_waitcnt: plain stores have then reached the
// L2, device-scope atomic stores the level every XCD reads), counts itself
// in at the sample's counter and waits until all K have (target K t). The
// counter is a relaxed device-scope atomic, so no cache is written back or
// invalidated. The wait is bounded: past kSplitSpinLimit polls, or once
// another workgroup has given up, it sets bit 2 of the error word and
// returns false, and the caller ends.
__device__ bool split_meet(uint32_t *cnt, uint32_t target, unsigned int *err, int *stop)
{
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        unsigned spins = 0;
        while (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
            if (++spins > kSplitSpinLimit ||
                ((spins & 63u) == 0 && (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & 4u))) {
                __hip_atomic_fetch_or(err, 4u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                *stop = 1;
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    __syncthreads();
    return *stop == 0;
}

// First meeting of a sample's workgroups: each records its XCD (hardware
// register XCC_ID) next to the counter, and all decide alike, from the same
// K words, whether they share one (local exchange through its L2).
__device__ bool split_begin(uint32_t *sync, int K, int k, unsigned int *err, int *stop, int *local)
{
    if (threadIdx.x == 0) {
        unsigned id;
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(id));
        __hip_atomic_store(sync + 1 + k, id + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (!split_meet(sync, (uint32_t)K, err, stop))
        return false;
    if (threadIdx.x == 0) {
        const unsigned first = __hip_atomic_load(sync + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        int same = 1;
        for (int q = 1; q < K; ++q)
            same &= __hip_atomic_load(sync + 1 + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == first;
        *local = same;
    }
    __syncthreads();
    return true;
}

// Eight published words per lane, word u of lane t at word u * lanes + t
// of the sample's vector, and the wait for them, in one asm statement, so
// that no use of a result can be placed before the wait.
//  local: through the L2 only (sc0: the loads skip the CU's cache); each
//  lane's offsets clamped to the vector's last word, so that no line outside
//  the vector is brought into the CU's cache (see split_gather).
//  else: from memory past the L2s (sc1, as relaxed device-scope atomic
//  loads), one offset register and a scalar base per chunk of lanes; the
//  caller's array extends 8 * lanes words past the vector's start.
#define APML_LDL(I, J) "global_load_dwordx2 %" #I ", %" #J ", %[base] sc0\n\t"
#define APML_LDM(I, B) "global_load_dwordx2 %" #I ", %[off], %" #B " sc1\n\t"
#define APML_OUT8                                                                                             \
    "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]), "=&v"(v[7])

// The sample's n published 64-bit words (n <= 8 * lanes) into LDS.
template <typename T> __device__ __forceinline__ void split_gather(T *lds, const T *g, int n, bool local)
{
    static_assert(kSinkOwnersW / kT == 8, "eight words per lane");
    // the base in scalar registers: each 32-bit half read from the first lane
    // (the builtin takes 32-bit values; a 64-bit argument would be cut)
    const uint64_t a = (uint64_t)(uintptr_t)g;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
    const uint64_t base = ((uint64_t)hi << 32) | lo;
    uint64_t v[8];
    if (local) {
        uint32_t off[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            off[u] = (uint32_t)min(u * kT + (int)threadIdx.x, n - 1) * 8u;
        asm volatile("buffer_inv sc0\n\t" // no line of an earlier read may serve these loads
                     APML_LDL(0, 8) APML_LDL(1, 9) APML_LDL(2, 10) APML_LDL(3, 11) APML_LDL(4, 12) APML_LDL(5, 13)
                     APML_LDL(6, 14) APML_LDL(7, 15) "s_waitcnt vmcnt(0)"
                     : APML_OUT8
                     : "v"(off[0]), "v"(off[1]), "v"(off[2]), "v"(off[3]), "v"(off[4]), "v"(off[5]), "v"(off[6]),
                       "v"(off[7]), [base] "s"(reinterpret_cast<const void *>((uintptr_t)base))
                     : "memory");
    } else {
        const void *bs[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            bs[u] = reinterpret_cast<const void *>((uintptr_t)(base + (uint64_t)u * kT * 8u));
        const uint32_t off = threadIdx.x * 8u;
        asm volatile(APML_LDM(0, 8) APML_LDM(1, 9) APML_LDM(2, 10) APML_LDM(3, 11) APML_LDM(4, 12)
                         APML_LDM(5, 13) APML_LDM(6, 14) APML_LDM(7, 15) "s_waitcnt vmcnt(0)"
                     : APML_OUT8
                     : "s"(bs[0]), "s"(bs[1]), "s"(bs[2]), "s"(bs[3]), "s"(bs[4]), "s"(bs[5]), "s"(bs[6]),
                       "s"(bs[7]), [off] "v"(off)
                     : "memory");
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int o = u * kT + (int)threadIdx.x;
        if (o < n)
            lds[o] = __builtin_bit_cast(T, v[u]);
    }
}
#undef APML_OUT8
#undef APML_LDM
#undef APML_LDL

// The split reverse kernels' factors of one phase into LDS: lds[o] =
// (Y_o, (float) own_prev[o]) for the sample's n owners. Y is the word each
// owner's head published in this phase's region of fresh memory (32-bit
// words: through the L2 only when local, else past the caches); own_prev is
// the owners' saved scaling of the previous iteration, written by an earlier
// kernel. Every lane reads eight whole chunks of lanes: each phase's region
// is padded by kSinkOwnersW words, so a read past the sample's words stays
// within the region of the same phase (other samples' words, which this CU
// never uses), and the saved scalings are read only within the sample's n
// owners. Both loads are issued together after the meeting (one latency).
// The same float bits as the one-workgroup kernel's published pair.
#define APML_LDY(I, B, BITS) "global_load_dword %" #I ", %[off], %" #B " " BITS "\n\t"
#define APML_LOADY(BITS)                                                                                      \
    asm volatile(APML_LDY(0, 8, BITS) APML_LDY(1, 9, BITS) APML_LDY(2, 10, BITS) APML_LDY(3, 11, BITS)       \
                 APML_LDY(4, 12, BITS) APML_LDY(5, 13, BITS) APML_LDY(6, 14, BITS) APML_LDY(7, 15, BITS)     \
                 "s_waitcnt vmcnt(0)"                                                                         \
                 : "=&v"(y[0]), "=&v"(y[1]), "=&v"(y[2]), "=&v"(y[3]), "=&v"(y[4]), "=&v"(y[5]), "=&v"(y[6]), \
                   "=&v"(y[7])                                                                                \
                 : "s"(bs[0]), "s"(bs[1]), "s"(bs[2]), "s"(bs[3]), "s"(bs[4]), "s"(bs[5]), "s"(bs[6]),          \
                   "s"(bs[7]), [off] "v"(off)                                                                 \
                 : "memory")

// The saved scalings of the previous iteration that a gather pairs with the
// exchanged words. The forward kernel wrote them, so they are loaded before
// the meeting, in its shadow.
__device__ __forceinline__ void load_prev(float (&sp)[8], const double *own_prev, int n)
{
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int o = u * kT + (int)threadIdx.x;
        sp[u] = o < n ? (float)own_prev[o] : 0.0f;
    }
}

__device__ __forceinline__ void split_gather_factors(float2 *lds, const float *yv, const float (&sp)[8], int n,
                                                     bool local)
{
    static_assert(kSinkOwnersW / kT == 8, "eight words per lane");
    // the base in scalar registers: each 32-bit half read from the first lane
    const uint64_t a = (uint64_t)(uintptr_t)yv;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
    const uint64_t base = ((uint64_t)hi << 32) | lo;
    const void *bs[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
        bs[u] = reinterpret_cast<const void *>((uintptr_t)(base + (uint64_t)u * kT * 4u));
    const uint32_t off = threadIdx.x * 4u;
    uint32_t y[8];
    if (local) {
        asm volatile("buffer_inv sc0" ::: "memory"); // no line of an earlier read may serve these loads
        APML_LOADY("sc0");
    } else {
        APML_LOADY("sc1");
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int o = u * kT + (int)threadIdx.x;
        if (o < n)
            lds[o] = make_float2(__builtin_bit_cast(float, y[u]), sp[u]);
    }
}
#undef APML_LOADY
#undef APML_LDY


__global__ __launch_bounds__(kT) void k_sinkhorn_fwd_ws(DevPlan d, double eps, int K)
{
    __shared__ double va[kSinkOwnersW], vb[kSinkOwnersW], part[kT / 64];
    __shared__ int stop, local;
    int b, k;
    if (!split_member(blockIdx.x, d.B, K, b, k))
        return;
    const int tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    uint32_t *cnt = d.split_sync + ((size_t)b * 2 + 0) * kSplitSyncStride;
    const int n_row = __builtin_amdgcn_readfirstlane(d.wk_row.n_pos[b]);
    const int n_col = __builtin_amdgcn_readfirstlane(d.wk_col.n_pos[b]);
    for (int o = tid; o < N; o += kT) {
        va[o] = 1.0;
        if (k == 0)
            d.alpha[(size_t)b * N + o] = 1.0;
    }
    for (int o = tid; o < M; o += kT) {
        vb[o] = 1.0;
        if (k == 0)
            d.beta[(size_t)b * M + o] = 1.0;
    }
    if (tid == 0)
        stop = 0;
    lds_barrier();
    if (!split_begin(cnt, K, k, &d.ctr->error, &stop, &local))
        return;
    const bool loc = local != 0;
    uint32_t t = 1;
    for (int l = 1; l <= L; ++l) {
        // column scaling (Eq. 3) of this workgroup's owners, then all of them
        double *gb = d.beta + l * BM + (size_t)b * M;
        wide_sweep<true>(d.wk_col, b, n_col, va, vb, eps, gb, k, K, loc);
        if (!split_meet(cnt, (uint32_t)K * ++t, &d.ctr->error, &stop))
            return;
        split_gather(vb, gb, M, loc);
        lds_barrier();
        // row scaling (Eq. 4)
        double *ga = d.alpha + l * BN + (size_t)b * N;
        wide_sweep<true>(d.wk_row, b, n_row, vb, va, eps, ga, k, K, loc);
        if (!split_meet(cnt, (uint32_t)K * ++t, &d.ctr->error, &stop))
            return;
        split_gather(va, ga, N, loc);
        lds_barrier();
    }
    if (k == 0) // as the one-workgroup kernel, for the same bits
        sample_loss(d, b, d.row_ptr[(size_t)b * N], d.row_ptr[(size_t)(b + 1) * N], va, vb, part);
}

// The reverse sweeps split over K workgroups. After each phase the owners'
// heads publish one word each, Y (Yr_i = d_i alpha^l_i, Yc_j = e_j beta^l_j),
// into a region of fresh memory for that phase (d.yr, d.yc: a word is never
// written twice within the kernel, so the exchange may go through the L2, as
// in the forward kernels); the pair's other factor is the owner's saved
// scaling of the previous iteration, which every reader loads itself.
__global__ __launch_bounds__(kT) void k_sinkhorn_bwd_ws(DevPlan d, int K)
{
    __shared__ float2 fr[kSinkOwnersW]; // row factors (Yr_i, alpha^(l-1)_i)
    __shared__ float2 fc[kSinkOwnersW]; // column factors (Yc_j, beta^(l-1)_j)
    __shared__ int stop, local;
    int b, k;
    if (!split_member(blockIdx.x, d.B, K, b, k))
        return;
    const int tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const double *alpha = d.alpha + (size_t)b * N, *beta = d.beta + (size_t)b * M; // + l * BN, + l * BM
    uint32_t *cnt = d.split_sync + ((size_t)b * 2 + 1) * kSplitSyncStride;
    const int n_row = __builtin_amdgcn_readfirstlane(d.wk_row.n_pos[b]);
    const int n_col = __builtin_amdgcn_readfirstlane(d.wk_col.n_pos[b]);
    wide_reverse_start(d, b, n_row, n_col, k, K);
    for (int o = tid; o < M; o += kT) // no pending column update before row phase L
        fc[o] = make_float2(0.0f, (float)beta[(size_t)L * BM + o]);
    if (tid == 0)
        stop = 0;
    lds_barrier();
    if (!split_begin(cnt, K, k, &d.ctr->error, &stop, &local))
        return;
    const bool loc = local != 0;
    uint32_t t = 1;
    for (int l = L; l >= 1; --l) {
        float *yr = d.yr + (size_t)(L - l) * (BN + kSinkOwnersW) + (size_t)b * N;
        wide_reverse<true>(d.wk_row, b, n_row, d.wr, fc, nullptr, alpha + l * BN, alpha + (l - 1) * BN, k, K, loc,
                           yr);
        float sp[8];
        load_prev(sp, alpha + (l - 1) * BN, N);
        if (!split_meet(cnt, (uint32_t)K * ++t, &d.ctr->error, &stop))
            return;
        split_gather_factors(fr, yr, sp, N, loc);
        lds_barrier();
        float *yc = d.yc + (size_t)(L - l) * (BM + kSinkOwnersW) + (size_t)b * M;
        wide_reverse<true>(d.wk_col, b, n_col, d.wc, fr, nullptr, beta + l * BM, beta + (l - 1) * BM, k, K, loc,
                           yc);
        load_prev(sp, beta + (l - 1) * BM, M);
        if (!split_meet(cnt, (uint32_t)K * ++t, &d.ctr->error, &stop))
            return;
        split_gather_factors(fc, yc, sp, M, loc);
        lds_barrier();
    }
    wide_reverse_end(d, b, n_row, fc, k, K);
}

// Register-resident split kernels: when a workgroup's share is at most SW
// slots per lane and order, its pieces (and in the reverse kernel both
// adjoint copies of its positions) are loaded once and kept in registers for
// every sweep, so a half-sweep reads nothing from memory but the owners'
// saved scalings and the exchanged vector. Same lanes, same arithmetic in the
// same order as the streamed kernels: the same bits. A reverse share of up to
// kSplitAdjBwd slots keeps only the adjoint copies (the state the sweeps
// write) in registers and loads its pieces again in every phase: 28 bytes
// read per slot and phase instead of 60 read and written.
constexpr int kSplitRegFwd = 3; // slots per lane and order held by the forward kernel
constexpr int kSplitRegBwd = 2; // and by the reverse kernel
// adjoint copies held by the reverse kernel, pieces loaded per phase (at 4
// slots it spills: 72 x 8000 x 8000, 0.413 ms against 0.399 ms streamed)
constexpr int kSplitAdjBwd = 3;

// Slots of the calling wave that workgroup k of K takes (wave-uniform).
__device__ __forceinline__ int split_slots(int n_used, int k, int K)
{
    const int ns = wave_slots(n_used);
    return ns > k ? (ns - k + K - 1) / K : 0;
}

template <int SW, class Order>
__device__ __forceinline__ void load_my_slots(WSlot (&w)[SW], const Order &pk, int b, int n, int k, int K)
{
#pragma unroll
    for (int q = 0; q < SW; ++q)
        if (q < n)
            w[q] = load_wslot(pk, b, k + q * K);
}

// The same loads, for a kernel that repeats them in every phase. They are
// raw buffer loads: one descriptor per array and sample (scalar registers),
// the slot and word as a scalar offset, and one lane offset shared by every
// load. Plain pointers let the compiler hoist all the per-word addresses out
// of the sweeps' loop and keep them in vector registers, which spilled. The
// descriptor's size also bounds every load to the sample's own positions.
struct SlotRsrc {
    __amdgpu_buffer_rsrc_t p0, gi, info;
};

constexpr int kBufFlags = 0x00020000; // word 3 of a raw 32-bit buffer descriptor (gfx9 family)

template <class Order> __device__ __forceinline__ SlotRsrc slot_rsrc(const Order &pk, int b)
{
    const size_t bs = (size_t)b * pk.slots;
    SlotRsrc r;
    r.p0 = __builtin_amdgcn_make_buffer_rsrc(pk.p0 + bs * kP * kT, (short)0, pk.slots * kP * kT * 4, kBufFlags);
    r.gi = __builtin_amdgcn_make_buffer_rsrc(pk.gi + bs * (kP / 2) * kT, (short)0, pk.slots * (kP / 2) * kT * 4,
                                             kBufFlags);
    r.info = __builtin_amdgcn_make_buffer_rsrc(pk.info + bs * kT, (short)0, pk.slots * kT * 4, kBufFlags);
    return r;
}

template <int SW>
__device__ __forceinline__ void stream_my_slots(WSlot (&w)[SW], const SlotRsrc &r, int n, int k, int K)
{
    const int lane = (int)threadIdx.x * 4;
#pragma unroll
    for (int q = 0; q < SW; ++q)
        if (q < n) {
            const int s = k + q * K;
#pragma unroll
            for (int e = 0; e < kP; ++e)
                w[q].p0[e] = __builtin_bit_cast(
                    float, __builtin_amdgcn_raw_buffer_load_b32(r.p0, lane, (s * kP + e) * kT * 4, 0));
#pragma unroll
            for (int e = 0; e < kP / 2; ++e)
                w[q].gi[e] = __builtin_amdgcn_raw_buffer_load_b32(r.gi, lane, (s * (kP / 2) + e) * kT * 4, 0);
            w[q].info = __builtin_amdgcn_raw_buffer_load_b32(r.info, lane, s * kT * 4, 0);
        } else {
            w[q] = WSlot{}; // not read; keeps the compiler from holding earlier contents
        }
}

// One forward half-sweep over the slots held in registers (as wide_sweep).
template <int SW>
__device__ __forceinline__ void reg_sweep(const WSlot (&w)[SW], int n, const double *vals, const double *own, double eps,
                                          double *g_val, bool local)
{
#pragma unroll
    for (int q = 0; q < SW; ++q) {
        if (q >= n)
            break;
        const Unpack u = Unpack::make();
        double g[kP];
#pragma unroll
        for (int e = 0; e < kP; ++e)
            g[e] = lds_at<double>(vals, u.half(w[q].gi[e / 2], e));
        double acc = (double)w[q].p0[0] * g[0];
#pragma unroll
        for (int e = 1; e < kP; ++e)
            acc = __builtin_fma((double)w[q].p0[e], g[e], acc);
        acc = group_reduce_lg(acc, (int)u.bits(w[q].info, 13, 3));
        if (u.bits(w[q].info, 16, 2) == 3u) { // head and valid
            const int o = (int)u.bits(w[q].info, 0, 13);
            const double c = own[o];
            publish64(g_val + o, __builtin_bit_cast(uint64_t, quotient(c, c * acc + eps)), local);
        }
    }
}

template <int SW> __global__ __launch_bounds__(kT) void k_sinkhorn_fwd_wr(DevPlan d, double eps, int K)
{
    __shared__ double va[kSinkOwnersW], vb[kSinkOwnersW], part[kT / 64];
    __shared__ int stop, local;
    int b, k;
    if (!split_member(blockIdx.x, d.B, K, b, k))
        return;
    const int tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    uint32_t *cnt = d.split_sync + ((size_t)b * 2 + 0) * kSplitSyncStride;
    const int mr = split_slots(__builtin_amdgcn_readfirstlane(d.wk_row.n_pos[b]), k, K);
    const int mc = split_slots(__builtin_amdgcn_readfirstlane(d.wk_col.n_pos[b]), k, K);
    WSlot pr[SW], pc[SW];
    load_my_slots(pr, d.wk_row, b, mr, k, K);
    load_my_slots(pc, d.wk_col, b, mc, k, K);
    for (int o = tid; o < N; o += kT) {
        va[o] = 1.0;
        if (k == 0)
            d.alpha[(size_t)b * N + o] = 1.0;
    }
    for (int o = tid; o < M; o += kT) {
        vb[o] = 1.0;
        if (k == 0)
            d.beta[(size_t)b * M + o] = 1.0;
    }
    if (tid == 0)
        stop = 0;
    lds_barrier();
    if (!split_begin(cnt, K, k, &d.ctr->error, &stop, &local))
        return;
    const bool loc = local != 0;
    uint32_t t = 1;
    for (int l = 1; l <= L; ++l) {
        double *gb = d.beta + l * BM + (size_t)b * M;
        reg_sweep(pc, mc, va, vb, eps, gb, loc); // Eq. 3
        if (!split_meet(cnt, (uint32_t)K * ++t, &d.ctr->error, &stop))
            return;
        split_gather(vb, gb, M, loc);
        lds_barrier();
        double *ga = d.alpha + l * BN + (size_t)b * N;
        reg_sweep(pr, mr, vb, va, eps, ga, loc); // Eq. 4
        if (!split_meet(cnt, (uint32_t)K * ++t, &d.ctr->error, &stop))
            return;
        split_gather(va, ga, N, loc);
        lds_barrier();
    }
    if (k == 0)
        sample_loss(d, b, d.row_ptr[(size_t)b * N], d.row_ptr[(size_t)(b + 1) * N], va, vb, part);
}

// One reverse half-sweep over the slots held in registers (as wide_reverse),
// with the owners' saved scalings al (iteration l) and alp (l - 1) loaded
// beforehand.
template <int SW, int OB>
__device__ __forceinline__ void reg_reverse(const WSlot (&w)[SW], float (&cp)[SW][kP], int n, const double (&al)[SW],
                                            const double (&alp)[SW], const float2 *fin, float *yout, bool local)
{
#pragma unroll
    for (int q = 0; q < SW; ++q) {
        if (q >= n)
            break;
        const Unpack u = Unpack::make();
        const int o = (int)u.bits(w[q].info, 0, OB);
        float2 f[kP];
#pragma unroll
        for (int e = 0; e < kP; ++e)
            f[e] = lds_at<float2>(fin, u.half(w[q].gi[e / 2], e));
        // rho_e = cp_e - f_e.x is formed again in the update (the same value):
        // keeping all of them would spill at two slots
        double acc = 0.0;
#pragma unroll
        for (int e = 0; e < kP; ++e) {
            const double rho = (double)cp[q][e] - (double)f[e].x;
            const double p0 = (double)w[q].p0[e];
            acc = e == 0 ? rho * p0 : __builtin_fma(rho, p0, acc);
        }
        const double dsum = al[q] * group_reduce_lg(acc, (int)u.bits(w[q].info, OB, 3));
        const double qt = quotient(al[q], alp[q]);
#pragma unroll
        for (int e = 0; e < kP; ++e) {
            const double rho = (double)cp[q][e] - (double)f[e].x;
            cp[q][e] = w[q].p0[e] != 0.0f ? (float)((rho - dsum * (double)f[e].y) * qt) : 0.0f;
        }
        if (u.bits(w[q].info, OB + 3, 2) == 3u) // head and valid
            publish32(yout + o, (float)(dsum * al[q]), local); // alp: read from the saved scalings
    }
}

// The owners' saved scalings of iteration l and l - 1 for the slots held.
template <int SW, int OB>
__device__ __forceinline__ void owner_scalings(const WSlot (&w)[SW], int n, const double *own_l, const double *own_prev,
                                               double (&al)[SW], double (&alp)[SW])
{
#pragma unroll
    for (int q = 0; q < SW; ++q)
        if (q < n) {
            const int o = (int)(w[q].info & ((1u << OB) - 1u));
            al[q] = own_l[o];
            alp[q] = own_prev[o];
        }
}

// The owners' saved scalings of iteration l - 1 alone.
template <int SW, int OB>
__device__ __forceinline__ void owner_prev(const WSlot (&w)[SW], int n, const double *own_prev, double (&alp)[SW])
{
#pragma unroll
    for (int q = 0; q < SW; ++q)
        if (q < n)
            alp[q] = own_prev[w[q].info & ((1u << OB) - 1u)];
}

template <int SW, bool HOLD> __global__ __launch_bounds__(kT) void k_sinkhorn_bwd_wr(DevPlan d, int K)
{
    constexpr int OB = 13; // owner bits of the streamed layout's info word
    __shared__ float2 fr[kSinkOwnersW]; // row factors (Yr_i, alpha^(l-1)_i)
    __shared__ float2 fc[kSinkOwnersW]; // column factors (Yc_j, beta^(l-1)_j)
    __shared__ int stop, local;
    int b, k;
    if (!split_member(blockIdx.x, d.B, K, b, k))
        return;
    const int tid = threadIdx.x;
    const int N = d.N, M = d.M, L = d.L;
    const size_t BN = (size_t)d.B * N, BM = (size_t)d.B * M;
    const double *alpha = d.alpha + (size_t)b * N, *beta = d.beta + (size_t)b * M; // + l * BN, + l * BM
    uint32_t *cnt = d.split_sync + ((size_t)b * 2 + 1) * kSplitSyncStride;
    const int mr = split_slots(__builtin_amdgcn_readfirstlane(d.wk_row.n_pos[b]), k, K);
    const int mc = split_slots(__builtin_amdgcn_readfirstlane(d.wk_col.n_pos[b]), k, K);
    WSlot pr[SW], pc[SW];
    load_my_slots(pr, d.wk_row, b, mr, k, K);
    load_my_slots(pc, d.wk_col, b, mc, k, K);
    // the copies start as grad_loss C beta^L_j (rows) and grad_loss C alpha^L_i (columns)
    float rr[SW][kP], rc[SW][kP];
    {
        const float *xb = d.x + (size_t)b * N * 3, *yb = d.y + (size_t)b * M * 3;
        const double gl = d.grad_loss[b];
        const Unpack u = Unpack::make();
#pragma unroll
        for (int q = 0; q < SW; ++q) {
#pragma unroll
            for (int e = 0; e < kP; ++e) {
                rr[q][e] = 0.0f;
                rc[q][e] = 0.0f;
            }
            if (q < mr) {
                const int i = (int)u.bits(pr[q].info, 0, OB);
#pragma unroll
                for (int e = 0; e < kP; ++e) {
                    const int j = (int)(u.half(pr[q].gi[e / 2], e) >> 3);
                    if (pr[q].p0[e] != 0.0f)
                        rr[q][e] = (float)(gl * dist_f64(xb + 3 * i, yb + 3 * j) * beta[(size_t)L * BM + j]);
                }
            }
            if (q < mc) {
                const int j = (int)u.bits(pc[q].info, 0, OB);
#pragma unroll
                for (int e = 0; e < kP; ++e) {
                    const int i = (int)(u.half(pc[q].gi[e / 2], e) >> 3);
                    if (pc[q].p0[e] != 0.0f)
                        rc[q][e] = (float)(gl * dist_f64(xb + 3 * i, yb + 3 * j) * alpha[(size_t)L * BN + i]);
                }
            }
        }
    }
    for (int o = tid; o < M; o += kT) // no pending column update before row phase L
        fc[o] = make_float2(0.0f, (float)beta[(size_t)L * BM + o]);
    if (tid == 0)
        stop = 0;
    lds_barrier();
    // the exchange as in k_sinkhorn_bwd_ws: a fresh region per phase
    if (!split_begin(cnt, K, k, &d.ctr->error, &stop, &local))
        return;
    const bool loc = local != 0;
    const SlotRsrc rsr = slot_rsrc(d.wk_row, b), rsc = slot_rsrc(d.wk_col, b);
    // Loads that do not depend on the exchange are issued ahead of it: a
    // phase's pieces (when streamed) and the gather's saved scalings before
    // the meeting, the owners' scalings before the gather. The owners of a
    // workgroup's slots are the same in every phase, so each phase loads only
    // their scalings of the previous iteration (alp); those of this iteration
    // (ar for the row owners, ac for the column owners) are the previous
    // phase's alp of the same side.
    double ar[SW], ac[SW], alp[SW];
    owner_scalings<SW, OB>(pr, mr, alpha + L * BN, alpha + (L - 1) * BN, ar, alp);
    {
        double unused[SW];
        owner_scalings<SW, OB>(pc, mc, beta + L * BM, beta + L * BM, ac, unused);
    }
    uint32_t t = 1;
    for (int l = L; l >= 1; --l) {
        float *yr = d.yr + (size_t)(L - l) * (BN + kSinkOwnersW) + (size_t)b * N;
        reg_reverse<SW, OB>(pr, rr, mr, ar, alp, fc, yr, loc); // reverse of Eq. 4
#pragma unroll
        for (int q = 0; q < SW; ++q)
            ar[q] = alp[q];
        if constexpr (!HOLD)
            stream_my_slots(pc, rsc, mc, k, K);
        float sp[8];
        if constexpr (HOLD)
            load_prev(sp, alpha + (l - 1) * BN, N);
        if (!split_meet(cnt, (uint32_t)K * ++t, &d.ctr->error, &stop))
            return;
        owner_prev<SW, OB>(pc, mc, beta + (l - 1) * BM, alp);
        if constexpr (!HOLD)
            load_prev(sp, alpha + (l - 1) * BN, N);
        split_gather_factors(fr, yr, sp, N, loc);
        lds_barrier();
        float *yc = d.yc + (size_t)(L - l) * (BM + kSinkOwnersW) + (size_t)b * M;
        reg_reverse<SW, OB>(pc, rc, mc, ac, alp, fr, yc, loc); // reverse of Eq. 3
#pragma unroll
        for (int q = 0; q < SW; ++q)
            ac[q] = alp[q];
        if constexpr (!HOLD)
            stream_my_slots(pr, rsr, mr, k, K); // the next row phase's, or the closing pass's
        if constexpr (HOLD)
            load_prev(sp, beta + (l - 1) * BM, M);
        if (!split_meet(cnt, (uint32_t)K * ++t, &d.ctr->error, &stop))
            return;
        if (l > 1)
            owner_prev<SW, OB>(pr, mr, alpha + (l - 2) * BN, alp);
        if constexpr (!HOLD)
            load_prev(sp, beta + (l - 1) * BM, M);
        split_gather_factors(fc, yc, sp, M, loc);
        lds_barrier();
    }
    // the adjoint with respect to P0, r - Yc_j, in row-major order
    {
        const Unpack u = Unpack::make();
#pragma unroll
        for (int q = 0; q < SW; ++q) {
            if (q >= mr || u.bits(pr[q].info, OB + 4, 1) == 0u)
                continue;
            const int i = (int)u.bits(pr[q].info, 0, OB), lg = (int)u.bits(pr[q].info, OB, 3);
            const int p = (k + q * K) * kT + tid, qq = p & ((1 << lg) - 1); // groups are aligned to their size
            const int r0 = d.row_ptr[(size_t)b * N + i], len = d.row_ptr[(size_t)b * N + i + 1] - r0;
#pragma unroll
            for (int e = 0; e < kP; ++e)
                if (qq * kP + e < len) {
                    const float2 f = lds_at<float2>(fc, u.half(pr[q].gi[e / 2], e));
                    d.adj[r0 + qq * kP + e] = (double)rr[q][e] - (double)f.x;
                }
        }
    }
}

__global__ __launch_bounds__(kBlock) void k_zero_u32(uint32_t *a, int n)
{
    const int k = blockIdx.x * kBlock + threadIdx.x;
    if (k < n)
        a[k] = 0u;
}

// per-iteration kernels (any N, M): one launch per sweep
// ---------------------------------------------------------------------------
//
// G lanes per owner (row or column; steps_lanes); each lane issues the loads
// of kSB of its pairs together before using them (kSBRev in the reverse
// launches, whose pairs carry 12 registers each: with 8 they held 101
// registers, four waves per SIMD; with 4, 61 and eight waves: reverse sweeps
// 0.525 -> 0.474 ms on 16 x 4096 x 16384 points, 0.455 -> 0.444 ms on
// 4 x 65536, measured side by side on one MI355X; 2 was slower than 4). Sums are per
// lane in pair order, then a butterfly over the group, so results do not
// depend on scheduling.
constexpr int kSG = 4;
constexpr int kSB = 8;
constexpr int kSBRev = 4;

__global__ __launch_bounds__(kBlock) void k_fill_ones(double *a, int n)
{
    const int k = blockIdx.x * kBlock + threadIdx.x;
    if (k < n)
        a[k] = 1.0;
}

// Sum over owner o's pairs k = lg, lg + kSG, ... of f(k, position) with the
// loads of kSB pairs in flight at once.
template <int G = kSG, int SB = kSB, class Load, class Use>
__device__ __forceinline__ double owner_sum(int n, int lg, Load load, Use use)
{
    double acc = 0.0;
    for (int k0 = lg; k0 < n; k0 += G * SB) {
        decltype(load(0)) v[SB];
#pragma unroll
        for (int u = 0; u < SB; ++u)
            v[u] = load(k0 + G * u < n ? k0 + G * u : -1);
#pragma unroll
        for (int u = 0; u < SB; ++u)
            if (k0 + G * u < n)
                acc += use(v[u]);
    }
    return group_sum<G>(acc);
}

// Column step (Eq. 3, COL) or row step (Eq. 4) of iteration l for all owners.
template <bool COL, int G> __global__ __launch_bounds__(kBlock) void k_sink_step(DevPlan d, int l, double eps)
{
    // each XCD takes a contiguous range of owners: its L2 holds only the
    // other side's scalings of those owners' samples
    const int gid = xcd_contiguous(blockIdx.x, gridDim.x) * kBlock + threadIdx.x;
    const int o = gid / G, lg = gid % G;
    const int n_own = COL ? d.M : d.N, n_oth = COL ? d.N : d.M;
    if (o >= d.B * n_own)
        return;
    const int b = o / n_own;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * d.M;
    const int32_t *ptr = COL ? d.col_ptr : d.row_ptr;
    const int32_t *idx = COL ? d.csc_row : d.csr_col;
    const float *p0 = COL ? d.p0c : d.p0r;
    // the other side's scalings: alpha^(l-1) for columns, beta^l for rows
    const double *oth = (COL ? d.alpha + (size_t)(l - 1) * BN : d.beta + (size_t)l * BM) + (size_t)b * n_oth;
    double *cur = COL ? d.beta : d.alpha;
    const size_t BO = COL ? BM : BN;
    const double prev = cur[(size_t)(l - 1) * BO + o]; // loaded with the segment bounds
    const int s0 = ptr[o], n = ptr[o + 1] - s0;
    struct V {
        float p;
        double x;
    };
    const double acc = owner_sum<G>(n, lg,
                                 [&](int k) {
                                     V v{0.0f, 0.0};
                                     if (k >= 0) {
                                         v.p = p0[s0 + k];
                                         v.x = oth[idx[s0 + k]];
                                     }
                                     return v;
                                 },
                                 [&](const V &v) { return (double)v.p * v.x; });
    if (lg == 0) {
        const double den = prev * acc + eps;
        cur[(size_t)l * BO + o] = prev / den;
    }
}

template <int G> __global__ __launch_bounds__(kBlock) void k_loss_rows(DevPlan d, double *loss_rows)
{
    const int gid = xcd_contiguous(blockIdx.x, gridDim.x) * kBlock + threadIdx.x; // as in k_sink_step
    const int r = gid / G, lg = gid % G;
    if (r >= d.B * d.N)
        return;
    const int b = r / d.N;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * d.M;
    const double *beta = d.beta + (size_t)d.L * BM + (size_t)b * d.M;
    const int t0 = d.row_ptr[r], n = d.row_ptr[r + 1] - t0;
    struct V {
        float p;
        double bc;
    };
    const double acc = owner_sum<G>(n, lg,
                                 [&](int k) {
                                     V v{0.0f, 0.0};
                                     if (k >= 0) {
                                         v.p = d.p0r[t0 + k];
                                         v.bc = beta[d.csr_col[t0 + k]] * d.cost[t0 + k];
                                     }
                                     return v;
                                 },
                                 [&](const V &v) { return (double)v.p * v.bc; });
    if (lg == 0)
        loss_rows[r] = d.alpha[(size_t)d.L * BN + r] * acc;
}

// Per sample: the sum of its row losses. 1024 threads, four partial sums per
// thread so that four loads are in flight; fixed association.
constexpr int kLossT = 1024;

__global__ __launch_bounds__(kLossT) void k_loss_reduce(DevPlan d, const double *loss_rows)
{
    __shared__ double part[kLossT / 64];
    const int b = blockIdx.x;
    const double *lr = loss_rows + (size_t)b * d.N;
    double s[4] = {0.0, 0.0, 0.0, 0.0};
    for (int i0 = threadIdx.x; i0 < d.N; i0 += 4 * kLossT)
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (i0 + u * kLossT < d.N)
                s[u] += lr[i0 + u * kLossT];
    double t = wave_sum((s[0] + s[1]) + (s[2] + s[3]));
    if (lane_id() == 0)
        part[threadIdx.x >> 6] = t;
    __syncthreads();
    if (threadIdx.x == 0) {
        double a = 0.0;
        for (int w = 0; w < kLossT / 64; ++w)
            a += part[w];
        d.loss[b] = (float)a;
    }
}

// Reverse sweeps, one launch per half-step. The adjoint is kept twice in
// double precision, in row order (rz) and in column order (kz), in the
// scaled form of the per-sample kernel (adjoint * alpha^l before a row
// phase, * beta^l before a column phase), and each copy is brought up to
// date in its own order, so no launch reads or writes pairs out of order:
//   row launch l:    rz <- column update of iteration l+1 (l < L), then the
//                    row update of iteration l; row sums; row values
//                    X_i = alpha^l_i, Y_i = d_i alpha^l_i and 1/alpha^l_i into xyr
//   column launch l: kz <- row update of iteration l, then the column update
//                    of iteration l; column sums; column values X_j =
//                    beta^l_j, Y_j = e_j beta^l_j and 1/beta^l_j into xyc
// where the row update of iteration l is z' = (z / alpha^l_i) X_j - Y_j with
// the column values published last, and the column update z' = (z / beta^l_j)
// X_i - Y_i with the row values of iteration l. The other side's values of a
// pair arrive in one 32-byte gather; values, sums and updates are double
// (single-precision factors left gradient errors of 1e-5 that moved with the
// rounding of the sums).
__global__ __launch_bounds__(kBlock) void k_bwd_init(DevPlan d)
{
    const int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const size_t BN = (size_t)d.B * d.N, BM = (size_t)d.B * d.M;
    if (g < d.nnz) { // row order: grad_loss * C, times alpha^L_i
        const int r = d.csr_row[g], b = r / d.N;
        d.rz[g] = d.grad_loss[b] * d.cost[g] * d.alpha[(size_t)d.L * BN + r];
        // column order: the same pair through the permutation
        const int t = d.csc_perm[g], rr = d.csr_row[t], bb = rr / d.N;
        d.kz[g] = d.grad_loss[bb] * d.cost[t] * d.alpha[(size_t)d.L * BN + rr];
    }
    if (g < (int64_t)BM) { // no pending column update before the last iteration
        const double bl = d.beta[(size_t)d.L * BM + g];
        d.xyc[g] = make_double4(bl, 0.0, 1.0 / bl, 0.0);
    }
}

template <int G> __global__ __launch_bounds__(kBlock) void k_bwd_rows(DevPlan d, int l)
{
    const int gid = xcd_contiguous(blockIdx.x, gridDim.x) * kBlock + threadIdx.x; // as in k_sink_step
    const int r = gid / G, lg = gid % G;
    if (r >= d.B * d.N)
        return;
    const int b = r / d.N;
    const size_t BN = (size_t)d.B * d.N;
    const double4 *xyc = d.xyc + (size_t)b * d.M;
    const bool pending = l < d.L;
    const double4 mine = pending ? d.xyr[r] : make_double4(0.0, 0.0, 0.0, 0.0); // row values of iteration l+1
    const double al = d.alpha[(size_t)l * BN + r];
    const double inv_a = 1.0 / al;
    const int t0 = d.row_ptr[r], n = d.row_ptr[r + 1] - t0;
    struct V {
        double z;
        float p;
        int k;
        double4 c;
    };
    const double acc = owner_sum<G, kSBRev>(n, lg,
                                         [&](int k) {
                                             V v{0.0, 0.0f, k, make_double4(0.0, 0.0, 1.0, 0.0)};
                                             if (k >= 0) {
                                                 const int j = d.csr_col[t0 + k];
                                                 v.z = d.rz[t0 + k];
                                                 v.p = d.p0r[t0 + k];
                                                 v.c = xyc[j];
                                             }
                                             return v;
                                         },
                                         [&](const V &v) {
                                             double z = v.z;
                                             if (pending) // 1/beta^(l+1)_j
                                                 z = __builtin_fma(z * v.c.z, mine.x, -mine.y);
                                             z = __builtin_fma(z * inv_a, v.c.x, -v.c.y);
                                             d.rz[t0 + v.k] = z;
                                             return z * (double)v.p;
                                         });
    if (lg == 0) { // adjoint of Eq. 4: d_i = alpha^l_i * sum
        const double dsum = al * acc;
        d.xyr[r] = make_double4(al, dsum * al, inv_a, 0.0);
    }
}

template <int G> __global__ __launch_bounds__(kBlock) void k_bwd_cols(DevPlan d, int l)
{
    const int gid = xcd_contiguous(blockIdx.x, gridDim.x) * kBlock + threadIdx.x; // as in k_sink_step
    const int gc = gid / G, lg = gid % G;
    if (gc >= d.B * d.M)
        return;
    const int b = gc / d.M;
    const size_t BM = (size_t)d.B * d.M;
    const double4 *xyr = d.xyr + (size_t)b * d.N;
    const double4 mine = d.xyc[gc]; // column values published last
    const double bl = d.beta[(size_t)l * BM + gc];
    const double inv_b = 1.0 / bl;
    const int s0 = d.col_ptr[gc], n = d.col_ptr[gc + 1] - s0;
    struct V {
        double z;
        float p;
        int k;
        double4 rw;
    };
    const double acc = owner_sum<G, kSBRev>(n, lg,
                                         [&](int k) {
                                             V v{0.0, 0.0f, k, make_double4(0.0, 0.0, 1.0, 0.0)};
                                             if (k >= 0) {
                                                 const int i = d.csc_row[s0 + k];
                                                 v.z = d.kz[s0 + k];
                                                 v.p = d.p0c[s0 + k];
                                                 v.rw = xyr[i];
                                             }
                                             return v;
                                         },
                                         [&](const V &v) { // v.rw.z = 1/alpha^l_i
                                             double z = __builtin_fma(v.z * v.rw.z, mine.x, -mine.y);
                                             z = __builtin_fma(z * inv_b, v.rw.x, -v.rw.y);
                                             d.kz[s0 + v.k] = z;
                                             return z * (double)v.p;
                                         });
    if (lg == 0) { // adjoint of Eq. 3: e_j = beta^l_j * sum
        const double esum = bl * acc;
        d.xyc[gc] = make_double4(bl, esum * bl, inv_b, 0.0);
    }
}

// dLoss/dP0 in row order: the column update of iteration 1, then the row
// update of iteration 0 (alpha^0 = 1).
__global__ __launch_bounds__(kBlock) void k_bwd_final(DevPlan d)
{
    const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (t >= d.nnz)
        return;
    const int r = d.csr_row[t], b = r / d.N, j = d.csr_col[t];
    const double4 rw = d.xyr[r];
    const double4 c = d.xyc[(size_t)b * d.M + j]; // c.z = 1/beta^1_j
    double z = __builtin_fma(d.rz[t] * c.z, rw.x, -rw.y);
    d.adj[t] = z * c.x - c.y;
}

} // namespace

int sinkhorn_slots(int N, int M, const int32_t *counts, int B)
{
    if (N > kSinkOwners || M > kSinkOwners)
        return 0;
    int most = 1;
    for (int b = 0; b < B; ++b) {
        if (counts[4 * b + 2] > kSinkMaxGroup || counts[4 * b + 3] > kSinkMaxGroup)
            return 0;
        most = std::max({most, counts[4 * b], counts[4 * b + 1]});
    }
    const int slots = (most + kT - 1) / kT;
    return slots <= kSinkMaxSlots ? slots : 0;
}

int sinkhorn_slots_wide(int N, int M, const int32_t *counts, int B)
{
    if (N > kSinkOwnersW || M > kSinkOwnersW)
        return 0;
    int most = 1;
    for (int b = 0; b < B; ++b) {
        if (counts[4 * b + 2] > kSinkMaxGroup || counts[4 * b + 3] > kSinkMaxGroup)
            return 0;
        most = std::max({most, counts[4 * b], counts[4 * b + 1]});
    }
    const int slots = (most + kT - 1) / kT;
    return slots <= kSinkMaxSlotsW ? slots : 0;
}

void launch_wide_pack(const DevPlan &d, int32_t *place, hipStream_t s)
{
    hipLaunchKernelGGL(k_place_w, dim3(d.B, 2), dim3(kT), 0, s, d, place);
    hipLaunchKernelGGL(k_pack_w, dim3(blocks_for(2 * d.nnz, kBlock)), dim3(kBlock), 0, s, d, (const int32_t *)place);
}

int sinkhorn_split_factor(int B)
{
    const char *env = std::getenv("APML_SINKHORN_SPLIT");
    if (env && env[0] == '0')
        return 1;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64 || B < 1)
        return 1;
    // workgroups of the split kernels resident at once on each device, plus 1
    // (0: not yet queried)
    static std::atomic<int> resident[64];
    int c = resident[dev].load(std::memory_order_relaxed);
    if (c == 0) {
        int cus = 0, coop = 0, f = 0, r = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&f, reinterpret_cast<const void *>(k_sinkhorn_fwd_ws), kT, 0) !=
                hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&r, reinterpret_cast<const void *>(k_sinkhorn_bwd_ws), kT, 0) !=
                hipSuccess) {
            (void)hipGetLastError();
            cus = coop = 0;
        }
        c = (coop ? cus * std::min(f, r) : 0) + 1;
        resident[dev].store(c, std::memory_order_relaxed);
    }
    // the grid rounds B up to whole rounds of the eight XCDs
    const int K = std::min(kSplitMax, (c - 1) / split_grid(B, 1));
    return K >= 2 ? K : 1;
}

namespace {

// Clears the sample's meeting counters, then launches the split kernel over
// B K workgroups, all resident at once; false when the cooperative launch
// is refused (the caller then takes the one-workgroup kernel).
bool launch_split(const void *kernel, void **args, const DevPlan &d, int K, hipStream_t s)
{
    const int n = d.B * 2 * kSplitSyncStride;
    hipLaunchKernelGGL(k_zero_u32, dim3(blocks_for(n, kBlock)), dim3(kBlock), 0, s, d.split_sync, n);
    if (hipGetLastError() != hipSuccess)
        return false;
    if (hipLaunchCooperativeKernel(kernel, dim3(split_grid(d.B, K)), dim3(kT), args, 0, s) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    return true;
}

// APML_SINKHORN_SPLIT=streamed keeps the split kernels but takes their
// streamed variants at any share (the variants give the same bits; this
// lets them be compared).
bool split_streamed_only()
{
    const char *env = std::getenv("APML_SINKHORN_SPLIT");
    return env && env[0] == 's';
}

// The split kernel for a workgroup share of sw slots per lane and order:
// registers up to the limit, else streamed.
const void *split_fwd_kernel(int sw)
{
    if (split_streamed_only())
        return reinterpret_cast<const void *>(k_sinkhorn_fwd_ws);
    switch (sw) {
    case 1: return reinterpret_cast<const void *>(k_sinkhorn_fwd_wr<1>);
    case 2: return reinterpret_cast<const void *>(k_sinkhorn_fwd_wr<2>);
    case 3: return reinterpret_cast<const void *>(k_sinkhorn_fwd_wr<3>);
    default: return reinterpret_cast<const void *>(k_sinkhorn_fwd_ws);
    }
}

const void *split_bwd_kernel(int sw)
{
    if (split_streamed_only())
        return reinterpret_cast<const void *>(k_sinkhorn_bwd_ws);
    switch (sw) {
    case 1: return reinterpret_cast<const void *>(k_sinkhorn_bwd_wr<1, true>);
    case 2: return reinterpret_cast<const void *>(k_sinkhorn_bwd_wr<2, true>);
    case 3: return reinterpret_cast<const void *>(k_sinkhorn_bwd_wr<3, false>);
    default: return reinterpret_cast<const void *>(k_sinkhorn_bwd_ws);
    }
}

static_assert(kSplitRegFwd == 3 && kSplitRegBwd == 2 && kSplitAdjBwd == 3, "instances above");

} // namespace

hipError_t launch_sinkhorn_fwd_wide(const DevPlan &d, double eps, hipStream_t s)
{
    // a forward half-sweep over fewer slots is shorter than the meeting that
    // splitting it needs (measured: 3000 to 4096 points per cloud, 4 to 6
    // slots, 0.09 -> 0.13 ms; large-batch workload, 12 slots, 0.51 -> 0.35 ms)
    constexpr int kSplitFwdMinSlots = 8;
    int K = d.wk_row.slots >= kSplitFwdMinSlots ? sinkhorn_split_factor(d.B) : 1;
    if (K > 1 && d.split_sync) {
        DevPlan dc = d;
        double e = eps;
        void *args[] = {&dc, &e, &K};
        if (launch_split(split_fwd_kernel((d.wk_row.slots + K - 1) / K), args, d, K, s))
            return hipSuccess;
    }
    hipLaunchKernelGGL(k_sinkhorn_fwd_w, dim3(d.B), dim3(kT), 0, s, d, eps);
    return hipGetLastError();
}

hipError_t launch_sinkhorn_bwd_wide(const DevPlan &d, hipStream_t s)
{
    int K = sinkhorn_split_factor(d.B);
    if (K > 1 && d.split_sync && d.yr && d.yc) {
        DevPlan dc = d;
        void *args[] = {&dc, &K};
        if (launch_split(split_bwd_kernel((d.wk_row.slots + K - 1) / K), args, d, K, s))
            return hipSuccess;
    }
    hipLaunchKernelGGL(k_sinkhorn_bwd_w, dim3(d.B), dim3(kT), 0, s, d);
    return hipGetLastError();
}

constexpr size_t kLdsBudget = 160 * 1024;

bool sinkhorn_bwd_fits(int slots, int64_t max_pairs)
{
    // the adjoint of every pair of a sample in LDS, at its row piece
    (void)max_pairs;
    return slots > 0 && bwd_fixed_lds_bytes() + 4 * (size_t)(adj_slots(slots) + 1) <= kLdsBudget;
}

size_t packed_order_words(int B, int slots) { return (size_t)B * slots * kP * kT; }

void launch_place(const DevPlan &d, int32_t *place, hipStream_t s)
{
    hipLaunchKernelGGL(k_place, dim3(d.B, 2), dim3(kT), 0, s, d, place);
}

void launch_pack(const DevPlan &d, int32_t *place, bool placed, hipStream_t s)
{
    if (!placed)
        hipLaunchKernelGGL(k_place, dim3(d.B, 2), dim3(kT), 0, s, d, place);
    hipLaunchKernelGGL(k_pack_pairs, dim3(blocks_for(2 * d.nnz, kBlock)), dim3(kBlock), 0, s, d, (const int32_t *)place);
}

// The kernel instance for the plan's slot count.
template <template <int> class K> static auto for_slots(int slots) -> decltype(K<1>::fn)
{
    switch (slots) {
    case 1: return K<1>::fn;
    case 2: return K<2>::fn;
    case 3: return K<3>::fn;
    case 4: return K<4>::fn;
    case 5: return K<5>::fn;
    default: return K<6>::fn;
    }
}
template <int S> struct FwdK { static constexpr auto fn = k_sinkhorn_fwd<S>; };
template <int S> struct BwdK { static constexpr auto fn = k_sinkhorn_bwd<S>; };

hipError_t launch_sinkhorn_fwd(const DevPlan &d, double eps, hipStream_t s)
{
    const auto k = for_slots<FwdK>(d.pk_row.slots);
    hipLaunchKernelGGL(k, dim3(d.B), dim3(kT), 0, s, d, eps);
    return hipGetLastError();
}

hipError_t launch_sinkhorn_bwd(const DevPlan &d, int64_t max_pairs, hipStream_t s)
{
    (void)max_pairs;
    const size_t bytes = 4 * (size_t)(adj_slots(d.pk_row.slots) + 1); // beyond the static arrays
    const auto k = for_slots<BwdK>(d.pk_row.slots);
    hipError_t e = set_dynamic_lds((const void *)k, bytes);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k, dim3(d.B), dim3(kT), bytes, s, d);
    return hipGetLastError();
}

namespace {

// Lanes per owner of the per-iteration kernels: the largest power of two
// up to the owners' mean pair count, within 4..16 (rows of 18 pairs on
// average: 16 lanes took the sweeps of the unequal workload from 0.38 / 0.79
// ms to 0.29 / 0.61 ms; at 5 pairs, 4 lanes stay the fastest).
int steps_lanes(int64_t nnz, int64_t owners)
{
    int g = kSG;
    while (g < 16 && (int64_t)g * 2 * owners <= nnz)
        g *= 2;
    return g;
}

template <template <int> class K, class... A>
void launch_lanes(int g, int64_t owners, hipStream_t s, A... args)
{
    switch (g) {
    case 8: hipLaunchKernelGGL(K<8>::fn, dim3(blocks_for(owners * 8, kBlock)), dim3(kBlock), 0, s, args...); break;
    case 16: hipLaunchKernelGGL(K<16>::fn, dim3(blocks_for(owners * 16, kBlock)), dim3(kBlock), 0, s, args...); break;
    default: hipLaunchKernelGGL(K<4>::fn, dim3(blocks_for(owners * 4, kBlock)), dim3(kBlock), 0, s, args...); break;
    }
}
template <int G> struct ColStep { static constexpr auto fn = k_sink_step<true, G>; };
template <int G> struct RowStep { static constexpr auto fn = k_sink_step<false, G>; };
template <int G> struct BwdRows { static constexpr auto fn = k_bwd_rows<G>; };
template <int G> struct BwdCols { static constexpr auto fn = k_bwd_cols<G>; };
template <int G> struct LossRows { static constexpr auto fn = k_loss_rows<G>; };

} // namespace

void launch_sinkhorn_fwd_steps(const DevPlan &d, double eps, hipStream_t s)
{
    const int BN = d.B * d.N, BM = d.B * d.M;
    const int gr = steps_lanes(d.nnz, BN), gc = steps_lanes(d.nnz, BM);
    hipLaunchKernelGGL(k_fill_ones, dim3(blocks_for(BN, kBlock)), dim3(kBlock), 0, s, d.alpha, BN);
    hipLaunchKernelGGL(k_fill_ones, dim3(blocks_for(BM, kBlock)), dim3(kBlock), 0, s, d.beta, BM);
    for (int l = 1; l <= d.L; ++l) {
        launch_lanes<ColStep>(gc, BM, s, d, l, eps);
        launch_lanes<RowStep>(gr, BN, s, d, l, eps);
    }
    // the backward scratch is free during the forward pass: use it for the row losses
    launch_lanes<LossRows>(gr, BN, s, d, d.dvec);
    hipLaunchKernelGGL(k_loss_reduce, dim3(d.B), dim3(kLossT), 0, s, d, (const double *)d.dvec);
}

void launch_sinkhorn_bwd_steps(const DevPlan &d, hipStream_t s)
{
    const int BN = d.B * d.N, BM = d.B * d.M;
    const int gr = steps_lanes(d.nnz, BN), gc = steps_lanes(d.nnz, BM);
    hipLaunchKernelGGL(k_bwd_init, dim3(blocks_for(std::max<int64_t>(d.nnz, BM), kBlock)), dim3(kBlock), 0, s, d);
    for (int l = d.L; l >= 1; --l) {
        launch_lanes<BwdRows>(gr, BN, s, d, l);
        launch_lanes<BwdCols>(gc, BM, s, d, l);
    }
    hipLaunchKernelGGL(k_bwd_final, dim3(blocks_for(d.nnz, kBlock)), dim3(kBlock), 0, s, d);
}

} // namespace apml
