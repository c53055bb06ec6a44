// HIP kernels of the sparse APML loss for gfx950 (wave64).
//
// Dense phase (all B*N*M pairs, VALU-bound, no matrix cores: the K=3
// contraction is not a GEMM):
//   k_top2    per row and per column, the minimum and second minimum of the
//             single-precision squared distance (Sec. III-A). Each lane owns
//             one point; the other cloud is streamed through scalar registers
//             (wave-uniform loads), so a pair costs 6 VALU ops for the
//             distance and 2 (min, med3) for the statistics.
//   k_emit    the candidate support: every pair inside the row radius or the
//             column radius (the kept set s >= tau is a ball, Sec. III-B), or
//             at most the second minimum. Each lane appends its row's pairs,
//             already in column order, to a private slot group.
// Sparse phase (O(nnz), memory-bound), all sums taken sequentially per
// segment so that results are bitwise reproducible:
//   scans, row-major (CSR) fill, column-major (CSC) permutation,
//   k_row_softmax / k_col_softmax  temperatures (Eq. 1 + clamp), softmaxes on
//             the kept support (Eq. 2, kept-sum normalisation), P0
//   k_sink_col / k_sink_row        Sinkhorn in scaling form (Eq. 3, Eq. 4)
//   k_loss_rows / k_loss_reduce    sum_t v_t C_t (Sec. III-D)
//   backward kernels               reverse Sinkhorn, softmax and temperature
//             adjoints, distance gradient (Eq. 5)
#include <cmath>

#include "apml_internal.h"

namespace apml {
namespace {

constexpr float kInf = __builtin_huge_valf();

// Squared distance in single precision, as d = a - b per coordinate, then
// dx*dx, fma(dy,dy,.), fma(dz,dz,.). The dense scans and the sparse passes
// evaluate exactly this sequence, so their values agree bit for bit.
__device__ __forceinline__ float sqdist_f32(float ax, float ay, float az, float bx, float by,
                                            float bz)
{
    const float dx = ax - bx, dy = ay - by, dz = az - bz;
    float s = dx * dx;
    s = __builtin_fmaf(dy, dy, s);
    s = __builtin_fmaf(dz, dz, s);
    return s;
}

// Cost C = ||a - b||_2 in double precision from float coordinates.
__device__ __forceinline__ double dist_f64(const float *a, const float *b)
{
    const double dx = (double)a[0] - (double)b[0];
    const double dy = (double)a[1] - (double)b[1];
    const double dz = (double)a[2] - (double)b[2];
    return sqrt(dx * dx + dy * dy + dz * dz);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// Read-only data seen through the constant address space: wave-uniform loads
// from it become scalar loads even in kernels that also store to memory.
template <typename T> using const_ptr = const __attribute__((address_space(4))) T *;
typedef float f32x4 __attribute__((ext_vector_type(4)));
template <typename T> __device__ __forceinline__ const_ptr<T> as_const(const T *p)
{
    return (const_ptr<T>)p;
}

// ---------------------------------------------------------------------------
// dense scan 1: minimum and second minimum per owner and chunk
// ---------------------------------------------------------------------------

struct Top2Args {
    ScanDir dir[2];
    int B;
};

__global__ __launch_bounds__(kBlock) void k_top2(Top2Args args)
{
    int t = blockIdx.x;
    const int which = t < args.dir[0].tiles ? 0 : 1;
    if (which)
        t -= args.dir[0].tiles;
    const ScanDir &d = args.dir[which];
    const int ob = t % d.owner_blocks;
    const int rest = t / d.owner_blocks;
    const int ch = rest % d.S;
    const int b = rest / d.S;
    const int a = ob * kBlock + threadIdx.x;
    const bool valid = a < d.n_own;
    const float *p = d.own + ((size_t)b * d.n_own + (valid ? a : d.n_own - 1)) * 3;
    const float ax = p[0], ay = p[1], az = p[2];
    const float *__restrict__ q = d.bcast + (size_t)b * d.n_bc * 3;
    const int j0 = ch * d.chunk;
    const int j1 = min(d.n_bc, j0 + d.chunk);
    float m1 = kInf, m2 = kInf;
    int j = j0;
    for (; j + kUnroll <= j1; j += kUnroll) {
        const float *__restrict__ qq = q + 3 * (size_t)j;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const float s = sqdist_f32(ax, ay, az, qq[3 * u], qq[3 * u + 1], qq[3 * u + 2]);
            m2 = __builtin_amdgcn_fmed3f(m1, m2, s); // second order statistic of the multiset
            m1 = fminf(m1, s);
        }
    }
    for (; j < j1; ++j) {
        const float s = sqdist_f32(ax, ay, az, q[3 * j], q[3 * j + 1], q[3 * j + 2]);
        m2 = __builtin_amdgcn_fmed3f(m1, m2, s);
        m1 = fminf(m1, s);
    }
    if (valid)
        d.partial[(size_t)ch * args.B * d.n_own + (size_t)b * d.n_own + a] = make_float2(m1, m2);
}

// ---------------------------------------------------------------------------
// merge of the chunk statistics, emission thresholds
// ---------------------------------------------------------------------------

struct FinalizeArgs {
    FinalizeDir dir[2];
    int B;
    int rows; // B * n_own of dir[0]
    Params p;
};

__global__ __launch_bounds__(kBlock) void k_finalize(FinalizeArgs args)
{
    int k = blockIdx.x * kBlock + threadIdx.x;
    const int which = k < args.rows ? 0 : 1;
    if (which)
        k -= args.rows;
    const FinalizeDir &d = args.dir[which];
    if (k >= args.B * d.n_own)
        return;
    const size_t stride = (size_t)args.B * d.n_own;
    float m1 = kInf, m2 = kInf;
    for (int c = 0; c < d.S; ++c) {
        const float2 v = d.partial[c * stride + k];
        // top-2 of the union of two top-2 multisets
        m2 = fminf(fmaxf(m1, v.x), fminf(m2, v.y));
        m1 = fminf(m1, v.x);
    }
    d.m12[k] = make_float2(m1, m2);
    // Radius of the kept ball from the single-precision minima. The exact
    // test s >= tau is applied later in double precision; the relative
    // margin covers the rounding of this estimate and of the distance.
    const Params &p = args.p;
    const double c1 = sqrt((double)m1), c2 = sqrt((double)m2);
    const double gap = (c2 - c1) + p.delta;
    const double g = gap < p.eps_gap ? p.eps_gap : gap;
    const double kappa = p.log_inv_tau / d.log_ratio; // log(1/tau) / (T g)
    const double radius = c1 + g * kappa;
    const double margin = 1e-5 * (1.0 + kappa);
    double e = radius * radius * (1.0 + margin);
    e = fmax(e, (double)m2); // the second minimum is always emitted
    const float E = isinf(e) ? kInf : __double2float_ru(e);
    if (which == 0) {
        d.E[k] = E;
    } else {
        const float *o = d.own + (size_t)k * 3;
        d.packed[k] = make_float4(o[0], o[1], o[2], E);
    }
}

// ---------------------------------------------------------------------------
// dense scan 2: candidate support, appended per (row, chunk) in column order
// ---------------------------------------------------------------------------

// Appends pair (row, j) to the lane's slot group, or to the overflow list.
__device__ __forceinline__ void emit_pair(const EmitArgs &a, int32_t *slot, int row, int ch, int j,
                                          int &cnt)
{
    if (cnt < a.K) {
        slot[cnt] = j;
    } else {
        const unsigned o = atomicAdd(&a.ctr->overflow, 1u);
        if (o < a.ovf_cap)
            a.ovf[o] = OverflowEntry{row, ch, cnt, j};
    }
    ++cnt;
}

// Handles column j once the wave knows some lane hit it: the hitting lanes
// append the pair, one lane adds the wave's hits to the column count.
__device__ __forceinline__ void emit_column(const EmitArgs &a, int32_t *slot, int row, int ch,
                                            int b, int j, unsigned long long m, int lane, int &cnt)
{
    if ((m >> lane) & 1ull)
        emit_pair(a, slot, row, ch, j, cnt);
    if (lane == __ffsll((unsigned long long)m) - 1)
        atomicAdd(&a.col_cnt[(size_t)b * a.M + j], (int)__popcll(m));
}

__global__ __launch_bounds__(kBlock) void k_emit(EmitArgs a)
{
    const int t = blockIdx.x;
    const int ob = t % a.owner_blocks;
    const int rest = t / a.owner_blocks;
    const int ch = rest % a.S;
    const int b = rest / a.S;
    const int i = ob * kBlock + threadIdx.x;
    const bool valid = i < a.N;
    const unsigned long long valid_mask = __builtin_amdgcn_ballot_w64(valid);
    const int row = b * a.N + (valid ? i : a.N - 1);
    const float *p = a.x + (size_t)row * 3;
    const float ax = p[0], ay = p[1], az = p[2];
    const float E = a.E_row[row];
    const_ptr<f32x4> q = as_const(reinterpret_cast<const f32x4 *>(a.ypack + (size_t)b * a.M));
    const int j0 = ch * a.chunk;
    const int j1 = min(a.M, j0 + a.chunk);
    int32_t *slot = a.slots + ((size_t)row * a.S + ch) * a.K;
    const int lane = lane_id();
    int cnt = 0;
    int j = j0;
    // Common path: per column the distance and two compares whose wave masks
    // are OR'ed on the scalar unit; one branch per 4 columns.
    for (; j + 4 <= j1; j += 4) {
        unsigned long long mk[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const f32x4 yv = q[j + u];
            const float s = sqdist_f32(ax, ay, az, yv.x, yv.y, yv.z);
            mk[u] = (__builtin_amdgcn_ballot_w64(s <= E) | __builtin_amdgcn_ballot_w64(s <= yv.w)) &
                    valid_mask;
        }
        if (mk[0] | mk[1] | mk[2] | mk[3]) {
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (mk[u])
                    emit_column(a, slot, row, ch, b, j + u, mk[u], lane, cnt);
        }
    }
    for (; j < j1; ++j) {
        const f32x4 yv = q[j];
        const float s = sqdist_f32(ax, ay, az, yv.x, yv.y, yv.z);
        const unsigned long long m =
            (__builtin_amdgcn_ballot_w64(s <= E) | __builtin_amdgcn_ballot_w64(s <= yv.w)) & valid_mask;
        if (m)
            emit_column(a, slot, row, ch, b, j, m, lane, cnt);
    }
    if (valid)
        a.cnt[(size_t)row * a.S + ch] = cnt;
    int w = cnt;
    for (int off = 32; off > 0; off >>= 1)
        w += __shfl_xor(w, off);
    if (lane == 0 && w)
        atomicAdd(&a.ctr->stored, (unsigned long long)w);
}

// ---------------------------------------------------------------------------
// exclusive prefix sums (three phases: tile sums, scan of tile sums, apply)
// ---------------------------------------------------------------------------

constexpr int kScanItems = 8;
constexpr int kScanTile = kBlock * kScanItems;

struct ScanPair {
    ScanArray a[2];
};

__device__ __forceinline__ int scan_load(const ScanArray &a, int k)
{
    if (k >= a.n)
        return 0;
    int s = 0;
    for (int c = 0; c < a.S; ++c)
        s += a.in[(size_t)k * a.S + c];
    return s;
}

// Exclusive scan of one value per thread over the block; *total gets the sum.
__device__ int block_exclusive_scan(int v, int *total)
{
    __shared__ int wave_sums[kBlock / 64];
    const int lane = lane_id(), wave = threadIdx.x >> 6;
    int inc = v;
    for (int off = 1; off < 64; off <<= 1) {
        const int n = __shfl_up(inc, off);
        if (lane >= off)
            inc += n;
    }
    if (lane == 63)
        wave_sums[wave] = inc;
    __syncthreads();
    int base = 0, all = 0;
    for (int w = 0; w < kBlock / 64; ++w) {
        if (w < wave)
            base += wave_sums[w];
        all += wave_sums[w];
    }
    __syncthreads();
    *total = all;
    return base + inc - v;
}

__global__ __launch_bounds__(kBlock) void k_scan_reduce(ScanPair sp)
{
    const ScanArray &a = sp.a[blockIdx.y];
    if ((int)blockIdx.x >= a.tiles)
        return;
    const int k0 = blockIdx.x * kScanTile + threadIdx.x * kScanItems;
    int s = 0;
    for (int u = 0; u < kScanItems; ++u)
        s += scan_load(a, k0 + u);
    int total;
    block_exclusive_scan(s, &total);
    if (threadIdx.x == 0)
        a.tile_sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kBlock) void k_scan_tiles(ScanPair sp)
{
    const ScanArray &a = sp.a[blockIdx.y];
    int carry = 0;
    for (int base = 0; base < a.tiles; base += kBlock) {
        const int k = base + threadIdx.x;
        const int v = k < a.tiles ? a.tile_sums[k] : 0;
        int total;
        const int ex = block_exclusive_scan(v, &total);
        if (k < a.tiles)
            a.tile_sums[k] = carry + ex;
        carry += total;
    }
    if (threadIdx.x == 0)
        a.out[a.n] = carry;
}

__global__ __launch_bounds__(kBlock) void k_scan_apply(ScanPair sp)
{
    const ScanArray &a = sp.a[blockIdx.y];
    if ((int)blockIdx.x >= a.tiles)
        return;
    const int k0 = blockIdx.x * kScanTile + threadIdx.x * kScanItems;
    int v[kScanItems];
    int s = 0;
    for (int u = 0; u < kScanItems; ++u) {
        v[u] = scan_load(a, k0 + u);
        s += v[u];
    }
    int total;
    int run = block_exclusive_scan(s, &total) + a.tile_sums[blockIdx.x];
    for (int u = 0; u < kScanItems; ++u) {
        if (k0 + u < a.n)
            a.out[k0 + u] = run;
        run += v[u];
    }
}

// ---------------------------------------------------------------------------
// row-major fill and column-major permutation
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_csr_fill(BuildArgs a)
{
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= a.B * a.N)
        return;
    int pos = a.row_ptr[r];
    for (int c = 0; c < a.S; ++c) {
        const int n = a.cnt[(size_t)r * a.S + c];
        const int m = min(n, a.K);
        const int32_t *sl = a.slots + ((size_t)r * a.S + c) * a.K;
        for (int k = 0; k < m; ++k)
            a.csr_col[pos + k] = sl[k];
        pos += n;
    }
}

__global__ __launch_bounds__(kBlock) void k_ovf_fill(BuildArgs a)
{
    const int o = blockIdx.x * kBlock + threadIdx.x;
    if (o >= a.n_ovf)
        return;
    const OverflowEntry e = a.ovf[o];
    int pos = a.row_ptr[e.row];
    for (int c = 0; c < e.chunk; ++c)
        pos += a.cnt[(size_t)e.row * a.S + c];
    a.csr_col[pos + e.rank] = e.col;
}

__global__ __launch_bounds__(kBlock) void k_csc_fill(BuildArgs a)
{
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= a.B * a.N)
        return;
    const int b = r / a.N, i = r - b * a.N;
    for (int t = a.row_ptr[r]; t < a.row_ptr[r + 1]; ++t) {
        const int gc = b * a.M + a.csr_col[t];
        const int k = atomicAdd(&a.col_fill[gc], 1);
        const int p = a.col_ptr[gc] + k;
        a.tmp_row[p] = i;
        a.tmp_src[p] = t;
        a.tmp_gc[p] = gc;
    }
}

// Canonical order inside each column (increasing row), independent of the
// order in which k_csc_fill's atomics placed the entries.
__global__ __launch_bounds__(kBlock) void k_csc_sort(BuildArgs a)
{
    const int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (p >= a.nnz)
        return;
    const int gc = a.tmp_gc[p];
    const int s0 = a.col_ptr[gc], s1 = a.col_ptr[gc + 1];
    const int key = a.tmp_row[p];
    int rank = 0;
    for (int q = s0; q < s1; ++q)
        rank += a.tmp_row[q] < key;
    a.csc_row[s0 + rank] = key;
    a.csc_perm[s0 + rank] = a.tmp_src[p];
}

// ---------------------------------------------------------------------------
// temperatures and softmaxes on the stored pairs
// ---------------------------------------------------------------------------

// Row direction (Alg. 1 step 1): find the stored positions of the minimum
// and second minimum, temperature (Eq. 1 with the clamp), kept-sum softmax.
__global__ __launch_bounds__(kBlock) void k_row_softmax(SoftmaxArgs a, Params p)
{
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= a.B * a.N)
        return;
    const int b = r / a.N;
    const float *xr = a.x + (size_t)r * 3;
    const float *yb = a.y + (size_t)b * a.M * 3;
    const float2 m = a.m12_row[r];
    const int t0 = a.row_ptr[r], t1 = a.row_ptr[r + 1];
    if (t1 - t0 < 2) { // a row always stores its minimum and second minimum
        atomicOr(&a.ctr->error, 1u);
        a.T_row[r] = 0.0;
        a.C1_row[r] = 0.0;
        a.g_row[r] = 1.0;
        a.pos_row[2 * (size_t)r] = a.pos_row[2 * (size_t)r + 1] = -1;
        a.clamp_row[r] = 1;
        for (int t = t0; t < t1; ++t) {
            a.p_row[t] = 0.0f;
            a.flags[t] = 0;
        }
        return;
    }
    int q1 = -1, q2 = -1;
    for (int t = t0; t < t1; ++t) {
        const float *yj = yb + 3 * (size_t)a.csr_col[t];
        const float s = sqdist_f32(xr[0], xr[1], xr[2], yj[0], yj[1], yj[2]);
        if (s == m.x && q1 < 0)
            q1 = t;
        else if (s == m.y && q2 < 0)
            q2 = t;
    }
    if (q1 < 0 || q2 < 0) {
        atomicOr(&a.ctr->error, 1u);
        q1 = q2 = t0;
    }
    const double c1 = dist_f64(xr, yb + 3 * (size_t)a.csr_col[q1]);
    const double c2 = dist_f64(xr, yb + 3 * (size_t)a.csr_col[q2]);
    const double gap = (c2 - c1) + p.delta;
    const bool clamped = gap < p.eps_gap;
    const double g = clamped ? p.eps_gap : gap;
    const double T = p.lk_row / g;
    double z = 0.0;
    for (int t = t0; t < t1; ++t) {
        const double s = exp(-T * (dist_f64(xr, yb + 3 * (size_t)a.csr_col[t]) - c1));
        if (s >= p.tau)
            z += s;
    }
    for (int t = t0; t < t1; ++t) {
        const double s = exp(-T * (dist_f64(xr, yb + 3 * (size_t)a.csr_col[t]) - c1));
        const bool keep = s >= p.tau;
        a.p_row[t] = keep ? (float)(s / z) : 0.0f;
        a.flags[t] = keep ? 1 : 0;
    }
    a.T_row[r] = T;
    a.C1_row[r] = c1;
    a.g_row[r] = g;
    a.pos_row[2 * (size_t)r] = q1;
    a.pos_row[2 * (size_t)r + 1] = q2;
    a.clamp_row[r] = clamped;
}

// Column direction (Alg. 1 step 2) and the symmetrized plan
// P0 = (P_row + P_col)/2 on the union support (Sec. III-C).
__global__ __launch_bounds__(kBlock) void k_col_softmax(SoftmaxArgs a, Params p)
{
    const int gc = blockIdx.x * kBlock + threadIdx.x;
    if (gc >= a.B * a.M)
        return;
    const int b = gc / a.M;
    const float *yc = a.y + (size_t)gc * 3;
    const float *xb = a.x + (size_t)b * a.N * 3;
    const float2 m = a.m12_col[gc];
    const int s0 = a.col_ptr[gc], s1 = a.col_ptr[gc + 1];
    if (s1 - s0 < 2) {
        atomicOr(&a.ctr->error, 2u);
        a.T_col[gc] = 0.0;
        a.C1_col[gc] = 0.0;
        a.g_col[gc] = 1.0;
        a.pos_col[2 * (size_t)gc] = a.pos_col[2 * (size_t)gc + 1] = -1;
        a.clamp_col[gc] = 1;
        for (int q = s0; q < s1; ++q) {
            const int t = a.csc_perm[q];
            a.p_col[q] = 0.0f;
            a.p0c[q] = a.p0r[t] = 0.5f * a.p_row[t];
        }
        return;
    }
    int q1 = -1, q2 = -1;
    for (int q = s0; q < s1; ++q) {
        const float *xi = xb + 3 * (size_t)a.csc_row[q];
        const float s = sqdist_f32(yc[0], yc[1], yc[2], xi[0], xi[1], xi[2]);
        if (s == m.x && q1 < 0)
            q1 = q;
        else if (s == m.y && q2 < 0)
            q2 = q;
    }
    if (q1 < 0 || q2 < 0) {
        atomicOr(&a.ctr->error, 2u);
        q1 = q2 = s0;
    }
    const double c1 = dist_f64(xb + 3 * (size_t)a.csc_row[q1], yc);
    const double c2 = dist_f64(xb + 3 * (size_t)a.csc_row[q2], yc);
    const double gap = (c2 - c1) + p.delta;
    const bool clamped = gap < p.eps_gap;
    const double g = clamped ? p.eps_gap : gap;
    const double T = p.lk_col / g;
    double z = 0.0;
    for (int q = s0; q < s1; ++q) {
        const double s = exp(-T * (dist_f64(xb + 3 * (size_t)a.csc_row[q], yc) - c1));
        if (s >= p.tau)
            z += s;
    }
    for (int q = s0; q < s1; ++q) {
        const double s = exp(-T * (dist_f64(xb + 3 * (size_t)a.csc_row[q], yc) - c1));
        const bool keep = s >= p.tau;
        const double pc = keep ? s / z : 0.0;
        const int t = a.csc_perm[q];
        a.flags[t] = (uint8_t)(a.flags[t] | (keep ? 2 : 0));
        const float p0 = (float)(0.5 * ((double)a.p_row[t] + pc));
        a.p_col[q] = (float)pc;
        a.p0c[q] = p0;
        a.p0r[t] = p0;
    }
    a.T_col[gc] = T;
    a.C1_col[gc] = c1;
    a.g_col[gc] = g;
    a.pos_col[2 * (size_t)gc] = q1;
    a.pos_col[2 * (size_t)gc + 1] = q2;
    a.clamp_col[gc] = clamped;
}

// ---------------------------------------------------------------------------
// Sinkhorn in scaling form: v = alpha_i P0 beta_j. A column step of Eq. 3
// divides a whole column by S_j + eps, i.e. beta_j /= S_j + eps with
// S_j = beta_j sum_i alpha_i P0_ij; a row step (Eq. 4) likewise for alpha.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_fill_ones(double *a, int n)
{
    const int k = blockIdx.x * kBlock + threadIdx.x;
    if (k < n)
        a[k] = 1.0;
}

__global__ __launch_bounds__(kBlock) void k_sink_col(SinkhornArgs a, int l, double eps)
{
    const int gc = blockIdx.x * kBlock + threadIdx.x;
    if (gc >= a.B * a.M)
        return;
    const int b = gc / a.M;
    const size_t BN = (size_t)a.B * a.N, BM = (size_t)a.B * a.M;
    const double *alpha_prev = a.alpha + (size_t)(l - 1) * BN + (size_t)b * a.N;
    double acc = 0.0;
    for (int q = a.col_ptr[gc]; q < a.col_ptr[gc + 1]; ++q)
        acc += (double)a.p0c[q] * alpha_prev[a.csc_row[q]];
    const double bprev = a.beta[(size_t)(l - 1) * BM + gc];
    const double den = bprev * acc + eps;
    a.beta[(size_t)l * BM + gc] = bprev / den;
    a.sden[(size_t)(l - 1) * BM + gc] = den;
}

__global__ __launch_bounds__(kBlock) void k_sink_row(SinkhornArgs a, int l, double eps)
{
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= a.B * a.N)
        return;
    const int b = r / a.N;
    const size_t BN = (size_t)a.B * a.N, BM = (size_t)a.B * a.M;
    const double *beta_cur = a.beta + (size_t)l * BM + (size_t)b * a.M;
    double acc = 0.0;
    for (int t = a.row_ptr[r]; t < a.row_ptr[r + 1]; ++t)
        acc += (double)a.p0r[t] * beta_cur[a.csr_col[t]];
    const double aprev = a.alpha[(size_t)(l - 1) * BN + r];
    const double den = aprev * acc + eps;
    a.alpha[(size_t)l * BN + r] = aprev / den;
    a.rden[(size_t)(l - 1) * BN + r] = den;
}

// ---------------------------------------------------------------------------
// loss
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_loss_rows(LossArgs a)
{
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= a.B * a.N)
        return;
    const int b = r / a.N;
    const float *xr = a.x + (size_t)r * 3;
    const float *yb = a.y + (size_t)b * a.M * 3;
    const double *beta = a.beta_L + (size_t)b * a.M;
    double acc = 0.0;
    for (int t = a.row_ptr[r]; t < a.row_ptr[r + 1]; ++t) {
        const int j = a.csr_col[t];
        acc += (double)a.p0r[t] * beta[j] * dist_f64(xr, yb + 3 * (size_t)j);
    }
    a.loss_rows[r] = a.alpha_L[r] * acc;
}

__global__ __launch_bounds__(kBlock) void k_loss_reduce(LossArgs a)
{
    __shared__ double part[kBlock / 64];
    const int b = blockIdx.x;
    double s = 0.0;
    for (int i = threadIdx.x; i < a.N; i += kBlock)
        s += a.loss_rows[(size_t)b * a.N + i];
    for (int off = 32; off > 0; off >>= 1)
        s += __shfl_xor(s, off);
    if (lane_id() == 0)
        part[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = 0.0;
        for (int w = 0; w < kBlock / 64; ++w)
            t += part[w];
        a.loss[b] = (float)t;
    }
}

// ---------------------------------------------------------------------------
// backward
// ---------------------------------------------------------------------------

// Adjoint of the row scaling of iteration l (Eq. 4): with u = w/(R+eps),
// R = sum_row w:  wbar = (ubar - sum_row ubar*u) / (R + eps). For the last
// iteration ubar = grad_loss * C (loss = sum v C).
__global__ __launch_bounds__(kBlock) void k_bwd_sink_row(BackwardArgs a, int l)
{
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= a.B * a.N)
        return;
    const int b = r / a.N;
    const size_t BN = (size_t)a.B * a.N, BM = (size_t)a.B * a.M;
    const float *xr = a.x + (size_t)r * 3;
    const float *yb = a.y + (size_t)b * a.M * 3;
    const double al = a.alpha[(size_t)l * BN + r];
    const double *bl = a.beta + (size_t)l * BM + (size_t)b * a.M;
    const bool first = l == a.L;
    const double gl = a.grad_loss[b];
    const int t0 = a.row_ptr[r], t1 = a.row_ptr[r + 1];
    double d = 0.0;
    for (int t = t0; t < t1; ++t) {
        const int j = a.csr_col[t];
        const double ub = first ? gl * dist_f64(xr, yb + 3 * (size_t)j) : a.adj[t];
        d += ub * (al * (double)a.p0r[t] * bl[j]);
    }
    const double den = a.rden[(size_t)(l - 1) * BN + r];
    for (int t = t0; t < t1; ++t) {
        const double ub = first ? gl * dist_f64(xr, yb + 3 * (size_t)a.csr_col[t]) : a.adj[t];
        a.adj[t] = (ub - d) / den;
    }
}

// Adjoint of the column scaling of iteration l (Eq. 3), same form with the
// plan w = alpha^(l-1) P0 beta^l before the row step.
__global__ __launch_bounds__(kBlock) void k_bwd_sink_col(BackwardArgs a, int l)
{
    const int gc = blockIdx.x * kBlock + threadIdx.x;
    if (gc >= a.B * a.M)
        return;
    const int b = gc / a.M;
    const size_t BN = (size_t)a.B * a.N, BM = (size_t)a.B * a.M;
    const double *ap = a.alpha + (size_t)(l - 1) * BN + (size_t)b * a.N;
    const double bl = a.beta[(size_t)l * BM + gc];
    const int s0 = a.col_ptr[gc], s1 = a.col_ptr[gc + 1];
    double e = 0.0;
    for (int q = s0; q < s1; ++q)
        e += a.adj[a.csc_perm[q]] * (ap[a.csc_row[q]] * (double)a.p0c[q] * bl);
    const double den = a.sden[(size_t)(l - 1) * BM + gc];
    for (int q = s0; q < s1; ++q) {
        const int t = a.csc_perm[q];
        a.adj[t] = (a.adj[t] - e) / den;
    }
}

// Column softmax and column temperature adjoints. With P = s/Z on the kept
// set, s = exp(-T (C - C1)): abar = P (Pbar - sum P Pbar), Cbar = -T abar,
// Tbar = -sum abar (C - C1); T = L_K/g gives gbar = -Tbar T/g, which reaches
// the cost of the second minimum (+) and of the minimum (-) when not clamped.
// Writes the column part of the cost adjoint for every stored pair.
__global__ __launch_bounds__(kBlock) void k_bwd_col_softmax(BackwardArgs a, Params p)
{
    const int gc = blockIdx.x * kBlock + threadIdx.x;
    if (gc >= a.B * a.M)
        return;
    const int b = gc / a.M;
    const float *yc = a.y + (size_t)gc * 3;
    const float *xb = a.x + (size_t)b * a.N * 3;
    const bool direct = a.L == 0;
    const double gl = a.grad_loss[b];
    const int s0 = a.col_ptr[gc], s1 = a.col_ptr[gc + 1];
    double sigma = 0.0;
    for (int q = s0; q < s1; ++q) {
        const int t = a.csc_perm[q];
        if (!(a.flags[t] & 2))
            continue;
        const double p0bar = direct ? gl * dist_f64(xb + 3 * (size_t)a.csc_row[q], yc) : a.adj[t];
        sigma += (double)a.p_col[q] * 0.5 * p0bar;
    }
    const double T = a.T_col[gc], c1 = a.C1_col[gc];
    double tbar = 0.0;
    for (int q = s0; q < s1; ++q) {
        const int t = a.csc_perm[q];
        if (!(a.flags[t] & 2))
            continue;
        const double c = dist_f64(xb + 3 * (size_t)a.csc_row[q], yc);
        const double p0bar = direct ? gl * c : a.adj[t];
        const double ab = (double)a.p_col[q] * (0.5 * p0bar - sigma);
        tbar -= ab * (c - c1);
    }
    const double gapbar = a.clamp_col[gc] ? 0.0 : -tbar * T / a.g_col[gc];
    const int q1 = a.pos_col[2 * (size_t)gc], q2 = a.pos_col[2 * (size_t)gc + 1];
    for (int q = s0; q < s1; ++q) {
        const int t = a.csc_perm[q];
        double cb = 0.0;
        if (a.flags[t] & 2) {
            const double p0bar = direct ? gl * dist_f64(xb + 3 * (size_t)a.csc_row[q], yc) : a.adj[t];
            cb = -T * (double)a.p_col[q] * (0.5 * p0bar - sigma);
        }
        if (q == q2)
            cb += gapbar;
        if (q == q1)
            cb -= gapbar;
        a.cbar[t] = cb;
    }
}

// Row softmax and row temperature adjoints, the direct term grad_loss * v of
// the loss, and the distance gradient (Eq. 5) summed into grad_x.
__global__ __launch_bounds__(kBlock) void k_bwd_row_softmax(BackwardArgs a, Params p, int keep_cbar)
{
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= a.B * a.N)
        return;
    const int b = r / a.N;
    const size_t BN = (size_t)a.B * a.N, BM = (size_t)a.B * a.M;
    const float *xr = a.x + (size_t)r * 3;
    const float *yb = a.y + (size_t)b * a.M * 3;
    const bool direct = a.L == 0;
    const double gl = a.grad_loss[b];
    const int t0 = a.row_ptr[r], t1 = a.row_ptr[r + 1];
    double sigma = 0.0;
    for (int t = t0; t < t1; ++t) {
        if (!(a.flags[t] & 1))
            continue;
        const double p0bar = direct ? gl * dist_f64(xr, yb + 3 * (size_t)a.csr_col[t]) : a.adj[t];
        sigma += (double)a.p_row[t] * 0.5 * p0bar;
    }
    const double T = a.T_row[r], c1 = a.C1_row[r];
    double tbar = 0.0;
    for (int t = t0; t < t1; ++t) {
        if (!(a.flags[t] & 1))
            continue;
        const double c = dist_f64(xr, yb + 3 * (size_t)a.csr_col[t]);
        const double p0bar = direct ? gl * c : a.adj[t];
        const double ab = (double)a.p_row[t] * (0.5 * p0bar - sigma);
        tbar -= ab * (c - c1);
    }
    const double gapbar = a.clamp_row[r] ? 0.0 : -tbar * T / a.g_row[r];
    const int q1 = a.pos_row[2 * (size_t)r], q2 = a.pos_row[2 * (size_t)r + 1];
    const double al = a.alpha[(size_t)a.L * BN + r];
    const double *bl = a.beta + (size_t)a.L * BM + (size_t)b * a.M;
    double gx = 0.0, gy = 0.0, gz = 0.0;
    for (int t = t0; t < t1; ++t) {
        const int j = a.csr_col[t];
        const float *yj = yb + 3 * (size_t)j;
        const double c = dist_f64(xr, yj);
        double cb = a.cbar[t] + gl * (al * (double)a.p0r[t] * bl[j]);
        if (a.flags[t] & 1) {
            const double p0bar = direct ? gl * c : a.adj[t];
            cb -= T * (double)a.p_row[t] * (0.5 * p0bar - sigma);
        }
        if (t == q2)
            cb += gapbar;
        if (t == q1)
            cb -= gapbar;
        const double w = cb / (c + p.eps_dist);
        gx += w * ((double)xr[0] - (double)yj[0]);
        gy += w * ((double)xr[1] - (double)yj[1]);
        gz += w * ((double)xr[2] - (double)yj[2]);
        if (keep_cbar)
            a.cbar[t] = cb;
    }
    float *o = a.grad_x + (size_t)r * 3;
    o[0] = (float)gx;
    o[1] = (float)gy;
    o[2] = (float)gz;
}

__global__ __launch_bounds__(kBlock) void k_bwd_grad_y(BackwardArgs a, Params p)
{
    const int gc = blockIdx.x * kBlock + threadIdx.x;
    if (gc >= a.B * a.M)
        return;
    const int b = gc / a.M;
    const float *yc = a.y + (size_t)gc * 3;
    const float *xb = a.x + (size_t)b * a.N * 3;
    double gx = 0.0, gy = 0.0, gz = 0.0;
    for (int q = a.col_ptr[gc]; q < a.col_ptr[gc + 1]; ++q) {
        const float *xi = xb + 3 * (size_t)a.csc_row[q];
        const double c = dist_f64(xi, yc);
        const double w = a.cbar[a.csc_perm[q]] / (c + p.eps_dist);
        gx -= w * ((double)xi[0] - (double)yc[0]);
        gy -= w * ((double)xi[1] - (double)yc[1]);
        gz -= w * ((double)xi[2] - (double)yc[2]);
    }
    float *o = a.grad_y + (size_t)gc * 3;
    o[0] = (float)gx;
    o[1] = (float)gy;
    o[2] = (float)gz;
}

__global__ __launch_bounds__(kBlock) void k_count_support(const int32_t *row_ptr,
                                                          const uint8_t *flags, int N,
                                                          unsigned long long *out)
{
    __shared__ unsigned long long part[kBlock / 64];
    const int b = blockIdx.x;
    const int t0 = row_ptr[(size_t)b * N], t1 = row_ptr[(size_t)(b + 1) * N];
    unsigned long long n = 0;
    for (int t = t0 + threadIdx.x; t < t1; t += kBlock)
        n += flags[t] != 0;
    for (int off = 32; off > 0; off >>= 1)
        n += __shfl_xor(n, off);
    if (lane_id() == 0)
        part[threadIdx.x >> 6] = n;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long s = 0;
        for (int w = 0; w < kBlock / 64; ++w)
            s += part[w];
        out[b] = s;
    }
}

inline unsigned blocks_for(int64_t n) { return (unsigned)((n + kBlock - 1) / kBlock); }

} // namespace

// ---------------------------------------------------------------------------
// launch wrappers
// ---------------------------------------------------------------------------

void launch_top2(const ScanDir &rows, const ScanDir &cols, int B, hipStream_t s)
{
    Top2Args a{{rows, cols}, B};
    hipLaunchKernelGGL(k_top2, dim3(rows.tiles + cols.tiles), dim3(kBlock), 0, s, a);
}

void launch_finalize(const FinalizeDir &rows, const FinalizeDir &cols, int B, const Params &p,
                     hipStream_t s)
{
    FinalizeArgs a{{rows, cols}, B, B * rows.n_own, p};
    hipLaunchKernelGGL(k_finalize, dim3(blocks_for((int64_t)B * (rows.n_own + cols.n_own))),
                       dim3(kBlock), 0, s, a);
}

void launch_emit(const EmitArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_emit, dim3(a.B * a.S * a.owner_blocks), dim3(kBlock), 0, s, a);
}

int scan_tile_items() { return kScanTile; }

void launch_scan(const ScanArray &a0, const ScanArray &a1, hipStream_t s)
{
    ScanPair sp{{a0, a1}};
    const int tiles = a0.tiles > a1.tiles ? a0.tiles : a1.tiles;
    hipLaunchKernelGGL(k_scan_reduce, dim3(tiles, 2), dim3(kBlock), 0, s, sp);
    hipLaunchKernelGGL(k_scan_tiles, dim3(1, 2), dim3(kBlock), 0, s, sp);
    hipLaunchKernelGGL(k_scan_apply, dim3(tiles, 2), dim3(kBlock), 0, s, sp);
}

void launch_build(const BuildArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_csr_fill, dim3(blocks_for((int64_t)a.B * a.N)), dim3(kBlock), 0, s, a);
    if (a.n_ovf > 0)
        hipLaunchKernelGGL(k_ovf_fill, dim3(blocks_for(a.n_ovf)), dim3(kBlock), 0, s, a);
    hipLaunchKernelGGL(k_csc_fill, dim3(blocks_for((int64_t)a.B * a.N)), dim3(kBlock), 0, s, a);
    if (a.nnz > 0)
        hipLaunchKernelGGL(k_csc_sort, dim3(blocks_for(a.nnz)), dim3(kBlock), 0, s, a);
}

void launch_softmax(const SoftmaxArgs &a, const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(k_row_softmax, dim3(blocks_for((int64_t)a.B * a.N)), dim3(kBlock), 0, s, a, p);
    hipLaunchKernelGGL(k_col_softmax, dim3(blocks_for((int64_t)a.B * a.M)), dim3(kBlock), 0, s, a, p);
}

void launch_sinkhorn_init(const SinkhornArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_fill_ones, dim3(blocks_for((int64_t)a.B * a.N)), dim3(kBlock), 0, s,
                       a.alpha, a.B * a.N);
    hipLaunchKernelGGL(k_fill_ones, dim3(blocks_for((int64_t)a.B * a.M)), dim3(kBlock), 0, s,
                       a.beta, a.B * a.M);
}

void launch_sinkhorn_step(const SinkhornArgs &a, int l, double eps, hipStream_t s)
{
    hipLaunchKernelGGL(k_sink_col, dim3(blocks_for((int64_t)a.B * a.M)), dim3(kBlock), 0, s, a, l, eps);
    hipLaunchKernelGGL(k_sink_row, dim3(blocks_for((int64_t)a.B * a.N)), dim3(kBlock), 0, s, a, l, eps);
}

void launch_loss(const LossArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_loss_rows, dim3(blocks_for((int64_t)a.B * a.N)), dim3(kBlock), 0, s, a);
    hipLaunchKernelGGL(k_loss_reduce, dim3(a.B), dim3(kBlock), 0, s, a);
}

void launch_bwd_sinkhorn_step(const BackwardArgs &a, int l, hipStream_t s)
{
    hipLaunchKernelGGL(k_bwd_sink_row, dim3(blocks_for((int64_t)a.B * a.N)), dim3(kBlock), 0, s, a, l);
    hipLaunchKernelGGL(k_bwd_sink_col, dim3(blocks_for((int64_t)a.B * a.M)), dim3(kBlock), 0, s, a, l);
}

void launch_bwd_softmax(const BackwardArgs &a, const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(k_bwd_col_softmax, dim3(blocks_for((int64_t)a.B * a.M)), dim3(kBlock), 0, s, a, p);
    hipLaunchKernelGGL(k_bwd_row_softmax, dim3(blocks_for((int64_t)a.B * a.N)), dim3(kBlock), 0, s, a, p,
                       a.grad_y != nullptr ? 1 : 0);
    if (a.grad_y)
        hipLaunchKernelGGL(k_bwd_grad_y, dim3(blocks_for((int64_t)a.B * a.M)), dim3(kBlock), 0, s, a, p);
}

void launch_count_support(const int32_t *row_ptr, const uint8_t *flags, int B, int N,
                          unsigned long long *out, hipStream_t s)
{
    hipLaunchKernelGGL(k_count_support, dim3(B), dim3(kBlock), 0, s, row_ptr, flags, N, out);
}

} // namespace apml
